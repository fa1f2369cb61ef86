// Recompute backward of ring-chunked attention, dQ part at head size 64: bf16 MFMA with fp32
// accumulation (gfx950).  At d = 64 a score element carries more vector work per matrix product
// than one wave can hide behind its own products, so this kernel runs two waves per SIMD (the
// d = 128 kernel in bwd_dq_bf16.hip runs one wave per SIMD on a fixed software-pipelined schedule).
//
// Query-stationary, like the forward: one workgroup = 8 waves = one (b, h) and 256 queries (32
// per wave).  The key/value sequence is streamed chunk by chunk (ring steps, arXiv 2507.16697
// Sec. III-A) in tiles of 64 keys that never straddle a chunk, double buffered in LDS and filled
// by direct global->LDS loads one tile ahead.  dQ accumulates over every tile of every chunk in
// fp32 registers and is written once, so it needs no atomics (the paper's "gradient for Q
// accumulated over N steps").  Per tile, with lane = query n and g = lane / 32:
//   S^T  = K Q^T      A = K rows (LDS),  B = Q^T from registers
//   dP^T = V dO^T     A = V rows (LDS),  B = dO^T from registers
//   P^T  = exp2(S^T * scale*log2e - lse_q*log2e),  dS^T = P^T (dP^T - D_q)   (lse_q, D_q are
//          per-lane scalars because each lane holds one query)
//   dQ^T += K^T dS^T  A = K^T by transposed reads of the row-major K tile, B = dS^T from the
//          registers (keys 4g..4g+3, 8+4g..8+4g+3 of each 16-key step, as in the forward)

#include "ringx_device.h"
#include "ringx_kernels.h"

namespace ringx {
namespace {

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

template <int D>
struct DqCfg {
  static constexpr int kThreads = 512;
  static constexpr int kWaves = 8;
  static constexpr int kQW = 32;
  static constexpr int kBQ = kWaves * kQW;
  static constexpr int kBK = 64;                   // keys per tile
  static constexpr int kRowBytes = D * 2;
  static constexpr int kChunks = D / 8;
  static constexpr int kTileBytes = kBK * kRowBytes;
  static constexpr int kKTiles = kBK / 32;
  static constexpr int kDSteps = D / 16;
  static constexpr int kKSteps = kBK / 16;
  static constexpr int kCT = D / 32;
  static constexpr int kLoads = kTileBytes / (kThreads * 16);
};

template <int D>
__device__ __forceinline__ int swz(int row) {
  if constexpr (D == 128) return ((row & 3) << 2) | ((row >> 2) & 3);
  else return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
}
template <int D>
__device__ __forceinline__ int tile_off(int row, int c) {
  return row * (D * 2) + ((c ^ swz<D>(row)) << 4);
}

template <int D>
__device__ __forceinline__ void load_offsets(int (&goff)[DqCfg<D>::kLoads],
                                             int (&grow)[DqCfg<D>::kLoads], int wave, int lane) {
  using C = DqCfg<D>;
#pragma unroll
  for (int u = 0; u < C::kLoads; ++u) {
    const int slot = (u * C::kWaves + wave) * 64 + lane;
    const int row = slot / C::kChunks;
    const int c = (slot % C::kChunks) ^ swz<D>(row);
    grow[u] = row;
    goff[u] = row * C::kRowBytes + c * 16;
  }
}

// Direct loads of one K/V tile starting at key `start`; rows at or past `hi` (only in the last
// tile of a chunk) are clamped to hi - 1.  Scalar tile bases plus 32-bit lane offsets.
template <int D>
__device__ __forceinline__ void issue_tile(const char* __restrict__ kb,
                                           const char* __restrict__ vb, uint32_t kdst,
                                           uint32_t vdst, uint32_t start, uint32_t hi,
                                           const int (&goff)[DqCfg<D>::kLoads],
                                           const int (&grow)[DqCfg<D>::kLoads], int wave) {
  using C = DqCfg<D>;
  const char* kt = kb + (uint64_t)start * C::kRowBytes;
  const char* vt = vb + (uint64_t)start * C::kRowBytes;
  if (start + C::kBK <= hi) {
#pragma unroll
    for (int u = 0; u < C::kLoads; ++u) {
      const uint32_t wbase =
          (uint32_t)__builtin_amdgcn_readfirstlane((u * C::kWaves + wave) * 1024);
      load_lds16_s(kt, (uint32_t)goff[u], kdst + wbase);
      load_lds16_s(vt, (uint32_t)goff[u], vdst + wbase);
    }
  } else {
    cold_path();
    const int last = (int)(hi - 1 - start);
#pragma unroll
    for (int u = 0; u < C::kLoads; ++u) {
      const int off = grow[u] <= last ? goff[u] : goff[u] - (grow[u] - last) * C::kRowBytes;
      const uint32_t wbase =
          (uint32_t)__builtin_amdgcn_readfirstlane((u * C::kWaves + wave) * 1024);
      load_lds16_s(kt, (uint32_t)off, kdst + wbase);
      load_lds16_s(vt, (uint32_t)off, vdst + wbase);
    }
  }
}

template <int D>
__global__ __launch_bounds__(512, 1) void bwd_dq_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    const __bf16* __restrict__ dout, const float* __restrict__ lse,
    const float* __restrict__ delta, float* __restrict__ dq, int BH, int H, int grp, int64_t Nq,
    int64_t Nk, int R, float c2, float scale, int accumulate) {
  using C = DqCfg<D>;
  __shared__ __attribute__((aligned(1024))) char lds_k[2 * C::kTileBytes];
  __shared__ __attribute__((aligned(1024))) char lds_v[2 * C::kTileBytes];

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int n = lane & 31;
  const int g = lane >> 5;

  const int64_t nqt = (Nq + C::kBQ - 1) / C::kBQ;
  const uint32_t wg = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t bh = wg / nqt;
  const int64_t q0 = (wg % nqt) * C::kBQ + wave * C::kQW;
  if (bh >= BH) return;

  const int64_t kvh = kv_head(bh, H, grp);
  const char* kb =
      static_cast<const char*>(uniform_ptr(reinterpret_cast<const char*>(k + kvh * Nk * D)));
  const char* vb =
      static_cast<const char*>(uniform_ptr(reinterpret_cast<const char*>(v + kvh * Nk * D)));
  int goff[C::kLoads], grow[C::kLoads];
  load_offsets<D>(goff, grow, wave, lane);

  // the chunked key sequence, one tile at a time (32-bit positions, no divisions)
  const uint32_t nk = (uint32_t)Nk;
  ChunkWalk walk{nk, nk / (uint32_t)R, nk % (uint32_t)R, 0, (uint32_t)R};
  KeyTile ct = walk.first();

  const uint32_t lk = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_k;
  const uint32_t lv = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_v;
  issue_tile<D>(kb, vb, lk, lv, ct.start, ct.hi, goff, grow, wave);

  // this lane's query: Q and dO fragments (B operands), -lse*log2e and D
  int64_t qi = q0 + n;
  const bool q_ok = qi < Nq;
  qi = q_ok ? qi : Nq - 1;
  bf16x8 qf[C::kDSteps], of[C::kDSteps];
  {
    const __bf16* qr = q + (bh * Nq + qi) * D;
    const __bf16* orow = dout + (bh * Nq + qi) * D;
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s) {
      qf[s] = *reinterpret_cast<const bf16x8*>(qr + s * 16 + g * 8);
      of[s] = *reinterpret_cast<const bf16x8*>(orow + s * 16 + g * 8);
    }
  }
  const float nl = -lse[bh * Nq + qi] * kLog2e;
  const float dq_d = delta[bh * Nq + qi];
  // the dP accumulators start from -D (the same for every key of this lane's query), so that they
  // come out of the matrix cores as dP - D
  f32x16 pinit;
#pragma unroll
  for (int rr = 0; rr < 16; ++rr) pinit[rr] = -dq_d;

  int koff[C::kDSteps];
#pragma unroll
  for (int s = 0; s < C::kDSteps; ++s) koff[s] = tile_off<D>(n, 2 * s + g);
  int toff[2][C::kCT];
  {
    const int G = lane >> 4;
    const int rr = (lane & 15) >> 2;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int ct = 0; ct < C::kCT; ++ct) {
        const int row = 4 * g + 8 * h + rr;
        const int col = 32 * ct + 16 * (G & 1) + 4 * (lane & 3);
        toff[h][ct] = tile_off<D>(row, col >> 3) + (col & 7) * 2;
      }
  }
  // The offsets address buffer `cur` of the K and V rings: an exclusive or with kTileBytes at the
  // end of every tile switches them to the other buffer (their lane parts stay below it), so each
  // read is one register plus an immediate.  Opaque, so that the compiler keeps them so.
  static_assert(32 * C::kRowBytes <= C::kTileBytes && (C::kTileBytes & (C::kTileBytes - 1)) == 0,
                "lane offsets below one tile, whose size is a power of two");
#pragma unroll
  for (int s = 0; s < C::kDSteps; ++s) asm volatile("" : "+v"(koff[s]));
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int c = 0; c < C::kCT; ++c) asm volatile("" : "+v"(toff[h][c]));

  f32x16 dqacc[C::kCT];
#pragma unroll
  for (int c = 0; c < C::kCT; ++c) dqacc[c] = f32x16{};

  int cur = 0;
  wait_vmem_all();
  __syncthreads();

  while (true) {
    const KeyTile nt = walk.next<C::kBK>(ct);
    const bool has_next = nt.start < nk;
    if (has_next)
      issue_tile<D>(kb, vb, lk + (cur ^ 1) * C::kTileBytes, lv + (cur ^ 1) * C::kTileBytes,
                    nt.start, nt.hi, goff, grow, wave);

    const char* kbuf = lds_k;   // koff and toff hold the buffer
    const char* vbuf = lds_v;
    const int nvalid = (int)min<uint32_t>(C::kBK, ct.hi - ct.start);

    f32x16 sacc[C::kKTiles], pacc[C::kKTiles];
#pragma unroll
    for (int kt = 0; kt < C::kKTiles; ++kt) {
      sacc[kt] = f32x16{};
      pacc[kt] = pinit;
    }
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s) {
#pragma unroll
      for (int kt = 0; kt < C::kKTiles; ++kt) {
        const int off = koff[s] + kt * 32 * C::kRowBytes;
        const bf16x8 ak = *reinterpret_cast<const bf16x8*>(kbuf + off);
        const bf16x8 av = *reinterpret_cast<const bf16x8*>(vbuf + off);
        sacc[kt] = mfma32(ak, qf[s], sacc[kt]);
        pacc[kt] = mfma32(av, of[s], pacc[kt]);
      }
    }
    if (nvalid < C::kBK) {
      cold_path();
#pragma unroll
      for (int kt = 0; kt < C::kKTiles; ++kt)
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int key = kt * 32 + 8 * (rr >> 2) + 4 * g + (rr & 3);
          if (key >= nvalid) sacc[kt][rr] = -INFINITY;
        }
    }
    // dS^T, packed as the B operand of the key-contraction (keys 8*(e/4) + 4g + e%4)
    bf16x8 sf[C::kKSteps];
#pragma unroll
    for (int kt = 0; kt < C::kKTiles; ++kt) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r0 = 8 * h + 2 * e;
          const float p0 = fast_exp2(__builtin_fmaf(sacc[kt][r0], c2, nl));
          const float p1 = fast_exp2(__builtin_fmaf(sacc[kt][r0 + 1], c2, nl));
          w[e] = pack_bf16x2(p0 * pacc[kt][r0], p1 * pacc[kt][r0 + 1]);
        }
        sf[2 * kt + h] = __builtin_bit_cast(bf16x8, w);
      }
    }
    // dQ^T += K^T dS^T
#pragma unroll
    for (int s = 0; s < C::kKSteps; ++s) {
#pragma unroll
      for (int c = 0; c < C::kCT; ++c) {
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (lds_bf16x4*)(kbuf + toff[0][c] + s * 16 * C::kRowBytes));
        const bf16x4 hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (lds_bf16x4*)(kbuf + toff[1][c] + s * 16 * C::kRowBytes));
        dqacc[c] = mfma32(__builtin_shufflevector(lo, hi4, 0, 1, 2, 3, 4, 5, 6, 7), sf[s], dqacc[c]);
      }
    }
    // transposed K reads run ahead of the matrix products that consume them
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int i = 0; i < C::kKSteps * C::kCT; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }

    if (!has_next) break;
    wait_vmem_all();
    __syncthreads();
    cur ^= 1;
    ct = nt;
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s) koff[s] ^= C::kTileBytes;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int c = 0; c < C::kCT; ++c) toff[h][c] ^= C::kTileBytes;
  }

  if (q_ok) {
    float* dqr = dq + (bh * Nq + qi) * D;
#pragma unroll
    for (int c = 0; c < C::kCT; ++c)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        f32x4 val = {dqacc[c][4 * rq] * scale, dqacc[c][4 * rq + 1] * scale,
                     dqacc[c][4 * rq + 2] * scale, dqacc[c][4 * rq + 3] * scale};
        f32x4* dst = reinterpret_cast<f32x4*>(dqr + c * 32 + 8 * rq + 4 * g);
        if (accumulate) val += *dst;
        *dst = val;
      }
  }
}

template <int D>
hipError_t launch(const BwdArgs& a) {
  using C = DqCfg<D>;
  const int64_t nqt = (a.Nq + C::kBQ - 1) / C::kBQ;
  const int64_t nwg = nqt * a.BH;
  hipLaunchKernelGGL((bwd_dq_kernel<D>), dim3((uint32_t)nwg), dim3(C::kThreads), 0, a.stream,
                     (const __bf16*)a.q, (const __bf16*)a.k, (const __bf16*)a.v,
                     (const __bf16*)a.dout, a.lse, a.delta, a.dq, (int)a.BH, (int)a.H, (int)a.G,
                     a.Nq, a.Nk,
                     (int)a.R, a.scale * kLog2e, a.scale, a.accumulate_dq ? 1 : 0);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd_dq_bf16_d64(const BwdArgs& a) { return launch<64>(a); }

}  // namespace ringx
