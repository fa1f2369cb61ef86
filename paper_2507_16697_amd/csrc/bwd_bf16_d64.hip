// Recompute backward of ring-chunked attention, dK/dV part at head size 64: bf16 MFMA with fp32
// accumulation (gfx950).  At d = 64 a score element carries twice the vector work per matrix
// product that it does at d = 128, more than one wave can hide behind its own products, so this
// kernel runs two waves per SIMD, each hiding its vector work behind the other's products (the
// d = 128 kernel in bwd_bf16.hip runs one wave per SIMD on a fixed software-pipelined schedule).
//
// One workgroup = 8 waves = one K/V head and a tile of 128 keys inside one chunk (a key tile never
// straddles a chunk boundary).  With the merged log-sum-exp saved by the forward, every chunk's
// gradients are independent (arXiv 2507.16697 Sec. III-A: K/V chunk gradients computed per
// chunk), so the workgroup sweeps every query tile of 128 queries once -- of every query head that
// shares the K/V head when G > 1 query heads share one (grouped-query attention).  Wave w owns keys
// 32*(w%4) .. +31 of the tile and query half w/4 of every query tile, and keeps fp32 dK^T, dV^T
// accumulators for its keys in registers.  Per query tile:
//   S    = Q K^T        A = Q rows (LDS),  B = K rows (LDS)             -> lane = key
//   D-dP = D + dO (-V)^T A = dO rows (LDS), B = -V rows (LDS), accumulators start at D
//   P    = exp2(S*scale*log2e + nl_i),  -dS = P (D - dP)                (fp32; nl_i = -lse_i*log2e
//                                                                       from the preprocess)
//   dV^T += dO^T P       A = dO^T by transposed LDS reads, B = P from registers
//   -dK^T += Q^T (-dS)   A = Q^T by transposed LDS reads,  B = -dS from registers
// (the V tile is negated in LDS once it lands; negating V and dK is exact, and lets the matrix
// cores subtract D)
// Q, dO, nl and D of the next query tile arrive by direct global->LDS loads while the current
// one is processed (double buffered, one barrier per tile).  K and V tiles are row-major in LDS
// with XOR-swizzled 16-byte chunks.  The two waves sharing a key block add their dK/dV through
// LDS at the end.

#include "ringx_device.h"
#include "ringx_kernels.h"


namespace ringx {
namespace {

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

template <int D>
struct DkvCfg {
  static constexpr int kThreads = 512;
  static constexpr int kWaves = 8;
  static constexpr int kBK = 128;                  // keys per workgroup (32 per key block)
  static constexpr int kBQ = 8192 / D;             // queries per tile: 64 (d=128), 128 (d=64)
  static constexpr int kQW = kBQ / 2;              // queries per wave
  static constexpr int kQB = kQW / 32;             // 32-query blocks per wave
  static constexpr int kRowBytes = 2 * D;          // Q, dO, K, V rows
  static constexpr int kDSteps = D / 16;
  static constexpr int kCT = D / 32;
  static constexpr int kQTile = kBQ * kRowBytes;   // bytes of one Q or dO tile (16 KiB)
  static constexpr int kKTile = kBK * kRowBytes;   // bytes of the K or V tile
  // LDS carve-up (bytes): the Q and dO buffers, read at every product, first, so that their
  // offsets fit the 16-bit immediate of the LDS reads; K, V, nl and D are read from registers
  // holding their bases
  static constexpr int kOffQ = 0;                       // 2 buffers
  static constexpr int kOffO = kOffQ + 2 * kQTile;      // 2 buffers
  static constexpr int kOffK = kOffO + 2 * kQTile;
  static constexpr int kOffV = kOffK + kKTile;
  static constexpr int kOffL = kOffV + kKTile;          // 2 x kBQ floats: nl
  static constexpr int kOffD = kOffL + 2 * kBQ * 4;     // 2 x kBQ floats: D
  static constexpr int kLds = kOffD + 2 * kBQ * 4;
  static_assert(kOffK <= 65536, "Q / dO buffers within the LDS immediate offset");
  static_assert(kQB * 32 * 2 == kBQ, "two query halves");
  static_assert(4 * kQTile >= kWaves / 2 * kCT * 16 * 64 * 4, "dK/dV exchange fits");
};

// XOR swizzle of the 16-byte chunks of a row of `RB` bytes (as in the forward kernel): 16
// consecutive rows read at one chunk, and 4 consecutive rows read at 2 chunks by transposed
// reads, hit distinct banks.
template <int RB>
__device__ __forceinline__ int swz(int row) {
  if constexpr (RB == 256) return ((row & 3) << 2) | ((row >> 2) & 3);
  else return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
}
template <int RB>
__device__ __forceinline__ int toff(int row, int c) {
  return row * RB + ((c ^ swz<RB>(row)) << 4);
}
// byte offset of element `col` (2-byte units) of `row`
template <int RB>
__device__ __forceinline__ int eoff(int row, int col) {
  return toff<RB>(row, col >> 3) + (col & 7) * 2;
}

// Rows of a [N, D] bf16 matrix from `src` (the tile's first row, the same for every lane) into a
// swizzled LDS tile at `dst`, rows past `last` (relative to the first) clamped to it, `per_wave`
// 1 KiB blocks per wave.  Scalar base plus 32-bit lane offsets: no per-lane 64-bit addresses.
template <int D>
__device__ __forceinline__ void issue_rows(const __bf16* __restrict__ src, uint32_t dst, int last,
                                           int per_wave, int wave, int lane, int nwaves) {
  constexpr int kCh = D / 8;
  for (int u = 0; u < per_wave; ++u) {
    const int blk = u * nwaves + wave;
    const int slot = blk * 64 + lane;
    const int row = slot / kCh;
    const int c = (slot % kCh) ^ swz<2 * D>(row);
    const int rr = row < last ? row : last;
    load_lds16_s(src, (uint32_t)(rr * 2 * D + c * 16),
                 dst + (uint32_t)__builtin_amdgcn_readfirstlane(blk * 1024));
  }
}

// nl and D of the BQ queries from `nlb` / `deltab` (the tile's first row; rows past `last`
// clamped to it) into LDS, 4 bytes per lane: waves 0 and 1 load nl, waves 2 and 3 load D.
template <int BQ>
__device__ __forceinline__ void issue_rowvals(const float* __restrict__ nlb,
                                              const float* __restrict__ deltab, uint32_t ldst,
                                              uint32_t ddst, int last, int wave, int lane) {
  static_assert(BQ <= 128, "two waves per array");
  const int part = wave & 1;
  if (wave < 4 && part * 64 < BQ) {
    int r = part * 64 + lane;
    r = r < last ? r : last;
    const uint32_t slot = (uint32_t)__builtin_amdgcn_readfirstlane(part * 256);
    if (wave < 2) load_lds4_s(nlb, (uint32_t)(4 * r), ldst + slot);
    else load_lds4_s(deltab, (uint32_t)(4 * r), ddst + slot);
  }
}

template <int D>
__global__ __launch_bounds__(512, 1) void bwd_dkdv_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    const __bf16* __restrict__ dout, const float* __restrict__ nl,
    const float* __restrict__ delta, float* __restrict__ dk, float* __restrict__ dv, int BHkv,
    int H, int grp,
    int64_t Nq, int64_t Nk, int R, int tiles_per_chunk, float c2, float scale, int accumulate) {
  using C = DkvCfg<D>;
  __shared__ __attribute__((aligned(1024))) char lds[C::kLds];
  const uint32_t lbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int n = lane & 31;
  const int g = lane >> 5;
  const int kb = wave & 3;          // key block of this wave
  const int qh = wave >> 2;         // query half of this wave

  const uint32_t wg = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t per_bh = (int64_t)R * tiles_per_chunk;
  const int64_t bh = wg / per_bh;   // K/V head (of B * H / G)
  const int r = (int)((wg % per_bh) / tiles_per_chunk);
  const int tile = (int)(wg % tiles_per_chunk);
  if (bh >= BHkv) return;
  const int64_t lo = (int64_t)r * Nk / R;
  const int64_t hi = (int64_t)(r + 1) * Nk / R;
  const int64_t k0 = lo + (int64_t)tile * C::kBK;
  if (k0 >= hi) return;                         // uniform over the workgroup
  const int nvalid = (int)min<int64_t>(C::kBK, hi - k0);

  const __bf16* kbp = k + bh * Nk * D;
  const __bf16* vbp = v + bh * Nk * D;
  // the grp query heads sharing this K/V head are swept one after the other: query tile it is
  // tile it % nqt of head qh0 + it / nqt
  const int64_t qh0 = (bh / (H / grp)) * H + (bh % (H / grp)) * grp;
  const __bf16* qb = q + qh0 * Nq * D;
  const __bf16* ob = dout + qh0 * Nq * D;
  const float* nlb = nl + qh0 * Nq;
  const float* deltab = delta + qh0 * Nq;

  // query positions within a head are 32-bit (the library takes at most 2^31 - 128 queries
  // per head), so that the tile bookkeeping stays scalar instructions
  const int nq = (int)Nq;
  const int nqt = (nq + C::kBQ - 1) / C::kBQ;

  // K and V tiles (kept for the whole sweep), then the first query tile
  issue_rows<D>(kbp + k0 * D, lbase + C::kOffK, (int)(hi - 1 - k0), C::kKTile / 1024 / C::kWaves,
                wave, lane, C::kWaves);
  issue_rows<D>(vbp + k0 * D, lbase + C::kOffV, (int)(hi - 1 - k0), C::kKTile / 1024 / C::kWaves,
                wave, lane, C::kWaves);
  issue_rows<D>(qb, lbase + C::kOffQ, nq - 1, C::kQTile / 1024 / C::kWaves, wave, lane,
                C::kWaves);
  issue_rows<D>(ob, lbase + C::kOffO, nq - 1, C::kQTile / 1024 / C::kWaves, wave, lane,
                C::kWaves);
  issue_rowvals<C::kBQ>(nlb, deltab, lbase + C::kOffL, lbase + C::kOffD, nq - 1, wave, lane);
  const float* lds_l = reinterpret_cast<const float*>(lds + C::kOffL);
  const float* lds_d = reinterpret_cast<const float*>(lds + C::kOffD);

  // per-lane LDS byte offsets (tile-relative)
  // S / dP: A = Q/dO rows (query qh*kQW + 32*b + n), B = K/V rows (key 32*kb + n); chunk 2s+g
  int aoff[C::kDSteps];
#pragma unroll
  for (int s = 0; s < C::kDSteps; ++s) aoff[s] = toff<2 * D>(n, 2 * s + g);   // + row block
  // transposed reads of Q/dO (rows = queries, cols = dims): 16-lane group G reads rows
  // j0 + (lane%16)/4 with j0 = 4g + 8h (+16*ks), columns 32*ct + 16*(G&1) + 4*(lane%4); lane i
  // of the group receives rows j0..j0+3 of column 32*ct + 16*(G&1) + i.
  const int G = lane >> 4;
  const int trr = (lane & 15) >> 2;
  const int trc = 16 * (G & 1) + 4 * (lane & 3);
  int qtoff[2][C::kCT];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int ct = 0; ct < C::kCT; ++ct)
      qtoff[h][ct] = eoff<2 * D>(4 * g + 8 * h + trr, 32 * ct + trc);
  // the same offsets with this wave's key block (K/V rows) and query half (Q/dO rows, nl and D)
  // folded in, as opaque registers: each read then adds only immediates (buffer, block, step)
  int kvo[C::kDSteps], qo[C::kDSteps], tqo[2][C::kCT];
#pragma unroll
  for (int s = 0; s < C::kDSteps; ++s) {
    kvo[s] = C::kOffK + aoff[s] + 32 * kb * C::kRowBytes;
    qo[s] = aoff[s] + qh * C::kQW * C::kRowBytes;
    asm volatile("" : "+v"(kvo[s]), "+v"(qo[s]));
  }
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int ct = 0; ct < C::kCT; ++ct) {
      tqo[h][ct] = qtoff[h][ct] + qh * C::kQW * C::kRowBytes;
      asm volatile("" : "+v"(tqo[h][ct]));
    }
  int so = C::kOffL + 4 * (qh * C::kQW + 4 * g);   // this lane's first query in the nl array
  asm volatile("" : "+v"(so));
  static_assert(C::kOffQ % (2 * C::kQTile) == 0 && C::kQTile >= C::kQW * 2 * C::kRowBytes,
                "Q / dO lane offsets below kQTile: xor with kQTile switches buffers");
  static_assert(C::kOffL % (4 * C::kBQ * 4) == 0 && 4 * (C::kQW + 4) <= C::kBQ * 4,
                "nl / D lane offsets below kBQ floats: xor with kBQ * 4 switches buffers");

  const bool key_ok = 32 * kb + n < nvalid;

  f32x16 dvt[C::kCT], dkt[C::kCT];
#pragma unroll
  for (int c = 0; c < C::kCT; ++c) {
    dvt[c] = f32x16{};
    dkt[c] = f32x16{};
  }

  wait_vmem_all();
  __syncthreads();
  // -V, once for the whole sweep
  for (int i = t; i < C::kKTile / 16; i += C::kThreads) {
    u32x4* x = reinterpret_cast<u32x4*>(lds + C::kOffV) + i;
    *x ^= (u32x4)0x80008000u;
  }
  __syncthreads();

  const int ntiles = grp * nqt;
  int q0 = 0;         // first row of the current tile within its head
  int qn = 0;         // first row of the next tile
  int64_t hn = 0;     // the offset (in rows) of the next tile's head
  for (int it = 0; it < ntiles; ++it) {
    const int cur = it & 1;
    // next query tile in flight: Q, dO rows and their nl, D straight into LDS
    qn = q0 + C::kBQ;
    if (qn >= nq) {
      qn = 0;
      hn += Nq;
    }
    if (it + 1 < ntiles) {
      const int64_t row = hn + qn;
      issue_rows<D>(qb + row * D, lbase + C::kOffQ + (cur ^ 1) * C::kQTile, nq - 1 - qn,
                    C::kQTile / 1024 / C::kWaves, wave, lane, C::kWaves);
      issue_rows<D>(ob + row * D, lbase + C::kOffO + (cur ^ 1) * C::kQTile, nq - 1 - qn,
                    C::kQTile / 1024 / C::kWaves, wave, lane, C::kWaves);
      issue_rowvals<C::kBQ>(nlb + row, deltab + row, lbase + C::kOffL + (cur ^ 1) * C::kBQ * 4,
                            lbase + C::kOffD + (cur ^ 1) * C::kBQ * 4, nq - 1 - qn, wave, lane);
    }
    // last query tile (rows past Nq are clamped copies) or a partial key tile
    const bool masked = q0 + C::kBQ > nq || nvalid < C::kBK;
    // qo, tqo and so point into buffer `cur` (toggled at the end of every tile)
    const char* qt = lds + C::kOffQ;
    const char* ot = lds + C::kOffO;
    const char* kt = lds;                        // kvo[s] holds the K tile's base
    const char* vt = lds + (C::kOffV - C::kOffK);
    const char* cl = lds + so;                   // so holds the nl array's base
    const char* cd = lds + so + (C::kOffD - C::kOffL);

    // S = Q K^T and D - dP = D + dO (-V)^T for this wave's 32 keys and kQW queries; the dP
    // accumulators start from D in accumulator order (element 4 rq + x is query 8 rq + 4 g + x)
    f32x16 sacc[C::kQB], pacc[C::kQB];
#pragma unroll
    for (int b = 0; b < C::kQB; ++b) {
      sacc[b] = f32x16{};
      const float* db = reinterpret_cast<const float*>(cd) + 32 * b;
      const f32x4 d0 = *reinterpret_cast<const f32x4*>(db);
      const f32x4 d1 = *reinterpret_cast<const f32x4*>(db + 8);
      const f32x4 d2 = *reinterpret_cast<const f32x4*>(db + 16);
      const f32x4 d3 = *reinterpret_cast<const f32x4*>(db + 24);
      pacc[b] = __builtin_shufflevector(__builtin_shufflevector(d0, d1, 0, 1, 2, 3, 4, 5, 6, 7),
                                        __builtin_shufflevector(d2, d3, 0, 1, 2, 3, 4, 5, 6, 7),
                                        0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
    }
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s) {
      const bf16x8 bk = *reinterpret_cast<const bf16x8*>(kt + kvo[s]);
      const bf16x8 bv = *reinterpret_cast<const bf16x8*>(vt + kvo[s]);
#pragma unroll
      for (int b = 0; b < C::kQB; ++b) {
        const int rowb = 32 * b * C::kRowBytes;
        const bf16x8 aq = *reinterpret_cast<const bf16x8*>(qt + rowb + qo[s]);
        const bf16x8 ao = *reinterpret_cast<const bf16x8*>(ot + rowb + qo[s]);
        sacc[b] = mfma32(aq, bk, sacc[b]);
        pacc[b] = mfma32(ao, bv, pacc[b]);
      }
    }
    // P and dS (fp32) -> bf16 B operands.  Accumulator r of block b is query
    // 32b + 8(r/4) + 4g + r%4; the 8 queries of k-step 2b+h are accumulators 8h .. 8h+7.
    // the vector work goes ahead of the other wave's matrix products on the SIMD
    __builtin_amdgcn_s_setprio(1);
    bf16x8 pf[2 * C::kQB], sf[2 * C::kQB];
#pragma unroll
    for (int b = 0; b < C::kQB; ++b) {
      float p[16], dsv[16];
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        // nl of 4 consecutive queries qh kQW + 32 b + 8 rq + 4 g ..
        const f32x4 nl4 = *reinterpret_cast<const f32x4*>(cl + 4 * (32 * b + 8 * rq));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float pe = fast_exp2(__builtin_fmaf(sacc[b][4 * rq + e], c2, nl4[e]));
          p[4 * rq + e] = pe;
          dsv[4 * rq + e] = pe * pacc[b][4 * rq + e];   // -dS
        }
      }
      if (masked) {
        // keys past the chunk end (one lane each) and queries past Nq (clamped copies) add nothing
        cold_path();
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int qi = qh * C::kQW + 32 * b + 8 * (rr >> 2) + 4 * g + (rr & 3);
          if (!key_ok || q0 + qi >= nq) {
            p[rr] = 0.f;
            dsv[rr] = 0.f;
          }
        }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        u32x4 wp, ws;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          wp[e] = pack_bf16x2(p[8 * h + 2 * e], p[8 * h + 2 * e + 1]);
          ws[e] = pack_bf16x2(dsv[8 * h + 2 * e], dsv[8 * h + 2 * e + 1]);
        }
        pf[2 * b + h] = __builtin_bit_cast(bf16x8, wp);
        sf[2 * b + h] = __builtin_bit_cast(bf16x8, ws);
      }
    }
    __builtin_amdgcn_s_setprio(0);
    // dV^T += dO^T P, dK^T += Q^T dS
#pragma unroll
    for (int ks = 0; ks < 2 * C::kQB; ++ks) {
      const int rowb = 16 * ks * C::kRowBytes;
#pragma unroll
      for (int c = 0; c < C::kCT; ++c) {
        const bf16x4 o0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(ot + rowb + tqo[0][c]));
        const bf16x4 o1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(ot + rowb + tqo[1][c]));
        const bf16x4 q0v = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(qt + rowb + tqo[0][c]));
        const bf16x4 q1v = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(qt + rowb + tqo[1][c]));
        dvt[c] = mfma32(__builtin_shufflevector(o0, o1, 0, 1, 2, 3, 4, 5, 6, 7), pf[ks], dvt[c]);
        dkt[c] = mfma32(__builtin_shufflevector(q0v, q1v, 0, 1, 2, 3, 4, 5, 6, 7), sf[ks], dkt[c]);
      }
    }
    // transposed Q / dO reads run ahead of the matrix products that consume them
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int i = 0; i < 4 * C::kQB * C::kCT; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    // next tile landed (the only vector memory operations in flight); this tile's reads done
    wait_vmem_all();
    __syncthreads();
    q0 = qn;
    // the read offsets move to the other buffer: its Q/dO tiles lie kQTile further (or back),
    // its nl / D kBQ floats; the lane parts of the offsets stay below either step, so an exclusive
    // or with the step switches buffers
#pragma unroll
    for (int s2 = 0; s2 < C::kDSteps; ++s2) qo[s2] ^= C::kQTile;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int ct = 0; ct < C::kCT; ++ct) tqo[h][ct] ^= C::kQTile;
    so ^= C::kBQ * 4;
  }

  // the two query halves of a key block add their dK^T / dV^T through LDS
  float* xch = reinterpret_cast<float*>(lds + C::kOffQ);
  const int64_t key = k0 + 32 * kb + n;
  float* dkr = dk + (bh * Nk + key) * D;
  float* dvr = dv + (bh * Nk + key) * D;
#pragma unroll
  for (int which = 0; which < 2; ++which) {
    f32x16* acc = which == 0 ? dkt : dvt;
    if (qh == 1) {
#pragma unroll
      for (int c = 0; c < C::kCT; ++c)
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) xch[((kb * C::kCT + c) * 16 + rr) * 64 + lane] = acc[c][rr];
    }
    __syncthreads();
    if (qh == 0) {
#pragma unroll
      for (int c = 0; c < C::kCT; ++c)
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) acc[c][rr] += xch[((kb * C::kCT + c) * 16 + rr) * 64 + lane];
      if (key_ok) {
        float* dst = which == 0 ? dkr : dvr;
        const float f = which == 0 ? -scale : 1.0f;   // the dK^T accumulators hold sums of -dS
#pragma unroll
        for (int c = 0; c < C::kCT; ++c)
#pragma unroll
          for (int rq = 0; rq < 4; ++rq) {
            const int col = c * 32 + 8 * rq + 4 * g;
            f32x4 val = {acc[c][4 * rq] * f, acc[c][4 * rq + 1] * f, acc[c][4 * rq + 2] * f,
                         acc[c][4 * rq + 3] * f};
            if (accumulate) val += *reinterpret_cast<const f32x4*>(dst + col);
            *reinterpret_cast<f32x4*>(dst + col) = val;
          }
      }
    }
    __syncthreads();
  }
}

template <int D>
hipError_t launch(const BwdArgs& a) {
  using C = DkvCfg<D>;
  const int64_t max_chunk = (a.Nk + a.R - 1) / a.R;
  const int64_t tpc = (max_chunk + C::kBK - 1) / C::kBK;
  const int64_t nwg = a.BH / a.G * a.R * tpc;
  hipLaunchKernelGGL((bwd_dkdv_kernel<D>), dim3((uint32_t)nwg), dim3(C::kThreads), 0, a.stream,
                     (const __bf16*)a.q, (const __bf16*)a.k, (const __bf16*)a.v,
                     (const __bf16*)a.dout, a.nl, a.delta, a.dk, a.dv, (int)(a.BH / a.G),
                     (int)a.H, (int)a.G, a.Nq, a.Nk,
                     (int)a.R, (int)tpc, a.scale * kLog2e, a.scale, a.accumulate_dkv ? 1 : 0);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd_dkdv_bf16_d64(const BwdArgs& a) { return launch<64>(a); }

}  // namespace ringx
