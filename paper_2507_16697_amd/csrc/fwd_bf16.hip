// Ring-chunked attention forward, bf16 storage, bf16 MFMA with fp32 accumulation (gfx950).
//
// One workgroup = 4 waves = one (b, h) and a tile of 128 queries (32 per wave).  The key/value
// sequence is visited as R chunks (ring steps, arXiv 2507.16697 Sec. III-A); every chunk is
// streamed through LDS in tiles of BK keys, double buffered (the on-chip analogue of the paper's
// ping-pong buffers) and filled by direct global->LDS loads issued one tile ahead.  Within a chunk
// each wave keeps an online softmax (Eqs. (2)-(4)); at the end of the chunk it forms the chunk's
// local result (loc_out, loc_lse) and folds it into the running Eq. (5) merge held in registers.
// PARTIALS = true writes the local results instead of merging them.
//
// Per wave, with g = lane / 32 and n = lane % 32:
//   S^T = K Q^T   A = K rows from LDS (key n, 8 dims), B = Q^T from registers (query n, 8 dims)
//                 -> lane holds query n and keys 8*(r/4) + 4g + r%4 of each 32-key block;
//   O^T += V^T P^T A = V^T read from the row-major V tile with ds_read_b64_tr_b16 (4 keys per
//                 read), B = P^T straight from the S^T registers (keys 4g..4g+3, 8+4g..8+4g+3).
// LDS tiles are row-major with the 16-byte chunks of each row XOR-swizzled by the row index, so
// that both the 16-byte K reads (16 rows, one chunk) and the transposed V reads (4 rows x 2
// chunks per 16 lanes) hit distinct banks.
// Softmax statistics are fp32 in the exp2 domain (t = scale*log2(e)*q.k).  The reference maximum
// of a row only moves when a tile's maximum exceeds it by more than kLazy (probabilities stay
// below 2^kLazy), so the accumulator rescale is skipped for most tiles.

#include "ringx_device.h"
#include "ringx_kernels.h"

namespace ringx {
namespace {

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr float kLazy = 8.0f;

template <int D>
struct FwdCfg {
  static constexpr int kThreads = 256;
  static constexpr int kWaves = 4;
  static constexpr int kQW = 32;                  // queries per wave
  static constexpr int kBQ = kWaves * kQW;        // queries per workgroup
  static constexpr int kBK = 8192 / D;            // keys per tile: 64 (d=128) or 128 (d=64)
  static constexpr int kRowBytes = D * 2;
  static constexpr int kChunks = D / 8;           // 16-byte chunks per row
  static constexpr int kTileBytes = kBK * kRowBytes;   // 16 KiB
  static constexpr int kKTiles = kBK / 32;        // 32-key blocks per tile
  static constexpr int kDSteps = D / 16;          // MFMA k-steps over the head dim
  static constexpr int kKSteps = kBK / 16;        // MFMA k-steps over the keys
  static constexpr int kCT = D / 32;              // 32-dim blocks of the output
  static constexpr int kLoads = kTileBytes / (kThreads * 16);   // 16-byte loads per thread
};

// Swizzled 16-byte chunk of (row, logical chunk c) inside a row-major tile.
template <int D>
__device__ __forceinline__ int swz(int row) {
  if constexpr (D == 128) return ((row & 3) << 2) | ((row >> 2) & 3);
  else return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
}
template <int D>
__device__ __forceinline__ int tile_off(int row, int c) {   // byte offset
  return row * (D * 2) + ((c ^ swz<D>(row)) << 4);
}


// Per-lane byte offsets (from the tile's first row) of this lane's direct loads: 16-byte slot
// `slot` of the swizzled tile holds logical chunk (slot % chunks) ^ swz(row) of row slot / chunks.
template <int D>
__device__ __forceinline__ void load_offsets(int (&goff)[FwdCfg<D>::kLoads],
                                             int (&grow)[FwdCfg<D>::kLoads], int wave, int lane) {
  using C = FwdCfg<D>;
#pragma unroll
  for (int u = 0; u < C::kLoads; ++u) {
    const int slot = (u * C::kWaves + wave) * 64 + lane;
    const int row = slot / C::kChunks;
    const int c = (slot % C::kChunks) ^ swz<D>(row);
    grow[u] = row;
    goff[u] = row * C::kRowBytes + c * 16;
  }
}

// Issue the direct loads of one K/V tile starting at key `start`; rows at or past `hi` (only in
// the last tile of a chunk) are clamped to hi - 1.
template <int D>
__device__ __forceinline__ void issue_tile(const char* __restrict__ kb,
                                           const char* __restrict__ vb, uint32_t kdst,
                                           uint32_t vdst, int64_t start, int64_t hi,
                                           const int (&goff)[FwdCfg<D>::kLoads],
                                           const int (&grow)[FwdCfg<D>::kLoads], int wave) {
  using C = FwdCfg<D>;
  const char* kt = kb + start * C::kRowBytes;
  const char* vt = vb + start * C::kRowBytes;
  if (start + C::kBK <= hi) {
#pragma unroll
    for (int u = 0; u < C::kLoads; ++u) {
      const uint32_t wbase =
          (uint32_t)__builtin_amdgcn_readfirstlane((u * C::kWaves + wave) * 1024);
      load_lds16(kt + goff[u], kdst + wbase);
      load_lds16(vt + goff[u], vdst + wbase);
    }
  } else {
    cold_path();
    const int last = (int)(hi - 1 - start);
#pragma unroll
    for (int u = 0; u < C::kLoads; ++u) {
      const int off = grow[u] <= last ? goff[u] : goff[u] - (grow[u] - last) * C::kRowBytes;
      const uint32_t wbase =
          (uint32_t)__builtin_amdgcn_readfirstlane((u * C::kWaves + wave) * 1024);
      load_lds16(kt + off, kdst + wbase);
      load_lds16(vt + off, vdst + wbase);
    }
  }
}

template <int D, bool PARTIALS>
__global__ __launch_bounds__(256, 2) void fwd_bf16_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    __bf16* __restrict__ out, float* __restrict__ lse, float* __restrict__ part_out,
    float* __restrict__ part_lse, int BH, int64_t Nq, int64_t Nk, int R, float c2) {
  using C = FwdCfg<D>;
  __shared__ __attribute__((aligned(1024))) char lds_k[2 * C::kTileBytes];
  __shared__ __attribute__((aligned(1024))) char lds_v[2 * C::kTileBytes];

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = t >> 6;
  const int n = lane & 31;
  const int g = lane >> 5;

  const int64_t nqt = (Nq + C::kBQ - 1) / C::kBQ;
  const uint32_t wg = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t bh = wg / nqt;
  const int64_t q0 = (wg % nqt) * C::kBQ + wave * C::kQW;
  if (bh >= BH) return;

  const __bf16* qb = q + bh * Nq * D;
  const char* kb = reinterpret_cast<const char*>(k + bh * Nk * D);
  const char* vb = reinterpret_cast<const char*>(v + bh * Nk * D);
  int goff[C::kLoads], grow[C::kLoads];
  load_offsets<D>(goff, grow, wave, lane);

  // chunk bookkeeping without divisions: chunk r has q_sz + (1 if the running remainder wraps)
  const int64_t q_sz = Nk / R;
  const int64_t rem = Nk % R;
  int64_t racc = 0;   // (r * rem) mod R
  int r = 0;
  int64_t start = 0;
  int64_t hi;
  {
    racc += rem;
    const int64_t extra = racc >= R ? 1 : 0;
    racc -= extra * R;
    hi = q_sz + extra;
  }

  // LDS byte addresses of the two K and two V buffers
  const uint32_t lk = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_k;
  const uint32_t lv = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_v;

  // first tile in flight while Q is loaded
  issue_tile<D>(kb, vb, lk, lv, start, hi, goff, grow, wave);

  // Q fragments (B operand of S^T = K Q^T): query n of this wave, dims 16*ks + 8g .. +8.
  bf16x8 qf[C::kDSteps];
  {
    int64_t qi = q0 + n;
    qi = qi < Nq ? qi : Nq - 1;
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s)
      qf[s] = *reinterpret_cast<const bf16x8*>(qb + qi * D + s * 16 + g * 8);
  }

  // per-lane LDS byte offsets (tile-relative)
  int koff[C::kDSteps];   // K fragment of 32-key block 0 at k-step s (block kt adds kt*32 rows)
#pragma unroll
  for (int s = 0; s < C::kDSteps; ++s) koff[s] = tile_off<D>(n, 2 * s + g);
  // V^T fragments via transposed reads: for 16-lane group G, rows j0 + (lane%16)/4 with
  // j0 = 16*ks + 4g (+8 for the second half), columns 32*ct + 16*(G%2) + 4*(lane%4).
  int voff[2][C::kCT];
  {
    const int G = lane >> 4;
    const int rr = (lane & 15) >> 2;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int ct = 0; ct < C::kCT; ++ct) {
        const int row = 4 * g + 8 * h + rr;
        const int col = 32 * ct + 16 * (G & 1) + 4 * (lane & 3);
        voff[h][ct] = tile_off<D>(row, col >> 3) + (col & 7) * 2;
      }
  }

  f32x16 oacc[C::kCT];
  f32x16 om[C::kCT];
#pragma unroll
  for (int c = 0; c < C::kCT; ++c) {
    oacc[c] = f32x16{};
    om[c] = f32x16{};
  }
  float m2 = -INFINITY;     // reference max of the row within the chunk (exp2 domain)
  float l = 0.f;            // this lane's share of the running sum within the chunk
  float lse2m = -INFINITY;  // merged log2-sum-exp over finished chunks

  int cur = 0;
  wait_vmem_all();
  __syncthreads();

  while (true) {
    // next tile: the following BK keys of this chunk, or the first tile of the next chunk
    int64_t nstart = start + C::kBK;
    int64_t nhi = hi;
    bool has_next = true;
    if (nstart >= hi) {
      if (r + 1 < R) {
        nstart = hi;
        racc += rem;
        const int64_t extra = racc >= R ? 1 : 0;
        racc -= extra * R;
        nhi = hi + q_sz + extra;
      } else {
        has_next = false;
      }
    }
    if (has_next)
      issue_tile<D>(kb, vb, lk + (cur ^ 1) * C::kTileBytes, lv + (cur ^ 1) * C::kTileBytes,
                    nstart, nhi, goff, grow, wave);

    const char* kbuf = lds_k + cur * C::kTileBytes;
    const char* vbuf = lds_v + cur * C::kTileBytes;
    const int nvalid = (int)min<int64_t>(C::kBK, hi - start);

    // S^T = K Q^T for the tile's 32-key blocks
    f32x16 sacc[C::kKTiles];
#pragma unroll
    for (int kt = 0; kt < C::kKTiles; ++kt) sacc[kt] = f32x16{};
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s) {
#pragma unroll
      for (int kt = 0; kt < C::kKTiles; ++kt) {
        const bf16x8 a =
            *reinterpret_cast<const bf16x8*>(kbuf + koff[s] + kt * 32 * C::kRowBytes);
        sacc[kt] = mfma32(a, qf[s], sacc[kt]);
      }
    }
    // keep two k-steps of K fragments in flight ahead of the MFMAs
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * C::kKTiles, 0);
#pragma unroll
    for (int s = 0; s < C::kDSteps - 2; ++s) {
      __builtin_amdgcn_sched_group_barrier(0x100, C::kKTiles, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, C::kKTiles, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2 * C::kKTiles, 0);
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
    // online softmax within the chunk (Eqs. (2)-(3) with a lazily moved reference max)
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < C::kKTiles; ++kt)
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) mx = fmaxf(mx, sacc[kt][rr]);
    {
      auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false,
                                                 false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    }
    const float mt = mx * c2;
    const bool need = mt > m2 + kLazy;
    if (__builtin_amdgcn_ballot_w64(need)) {
      cold_path();
      const float mnew = need ? mt : m2;
      const float alpha = fast_exp2(m2 - mnew);
      m2 = mnew;
      l *= alpha;
#pragma unroll
      for (int c = 0; c < C::kCT; ++c) oacc[c] *= alpha;
    }
    float lsum = 0.f;
    bf16x8 pf[C::kKSteps];
#pragma unroll
    for (int kt = 0; kt < C::kKTiles; ++kt) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = fast_exp2(__builtin_fmaf(sacc[kt][8 * h + 2 * e], c2, -m2));
          const float p1 = fast_exp2(__builtin_fmaf(sacc[kt][8 * h + 2 * e + 1], c2, -m2));
          lsum += p0 + p1;
          w[e] = pack_bf16x2(p0, p1);
        }
        pf[2 * kt + h] = __builtin_bit_cast(bf16x8, w);
      }
    }
    l += lsum;

    // O^T += V^T P^T
#pragma unroll
    for (int s = 0; s < C::kKSteps; ++s) {
#pragma unroll
      for (int c = 0; c < C::kCT; ++c) {
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (lds_bf16x4*)(vbuf + voff[0][c] + s * 16 * C::kRowBytes));
        const bf16x4 hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (lds_bf16x4*)(vbuf + voff[1][c] + s * 16 * C::kRowBytes));
        const bf16x8 a = __builtin_shufflevector(lo, hi4, 0, 1, 2, 3, 4, 5, 6, 7);
        oacc[c] = mfma32(a, pf[s], oacc[c]);
      }
    }
    // transposed V reads two MFMAs ahead
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int i = 0; i < C::kKSteps * C::kCT - 2; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);

    if (start + C::kBK >= hi) {
      // end of chunk r: local result (loc_out_r, loc_lse_r), then the Eq. (5) merge
      float lrow;
      {
        auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l), __float_as_uint(l), false,
                                                   false);
        lrow = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
      }
      const float inv = 1.0f / lrow;
      const float lse2r = m2 + fast_log2(lrow);
      const int64_t qi = q0 + n;
      if constexpr (PARTIALS) {
        if (qi < Nq) {
          const int64_t row = ((int64_t)r * BH + bh) * Nq + qi;
          float* po = part_out + row * D;
#pragma unroll
          for (int c = 0; c < C::kCT; ++c)
#pragma unroll
            for (int rq = 0; rq < 4; ++rq) {
              f32x4 val = {oacc[c][4 * rq] * inv, oacc[c][4 * rq + 1] * inv,
                           oacc[c][4 * rq + 2] * inv, oacc[c][4 * rq + 3] * inv};
              *reinterpret_cast<f32x4*>(po + c * 32 + 8 * rq + 4 * g) = val;
            }
          if (g == 0) part_lse[row] = lse2r * kLn2;
        }
      } else {
        const float M = fmaxf(lse2m, lse2r);
        const float a = fast_exp2(lse2m - M);
        const float b = fast_exp2(lse2r - M);
        const float den = a + b;
        const float wa = a / den;
        const float wb = b * inv / den;
#pragma unroll
        for (int c = 0; c < C::kCT; ++c) om[c] = om[c] * wa + oacc[c] * wb;
        lse2m = M + fast_log2(den);
      }
#pragma unroll
      for (int c = 0; c < C::kCT; ++c) oacc[c] = f32x16{};
      l = 0.f;
      m2 = -INFINITY;
      ++r;
    }

    if (!has_next) break;
    wait_vmem_all();
    __syncthreads();
    cur ^= 1;
    start = nstart;
    hi = nhi;
  }

  if constexpr (!PARTIALS) {
    const int64_t qi = q0 + n;
    if (qi < Nq) {
      __bf16* ob = out + (bh * Nq + qi) * D;
#pragma unroll
      for (int c = 0; c < C::kCT; ++c)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          u32x2 w;
          w[0] = pack_bf16x2(om[c][4 * rq], om[c][4 * rq + 1]);
          w[1] = pack_bf16x2(om[c][4 * rq + 2], om[c][4 * rq + 3]);
          *reinterpret_cast<u32x2*>(ob + c * 32 + 8 * rq + 4 * g) = w;
        }
      if (g == 0) lse[bh * Nq + qi] = lse2m * kLn2;
    }
  }
}

template <int D, bool PARTIALS>
hipError_t launch(const FwdArgs& a) {
  using C = FwdCfg<D>;
  const int64_t nqt = (a.Nq + C::kBQ - 1) / C::kBQ;
  const int64_t nwg = nqt * a.BH;
  hipLaunchKernelGGL((fwd_bf16_kernel<D, PARTIALS>), dim3((uint32_t)nwg), dim3(C::kThreads), 0,
                     a.stream, (const __bf16*)a.q, (const __bf16*)a.k, (const __bf16*)a.v,
                     (__bf16*)a.out, a.lse, a.part_out, a.part_lse, (int)a.BH, a.Nq, a.Nk,
                     (int)a.R, a.scale * kLog2e);
  return hipGetLastError();
}

}  // namespace

int64_t fwd_bf16_workgroups(int64_t BH, int64_t Nq, int64_t d) {
  const int64_t bq = 128;
  (void)d;
  return BH * ((Nq + bq - 1) / bq);
}

hipError_t launch_fwd_bf16(const FwdArgs& a, bool partials) {
  if (a.d == 128) return partials ? launch<128, true>(a) : launch<128, false>(a);
  return partials ? launch<64, true>(a) : launch<64, false>(a);
}

}  // namespace ringx
