// Ring-chunked attention forward, bf16 storage, bf16 MFMA with fp32 accumulation (gfx950).
//
// One workgroup = 4 waves = one (b, h) and a tile of 128 queries (32 per wave).  The key/value
// sequence is visited as R chunks (ring steps, arXiv 2507.16697 Sec. III-A); every chunk is
// streamed through LDS in tiles of BK keys, double buffered (the on-chip analogue of the paper's
// ping-pong buffers).  Within a chunk the wave keeps an online softmax (Eqs. (2)-(4)); at the
// end of the chunk it forms the chunk's local result (loc_out, loc_lse) and folds it into the
// running Eq. (5) merge held in registers.  PARTIALS = true writes the local results instead.
//
// Per wave, with g = lane / 32 and n = lane % 32:
//   S^T = K Q^T   A = K rows from LDS (key n, 8 dims), B = Q^T from registers (query n, 8 dims)
//                 -> lane holds query n and keys 8*(r/4) + 4g + r%4 of each 32-key block;
//   O^T += V^T P^T A = V^T from LDS (dim n, 8 keys), B = P^T straight from the S^T registers.
// The 8 keys a lane feeds to one PV MFMA are {4g..4g+3, 8+4g..8+4g+3} of a 16-key block, so the
// transposed V tile is written to LDS with the two middle 4-key groups of each 16-key block
// swapped (position = key offset with bits 2 and 3 exchanged): each A read is one 16-byte load.
// Softmax statistics stay in fp32 in the exp2 domain (t = scale * log2(e) * q.k).

#include "ringx_device.h"
#include "ringx_kernels.h"

namespace ringx {
namespace {

template <int D>
struct FwdCfg {
  static constexpr int kThreads = 256;
  static constexpr int kWaves = 4;
  static constexpr int kQW = 32;                  // queries per wave
  static constexpr int kBQ = kWaves * kQW;        // queries per workgroup
  static constexpr int kBK = 8192 / D;            // keys per tile: 64 (d=128) or 128 (d=64)
  static constexpr int kKS = D + 8;               // padded LDS row stride of the K tile (elements)
  static constexpr int kVS = kBK + 8;             // padded LDS row stride of the V^T tile
  static constexpr int kOcts = D / 8;             // 16-byte chunks per row
  static constexpr int kKTiles = kBK / 32;        // 32-key blocks per tile
  static constexpr int kDSteps = D / 16;          // MFMA k-steps over the head dim
  static constexpr int kKSteps = kBK / 16;        // MFMA k-steps over the keys
  static constexpr int kCT = D / 32;              // 32-dim blocks of the output
  static constexpr int kLdsK = kBK * kKS;         // elements per K buffer
  static constexpr int kLdsV = D * kVS;           // elements per V^T buffer
  static_assert(kBK * D == kThreads * 32, "each thread stages 32 elements of K and of V");
};

// Position of key offset o (0..kBK-1) inside the transposed V tile.
__device__ __forceinline__ int vt_pos(int o) {
  const int q4 = (o >> 2) & 3;
  const int q4s = ((q4 & 1) << 1) | (q4 >> 1);
  return (o & ~15) | (q4s << 2) | (o & 3);
}

template <int D>
struct Stage {
  u32x4 k[4];
  u32x4 v[4];
};

template <int D>
__device__ __forceinline__ void load_tile(Stage<D>& st, const __bf16* __restrict__ kb,
                                          const __bf16* __restrict__ vb, int64_t start,
                                          int64_t hi, int t) {
  using C = FwdCfg<D>;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int ci = t + C::kThreads * u;
    const int row = ci / C::kOcts;
    const int cc = ci % C::kOcts;
    int64_t key = start + row;
    key = key < hi ? key : hi - 1;
    st.k[u] = *reinterpret_cast<const u32x4*>(kb + key * D + cc * 8);
  }
  const int co = t % C::kOcts;
  const int kq = t / C::kOcts;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    int64_t key = start + kq * 4 + e;
    key = key < hi ? key : hi - 1;
    st.v[e] = *reinterpret_cast<const u32x4*>(vb + key * D + co * 8);
  }
}

template <int D>
__device__ __forceinline__ void store_tile(const Stage<D>& st, __bf16* ks_buf, __bf16* vt_buf,
                                           int nvalid, int t) {
  using C = FwdCfg<D>;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int ci = t + C::kThreads * u;
    const int row = ci / C::kOcts;
    const int cc = ci % C::kOcts;
    *reinterpret_cast<u32x4*>(ks_buf + row * C::kKS + cc * 8) = st.k[u];
  }
  const int co = t % C::kOcts;
  const int kq = t / C::kOcts;
  // keys beyond the chunk end get V = 0 (their probabilities are 0 as well)
  uint32_t keep[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) keep[e] = (kq * 4 + e < nvalid) ? 0xffffffffu : 0u;
  const int pos = vt_pos(kq * 4);
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    const int w = m >> 1;
    uint32_t x0, x1, x2, x3;
    if (m & 1) {
      x0 = st.v[0][w] >> 16; x1 = st.v[1][w] >> 16; x2 = st.v[2][w] >> 16; x3 = st.v[3][w] >> 16;
    } else {
      x0 = st.v[0][w] & 0xffffu; x1 = st.v[1][w] & 0xffffu;
      x2 = st.v[2][w] & 0xffffu; x3 = st.v[3][w] & 0xffffu;
    }
    u32x2 out;
    out[0] = (x0 & keep[0]) | ((x1 & keep[1]) << 16);
    out[1] = (x2 & keep[2]) | ((x3 & keep[3]) << 16);
    *reinterpret_cast<u32x2*>(vt_buf + (co * 8 + m) * C::kVS + pos) = out;
  }
}

template <int D, bool PARTIALS>
__global__ __launch_bounds__(256, 2) void fwd_bf16_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    __bf16* __restrict__ out, float* __restrict__ lse, float* __restrict__ part_out,
    float* __restrict__ part_lse, int BH, int64_t Nq, int64_t Nk, int R, float c2) {
  using C = FwdCfg<D>;
  __shared__ __attribute__((aligned(16))) __bf16 lds_k[2 * C::kLdsK];
  __shared__ __attribute__((aligned(16))) __bf16 lds_v[2 * C::kLdsV];

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
  const __bf16* kb = k + bh * Nk * D;
  const __bf16* vb = v + bh * Nk * D;

  // Q fragments (B operand of S^T = K Q^T): query n of this wave, dims 16*ks + 8g .. +8.
  bf16x8 qf[C::kDSteps];
  {
    int64_t qi = q0 + n;
    qi = qi < Nq ? qi : Nq - 1;
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s)
      qf[s] = *reinterpret_cast<const bf16x8*>(qb + qi * D + s * 16 + g * 8);
  }

  f32x16 oacc[C::kCT];
  f32x16 om[C::kCT];
#pragma unroll
  for (int c = 0; c < C::kCT; ++c) {
    oacc[c] = f32x16{};
    om[c] = f32x16{};
  }
  float m2 = -INFINITY;   // running max of t within the chunk (exp2 domain)
  float l = 0.f;          // this lane's share of the running sum within the chunk
  float lse2m = -INFINITY;  // merged log2-sum-exp over finished chunks

  int r = 0;
  int64_t hi = Nk / R;            // chunk 0 = [0, floor(Nk/R))
  int64_t start = 0;
  Stage<D> st;
  load_tile<D>(st, kb, vb, start, hi, t);
  int cur = 0;
  store_tile<D>(st, lds_k, lds_v, (int)min<int64_t>(C::kBK, hi - start), t);
  __syncthreads();

  while (true) {
    // next tile: the following BK keys of this chunk, or the first tile of the next chunk
    int64_t nstart = start + C::kBK;
    int nr = r;
    int64_t nhi = hi;
    bool has_next = true;
    if (nstart >= hi) {
      nr = r + 1;
      if (nr < R) {
        nstart = (int64_t)nr * Nk / R;
        nhi = (int64_t)(nr + 1) * Nk / R;
      } else {
        has_next = false;
      }
    }
    if (has_next) load_tile<D>(st, kb, vb, nstart, nhi, t);

    const __bf16* ks_buf = lds_k + cur * C::kLdsK;
    const __bf16* vt_buf = lds_v + cur * C::kLdsV;
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
            *reinterpret_cast<const bf16x8*>(ks_buf + (kt * 32 + n) * C::kKS + s * 16 + g * 8);
        sacc[kt] = mfma32(a, qf[s], sacc[kt]);
      }
    }
    if (nvalid < C::kBK) {
#pragma unroll
      for (int kt = 0; kt < C::kKTiles; ++kt)
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int key = kt * 32 + 8 * (rr >> 2) + 4 * g + (rr & 3);
          if (key >= nvalid) sacc[kt][rr] = -INFINITY;
        }
    }
    // online softmax within the chunk (Eqs. (2)-(3) with a running max)
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
    const float mnew = fmaxf(m2, mx * c2);
    const float alpha = fast_exp2(m2 - mnew);
    m2 = mnew;
    float lsum = 0.f;
    bf16x8 pf[C::kKSteps];
#pragma unroll
    for (int kt = 0; kt < C::kKTiles; ++kt) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = fast_exp2(__builtin_fmaf(sacc[kt][8 * h + 2 * e], c2, -mnew));
          const float p1 = fast_exp2(__builtin_fmaf(sacc[kt][8 * h + 2 * e + 1], c2, -mnew));
          lsum += p0 + p1;
          w[e] = pack_bf16x2(p0, p1);
        }
        pf[2 * kt + h] = __builtin_bit_cast(bf16x8, w);
      }
    }
    l = l * alpha + lsum;
#pragma unroll
    for (int c = 0; c < C::kCT; ++c) oacc[c] *= alpha;

    // O^T += V^T P^T
#pragma unroll
    for (int s = 0; s < C::kKSteps; ++s) {
#pragma unroll
      for (int c = 0; c < C::kCT; ++c) {
        const bf16x8 a =
            *reinterpret_cast<const bf16x8*>(vt_buf + (c * 32 + n) * C::kVS + s * 16 + g * 8);
        oacc[c] = mfma32(a, pf[s], oacc[c]);
      }
    }

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
    }

    if (!has_next) break;
    store_tile<D>(st, lds_k + (cur ^ 1) * C::kLdsK, lds_v + (cur ^ 1) * C::kLdsV,
                  (int)min<int64_t>(C::kBK, nhi - nstart), t);
    __syncthreads();
    cur ^= 1;
    start = nstart;
    r = nr;
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
