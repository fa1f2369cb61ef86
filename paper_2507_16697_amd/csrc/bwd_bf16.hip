// Recompute backward of ring-chunked attention, bf16 MFMA with fp32 accumulation (gfx950).
//
// One workgroup = 4 waves = one (b, h) and a tile of 128 keys inside one chunk (a key tile never
// straddles a chunk boundary).  Each wave owns 32 of those keys and keeps their K and V rows in
// registers and their dK^T, dV^T accumulators in registers for the whole sweep over the query
// tiles.  With the merged log-sum-exp saved by the forward, every chunk's gradients are
// independent (arXiv 2507.16697 Sec. III-A: K/V chunk gradients per chunk, dQ accumulated over
// all steps).  Per query tile of BQ queries:
//   S   = Q K^T          A = Q rows (LDS),          B = K rows (registers)  -> lane = key
//   dP  = dO V^T         A = dO rows (LDS),         B = V rows (registers)
//   P   = exp(S*scale - lse_i),  dS = P (dP - D_i)               (fp32, exp2 domain)
//   dV^T += dO^T P       A = dO^T (LDS, transposed), B = P from registers
//   dK^T += Q^T dS       A = Q^T  (LDS, transposed), B = dS from registers
//   dQ  += dS K          dS through LDS, A = dS rows, B = K^T (LDS); fp32 atomics into dq
// The transposed Q/dO tiles use the same key/query order permutation as the forward's V^T tile,
// so the 8 queries a lane feeds to the dV/dK MFMAs are one 16-byte LDS read.

#include "ringx_device.h"
#include "ringx_kernels.h"

namespace ringx {
namespace {

template <int D>
struct BwdCfg {
  static constexpr int kThreads = 256;
  static constexpr int kWaves = 4;
  static constexpr int kBK = 128;                    // keys per workgroup (32 per wave)
  static constexpr int kBQ = 4096 / D;               // queries per tile: 32 (d=128), 64 (d=64)
  static constexpr int kQB = kBQ / 32;               // 32-query blocks per tile
  static constexpr int kDSteps = D / 16;
  static constexpr int kQSteps = kBQ / 16;
  static constexpr int kCT = D / 32;
  static constexpr int kRS = D + 8;                  // row stride of Q, dO tiles (elements)
  static constexpr int kTS = kBQ + 8;                // row stride of Q^T, dO^T tiles
  static constexpr int kKTS = kBK + 8;               // row stride of K^T and dS tiles
  static constexpr int kDq4 = D / 4;                 // 4-dim groups per row
  static_assert(kBQ * D == kThreads * 16, "each thread stages 4 queries x 4 dims");
  static_assert(kQB * kCT == kWaves, "one 32x32 dQ tile per wave");
};

__device__ __forceinline__ int perm16(int o) {
  const int q4 = (o >> 2) & 3;
  const int q4s = ((q4 & 1) << 1) | (q4 >> 1);
  return (o & ~15) | (q4s << 2) | (o & 3);
}

template <int D>
struct QStage {
  u32x2 q[4];
  u32x2 o[4];
  float lse2;
  float delta;
};

// Thread t stages query quad qq (4 rows) x dim quad dq4 (4 dims) of Q and dO.
template <int D>
__device__ __forceinline__ void load_q_tile(QStage<D>& st, const __bf16* __restrict__ qb,
                                            const __bf16* __restrict__ ob,
                                            const float* __restrict__ lseb,
                                            const float* __restrict__ deltab, int64_t q0,
                                            int64_t Nq, int t) {
  using C = BwdCfg<D>;
  const int dq4 = t % C::kDq4;
  const int qq = t / C::kDq4;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int64_t qi = q0 + qq * 4 + e;
    if (qi < Nq) {
      st.q[e] = *reinterpret_cast<const u32x2*>(qb + qi * D + dq4 * 4);
      st.o[e] = *reinterpret_cast<const u32x2*>(ob + qi * D + dq4 * 4);
    } else {
      st.q[e] = u32x2{0u, 0u};
      st.o[e] = u32x2{0u, 0u};
    }
  }
  if (t < C::kBQ) {
    const int64_t qi = q0 + t;
    st.lse2 = qi < Nq ? lseb[qi] * kLog2e : INFINITY;   // padded rows: P = exp2(-inf) = 0
    st.delta = qi < Nq ? deltab[qi] : 0.f;
  }
}

template <int D>
__device__ __forceinline__ void store_q_tile(const QStage<D>& st, __bf16* qs, __bf16* os,
                                             __bf16* qt, __bf16* ot, float* lse2s, float* ds,
                                             int t) {
  using C = BwdCfg<D>;
  const int dq4 = t % C::kDq4;
  const int qq = t / C::kDq4;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    *reinterpret_cast<u32x2*>(qs + (qq * 4 + e) * C::kRS + dq4 * 4) = st.q[e];
    *reinterpret_cast<u32x2*>(os + (qq * 4 + e) * C::kRS + dq4 * 4) = st.o[e];
  }
  const int pos = perm16(qq * 4);
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int w = m >> 1;
    const int sh = (m & 1) * 16;
    u32x2 a, b;
    a[0] = ((st.q[0][w] >> sh) & 0xffffu) | (((st.q[1][w] >> sh) & 0xffffu) << 16);
    a[1] = ((st.q[2][w] >> sh) & 0xffffu) | (((st.q[3][w] >> sh) & 0xffffu) << 16);
    b[0] = ((st.o[0][w] >> sh) & 0xffffu) | (((st.o[1][w] >> sh) & 0xffffu) << 16);
    b[1] = ((st.o[2][w] >> sh) & 0xffffu) | (((st.o[3][w] >> sh) & 0xffffu) << 16);
    *reinterpret_cast<u32x2*>(qt + (dq4 * 4 + m) * C::kTS + pos) = a;
    *reinterpret_cast<u32x2*>(ot + (dq4 * 4 + m) * C::kTS + pos) = b;
  }
  if (t < C::kBQ) {
    lse2s[t] = st.lse2;
    ds[t] = st.delta;
  }
}

template <int D>
__global__ __launch_bounds__(256) void bwd_bf16_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    const __bf16* __restrict__ dout, const float* __restrict__ lse,
    const float* __restrict__ delta, float* __restrict__ dq, float* __restrict__ dk,
    float* __restrict__ dv, int BH, int64_t Nq, int64_t Nk, int R, int tiles_per_chunk,
    float c2, float scale, int accumulate) {
  using C = BwdCfg<D>;
  __shared__ __attribute__((aligned(16))) __bf16 kt_s[D * C::kKTS];       // K^T of the key tile
  __shared__ __attribute__((aligned(16))) __bf16 q_s[C::kBQ * C::kRS];
  __shared__ __attribute__((aligned(16))) __bf16 o_s[C::kBQ * C::kRS];
  __shared__ __attribute__((aligned(16))) __bf16 qt_s[D * C::kTS];
  __shared__ __attribute__((aligned(16))) __bf16 ot_s[D * C::kTS];
  __shared__ __attribute__((aligned(16))) __bf16 ds_s[C::kBQ * C::kKTS];  // dS [query][key]
  __shared__ __attribute__((aligned(16))) float lse2_s[C::kBQ];
  __shared__ __attribute__((aligned(16))) float d_s[C::kBQ];

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = t >> 6;
  const int n = lane & 31;
  const int g = lane >> 5;

  const uint32_t wg = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t per_bh = (int64_t)R * tiles_per_chunk;
  const int64_t bh = wg / per_bh;
  const int r = (int)((wg % per_bh) / tiles_per_chunk);
  const int tile = (int)(wg % tiles_per_chunk);
  if (bh >= BH) return;
  const int64_t lo = (int64_t)r * Nk / R;
  const int64_t hi = (int64_t)(r + 1) * Nk / R;
  const int64_t k0 = lo + (int64_t)tile * C::kBK;
  if (k0 >= hi) return;                         // uniform over the workgroup
  const int nvalid = (int)min<int64_t>(C::kBK, hi - k0);

  const __bf16* qb = q + bh * Nq * D;
  const __bf16* ob = dout + bh * Nq * D;
  const __bf16* kb = k + bh * Nk * D;
  const __bf16* vb = v + bh * Nk * D;
  const float* lseb = lse + bh * Nq;
  const float* deltab = delta + bh * Nq;
  float* dqb = dq + bh * Nq * D;

  // this lane's key: column of S, dP and of the dK^T/dV^T accumulators
  const int jl = wave * 32 + n;
  const bool key_ok = jl < nvalid;
  bf16x8 kf[C::kDSteps], vf[C::kDSteps];
  {
    const int64_t key = k0 + (key_ok ? jl : 0);
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s) {
      kf[s] = *reinterpret_cast<const bf16x8*>(kb + key * D + s * 16 + g * 8);
      vf[s] = *reinterpret_cast<const bf16x8*>(vb + key * D + s * 16 + g * 8);
    }
  }
  // K^T tile (dims x keys, natural key order), zero for keys past the chunk end
  for (int item = t; item < (C::kBK / 4) * C::kDq4; item += C::kThreads) {
    const int dq4 = item % C::kDq4;
    const int kq = item / C::kDq4;
    u32x2 x[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int jj = kq * 4 + e;
      x[e] = jj < nvalid ? *reinterpret_cast<const u32x2*>(kb + (k0 + jj) * D + dq4 * 4)
                         : u32x2{0u, 0u};
    }
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int w = m >> 1;
      const int sh = (m & 1) * 16;
      u32x2 a;
      a[0] = ((x[0][w] >> sh) & 0xffffu) | (((x[1][w] >> sh) & 0xffffu) << 16);
      a[1] = ((x[2][w] >> sh) & 0xffffu) | (((x[3][w] >> sh) & 0xffffu) << 16);
      *reinterpret_cast<u32x2*>(kt_s + (dq4 * 4 + m) * C::kKTS + kq * 4) = a;
    }
  }

  f32x16 dvt[C::kCT], dkt[C::kCT];
#pragma unroll
  for (int c = 0; c < C::kCT; ++c) {
    dvt[c] = f32x16{};
    dkt[c] = f32x16{};
  }

  const int64_t nqt = (Nq + C::kBQ - 1) / C::kBQ;
  QStage<D> st;
  load_q_tile<D>(st, qb, ob, lseb, deltab, 0, Nq, t);

  // this wave's dQ output tile
  const int dq_qb = wave / C::kCT;
  const int dq_ct = wave % C::kCT;

  for (int64_t it = 0; it < nqt; ++it) {
    const int64_t q0 = it * C::kBQ;
    __syncthreads();   // previous tile's LDS reads are done
    store_q_tile<D>(st, q_s, o_s, qt_s, ot_s, lse2_s, d_s, t);
    __syncthreads();
    if (it + 1 < nqt) load_q_tile<D>(st, qb, ob, lseb, deltab, q0 + C::kBQ, Nq, t);

    // S = Q K^T and dP = dO V^T  (lane = key n, rows = queries)
    f32x16 sacc[C::kQB], pacc[C::kQB];
#pragma unroll
    for (int b = 0; b < C::kQB; ++b) {
      sacc[b] = f32x16{};
      pacc[b] = f32x16{};
    }
#pragma unroll
    for (int s = 0; s < C::kDSteps; ++s) {
#pragma unroll
      for (int b = 0; b < C::kQB; ++b) {
        const bf16x8 aq = *reinterpret_cast<const bf16x8*>(q_s + (b * 32 + n) * C::kRS + s * 16 + g * 8);
        const bf16x8 ao = *reinterpret_cast<const bf16x8*>(o_s + (b * 32 + n) * C::kRS + s * 16 + g * 8);
        sacc[b] = mfma32(aq, kf[s], sacc[b]);
        pacc[b] = mfma32(ao, vf[s], pacc[b]);
      }
    }
    // P and dS (fp32), packed to bf16 B operands; dS also goes to LDS for dQ
    bf16x8 pf[C::kQSteps], sf[C::kQSteps];
#pragma unroll
    for (int b = 0; b < C::kQB; ++b) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        u32x4 wp, ws;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float p2[2], s2[2];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int rr = 8 * h + 2 * e + u;
            const int qi = b * 32 + 8 * (rr >> 2) + 4 * g + (rr & 3);
            float p = fast_exp2(__builtin_fmaf(sacc[b][rr], c2, -lse2_s[qi]));
            p = key_ok ? p : 0.f;
            p2[u] = p;
            s2[u] = p * (pacc[b][rr] - d_s[qi]);
          }
          wp[e] = pack_bf16x2(p2[0], p2[1]);
          ws[e] = pack_bf16x2(s2[0], s2[1]);
        }
        pf[2 * b + h] = __builtin_bit_cast(bf16x8, wp);
        sf[2 * b + h] = __builtin_bit_cast(bf16x8, ws);
        // dS to LDS, [query][key]
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int rr0 = 8 * h + 2 * e;
          const int qa = b * 32 + 8 * (rr0 >> 2) + 4 * g + (rr0 & 3);
          const uint32_t w = ws[e];
          *reinterpret_cast<uint16_t*>(ds_s + qa * C::kKTS + jl) = (uint16_t)(w & 0xffffu);
          *reinterpret_cast<uint16_t*>(ds_s + (qa + 1) * C::kKTS + jl) = (uint16_t)(w >> 16);
        }
      }
    }
    // dV^T += dO^T P, dK^T += Q^T dS
#pragma unroll
    for (int s = 0; s < C::kQSteps; ++s) {
#pragma unroll
      for (int c = 0; c < C::kCT; ++c) {
        const bf16x8 ao = *reinterpret_cast<const bf16x8*>(ot_s + (c * 32 + n) * C::kTS + s * 16 + g * 8);
        const bf16x8 aq = *reinterpret_cast<const bf16x8*>(qt_s + (c * 32 + n) * C::kTS + s * 16 + g * 8);
        dvt[c] = mfma32(ao, pf[s], dvt[c]);
        dkt[c] = mfma32(aq, sf[s], dkt[c]);
      }
    }
    __syncthreads();   // dS tile complete
    // dQ tile (queries dq_qb*32.., dims dq_ct*32..) = dS K over the workgroup's 128 keys
    f32x16 qacc = f32x16{};
#pragma unroll
    for (int s = 0; s < C::kBK / 16; ++s) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(ds_s + (dq_qb * 32 + n) * C::kKTS + s * 16 + g * 8);
      const bf16x8 b = *reinterpret_cast<const bf16x8*>(kt_s + (dq_ct * 32 + n) * C::kKTS + s * 16 + g * 8);
      qacc = mfma32(a, b, qacc);
    }
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      const int64_t qi = q0 + dq_qb * 32 + 8 * (rr >> 2) + 4 * g + (rr & 3);
      if (qi < Nq) unsafeAtomicAdd(dqb + qi * D + dq_ct * 32 + n, qacc[rr] * scale);
    }
  }

  // dK = scale * dK^T^T, dV = dV^T^T for this lane's key
  if (key_ok) {
    const int64_t key = k0 + jl;
    float* dkr = dk + (bh * Nk + key) * D;
    float* dvr = dv + (bh * Nk + key) * D;
#pragma unroll
    for (int c = 0; c < C::kCT; ++c)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int col = c * 32 + 8 * rq + 4 * g;
        f32x4 kv = {dkt[c][4 * rq] * scale, dkt[c][4 * rq + 1] * scale,
                    dkt[c][4 * rq + 2] * scale, dkt[c][4 * rq + 3] * scale};
        f32x4 vv = {dvt[c][4 * rq], dvt[c][4 * rq + 1], dvt[c][4 * rq + 2], dvt[c][4 * rq + 3]};
        if (accumulate) {
          kv += *reinterpret_cast<const f32x4*>(dkr + col);
          vv += *reinterpret_cast<const f32x4*>(dvr + col);
        }
        *reinterpret_cast<f32x4*>(dkr + col) = kv;
        *reinterpret_cast<f32x4*>(dvr + col) = vv;
      }
  }
}

template <int D>
hipError_t launch(const BwdArgs& a) {
  using C = BwdCfg<D>;
  const int64_t max_chunk = (a.Nk + a.R - 1) / a.R;
  const int64_t tpc = (max_chunk + C::kBK - 1) / C::kBK;
  const int64_t nwg = a.BH * a.R * tpc;
  hipLaunchKernelGGL((bwd_bf16_kernel<D>), dim3((uint32_t)nwg), dim3(C::kThreads), 0, a.stream,
                     (const __bf16*)a.q, (const __bf16*)a.k, (const __bf16*)a.v,
                     (const __bf16*)a.dout, a.lse, a.delta, a.dq, a.dk, a.dv, (int)a.BH, a.Nq,
                     a.Nk, (int)a.R, (int)tpc, a.scale * kLog2e, a.scale,
                     a.accumulate_dkv ? 1 : 0);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd_bf16(const BwdArgs& a) {
  if (a.d == 128) return launch<128>(a);
  return launch<64>(a);
}

}  // namespace ringx
