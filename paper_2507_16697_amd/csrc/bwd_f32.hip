// Recompute backward in fp32 (storage and arithmetic), any head dim 1..128: the exactness path.
//
// Two plain kernels: one thread per key accumulates dK_j, dV_j over every query (of every query
// head sharing the key's K/V head); one thread per query accumulates dQ_i over every key.  Both recompute P_ij = exp(scale q_i.k_j - lse_i) from
// the merged log-sum-exp and dS_ij = P_ij (dout_i.v_j - D_i).

#include "ringx_device.h"
#include "ringx_kernels.h"

namespace ringx {
namespace {

constexpr int kThreads = 128;

template <int DMAX>
__global__ __launch_bounds__(kThreads) void bwd_f32_dkdv_kernel(
    const float* __restrict__ q, const float* __restrict__ k, const float* __restrict__ v,
    const float* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ delta,
    float* __restrict__ dk, float* __restrict__ dv, int64_t Nq, int64_t Nk, int d, float scale,
    int accumulate, int H, int grp) {
  const int64_t bh = blockIdx.y;   // K/V head (of B * H / G)
  const int64_t j = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (j >= Nk) return;
  float kr[DMAX], vr[DMAX], gk[DMAX], gv[DMAX];
#pragma unroll
  for (int c = 0; c < DMAX; ++c) {
    kr[c] = c < d ? k[(bh * Nk + j) * d + c] : 0.f;
    vr[c] = c < d ? v[(bh * Nk + j) * d + c] : 0.f;
    gk[c] = 0.f;
    gv[c] = 0.f;
  }
  // the grp query heads sharing this K/V head each add their gradient contributions
  const int hkv = H / grp;
  const int64_t qh0 = (bh / hkv) * H + (bh % hkv) * grp;
  for (int jh = 0; jh < grp; ++jh) {
    const float* qb = q + (qh0 + jh) * Nq * d;
    const float* ob = dout + (qh0 + jh) * Nq * d;
    const float* lb = lse + (qh0 + jh) * Nq;
    const float* db = delta + (qh0 + jh) * Nq;
    for (int64_t i = 0; i < Nq; ++i) {
      float s = 0.f, dp = 0.f;
#pragma unroll
      for (int c = 0; c < DMAX; ++c)
        if (c < d) {
          s = __builtin_fmaf(qb[i * d + c], kr[c], s);
          dp = __builtin_fmaf(ob[i * d + c], vr[c], dp);
        }
      const float p = expf(s * scale - lb[i]);
      const float ds = p * (dp - db[i]);
#pragma unroll
      for (int c = 0; c < DMAX; ++c)
        if (c < d) {
          gv[c] = __builtin_fmaf(p, ob[i * d + c], gv[c]);
          gk[c] = __builtin_fmaf(ds, qb[i * d + c], gk[c]);
        }
    }
  }
#pragma unroll
  for (int c = 0; c < DMAX; ++c)
    if (c < d) {
      const int64_t o = (bh * Nk + j) * d + c;
      dk[o] = (accumulate ? dk[o] : 0.f) + gk[c] * scale;
      dv[o] = (accumulate ? dv[o] : 0.f) + gv[c];
    }
}

template <int DMAX>
__global__ __launch_bounds__(kThreads) void bwd_f32_dq_kernel(
    const float* __restrict__ q, const float* __restrict__ k, const float* __restrict__ v,
    const float* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ delta,
    float* __restrict__ dq, int64_t Nq, int64_t Nk, int d, float scale, int accumulate, int H,
    int grp) {
  const int64_t bh = blockIdx.y;
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= Nq) return;
  float qr[DMAX], orr[DMAX], gq[DMAX];
#pragma unroll
  for (int c = 0; c < DMAX; ++c) {
    qr[c] = c < d ? q[(bh * Nq + i) * d + c] : 0.f;
    orr[c] = c < d ? dout[(bh * Nq + i) * d + c] : 0.f;
    gq[c] = 0.f;
  }
  const float l = lse[bh * Nq + i];
  const float D = delta[bh * Nq + i];
  const int64_t kvh = kv_head(bh, H, grp);
  const float* kb = k + kvh * Nk * d;
  const float* vb = v + kvh * Nk * d;
  for (int64_t j = 0; j < Nk; ++j) {
    float s = 0.f, dp = 0.f;
#pragma unroll
    for (int c = 0; c < DMAX; ++c)
      if (c < d) {
        s = __builtin_fmaf(qr[c], kb[j * d + c], s);
        dp = __builtin_fmaf(orr[c], vb[j * d + c], dp);
      }
    const float ds = expf(s * scale - l) * (dp - D);
#pragma unroll
    for (int c = 0; c < DMAX; ++c)
      if (c < d) gq[c] = __builtin_fmaf(ds, kb[j * d + c], gq[c]);
  }
#pragma unroll
  for (int c = 0; c < DMAX; ++c)
    if (c < d) {
      float* dst = dq + (bh * Nq + i) * d + c;
      *dst = (accumulate ? *dst : 0.f) + gq[c] * scale;
    }
}

template <int DMAX>
hipError_t launch_dkdv(const BwdArgs& a) {
  const dim3 gk((uint32_t)((a.Nk + kThreads - 1) / kThreads), (uint32_t)(a.BH / a.G));
  hipLaunchKernelGGL((bwd_f32_dkdv_kernel<DMAX>), gk, dim3(kThreads), 0, a.stream,
                     (const float*)a.q, (const float*)a.k, (const float*)a.v,
                     (const float*)a.dout, a.lse, a.delta, a.dk, a.dv, a.Nq, a.Nk, (int)a.d,
                     a.scale, a.accumulate_dkv ? 1 : 0, (int)a.H, (int)a.G);
  return hipGetLastError();
}

template <int DMAX>
hipError_t launch_dq(const BwdArgs& a) {
  const dim3 gq((uint32_t)((a.Nq + kThreads - 1) / kThreads), (uint32_t)a.BH);
  hipLaunchKernelGGL((bwd_f32_dq_kernel<DMAX>), gq, dim3(kThreads), 0, a.stream,
                     (const float*)a.q, (const float*)a.k, (const float*)a.v,
                     (const float*)a.dout, a.lse, a.delta, a.dq, a.Nq, a.Nk, (int)a.d, a.scale,
                     a.accumulate_dq ? 1 : 0, (int)a.H, (int)a.G);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd_dkdv_f32(const BwdArgs& a) {
  if (a.d <= 32) return launch_dkdv<32>(a);
  if (a.d <= 64) return launch_dkdv<64>(a);
  return launch_dkdv<128>(a);
}

hipError_t launch_bwd_dq_f32(const BwdArgs& a) {
  if (a.d <= 32) return launch_dq<32>(a);
  if (a.d <= 64) return launch_dq<64>(a);
  return launch_dq<128>(a);
}

}  // namespace ringx
