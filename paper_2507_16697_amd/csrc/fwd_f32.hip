// Ring-chunked attention forward in fp32 (storage and arithmetic), any head dim 1..128.
//
// The exactness path: one thread per query row, keys streamed through LDS in tiles of 32.  For
// every chunk r the thread runs an online softmax over the chunk's keys (Eqs. (2)-(4) of arXiv
// 2507.16697 Sec. III-A), forms the chunk's local result (loc_out_r, loc_lse_r), and either writes
// it (partials mode) or folds it into the Eq. (5) merge.  The merged output accumulates in place in
// the fp32 output row, which only this thread touches: unnormalised, with Eq. (5)'s terms
// exp(loc_lse_r - M) loc_out_r = exp(m_r - M) o_r and exp(loc_lse_r - M) = exp(m_r - M) l_r kept
// relative to a running reference M (the largest m_r so far), and one division and one log at
// the end, so that rounding does not build up over many chunks.  Step mode (R = 1) folds the one
// chunk into a running fp32 (acc_out, acc_lse) left by earlier ring steps, which by the step
// contract holds the normalised result.

#include "ringx_device.h"
#include "ringx_kernels.h"

namespace ringx {
namespace {

constexpr int kF32Threads = 128;
constexpr int kF32Tile = 32;

template <int DMAX, int MODE>
__global__ __launch_bounds__(kF32Threads) void fwd_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ k, const float* __restrict__ v,
    float* __restrict__ out, float* __restrict__ lse, float* __restrict__ part_out,
    float* __restrict__ part_lse, float* __restrict__ acc_out, float* __restrict__ acc_lse,
    int first, int64_t BH, int H, int grp, int64_t Nq, int64_t Nk, int R, int d, float scale) {
  constexpr bool PARTIALS = MODE == (int)FwdMode::kPartials;
  constexpr bool STEP = MODE == (int)FwdMode::kStep;
  __shared__ float ks[kF32Tile * DMAX];
  __shared__ float vs[kF32Tile * DMAX];
  const int t = threadIdx.x;
  const int64_t bh = blockIdx.y;
  const int64_t qi = (int64_t)blockIdx.x * kF32Threads + t;
  const bool active = qi < Nq;
  const int64_t kvh = kv_head(bh, H, grp);
  const float* kb = k + kvh * Nk * d;
  const float* vb = v + kvh * Nk * d;

  float qr[DMAX];
#pragma unroll
  for (int c = 0; c < DMAX; ++c) qr[c] = (active && c < d) ? q[(bh * Nq + qi) * d + c] : 0.f;
  float* orow = (STEP ? acc_out : out) + (bh * Nq + (active ? qi : 0)) * d;
  // step mode starts from the running result of the earlier ring steps
  float lse_m = (STEP && !first && active) ? acc_lse[bh * Nq + qi] : -INFINITY;
  // fused mode: reference and denominator of the unnormalised merge
  float mref = -INFINITY, den = 0.f;

  for (int r = 0; r < R; ++r) {
    const int64_t lo = (int64_t)r * Nk / R;
    const int64_t hi = (int64_t)(r + 1) * Nk / R;
    float m = -INFINITY, l = 0.f;
    float o[DMAX];
#pragma unroll
    for (int c = 0; c < DMAX; ++c) o[c] = 0.f;
    for (int64_t j0 = lo; j0 < hi; j0 += kF32Tile) {
      const int nk = (int)min<int64_t>(kF32Tile, hi - j0);
      __syncthreads();
      for (int idx = t; idx < nk * d; idx += kF32Threads) {
        ks[(idx / d) * DMAX + idx % d] = kb[j0 * d + idx];
        vs[(idx / d) * DMAX + idx % d] = vb[j0 * d + idx];
      }
      __syncthreads();
      for (int j = 0; j < nk; ++j) {
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < DMAX; ++c)
          if (c < d) s = __builtin_fmaf(qr[c], ks[j * DMAX + c], s);
        s *= scale;
        const float mn = fmaxf(m, s);
        const float alpha = expf(m - mn);
        const float p = expf(s - mn);
        l = l * alpha + p;
#pragma unroll
        for (int c = 0; c < DMAX; ++c)
          if (c < d) o[c] = __builtin_fmaf(p, vs[j * DMAX + c], o[c] * alpha);
        m = mn;
      }
    }
    if (!active) continue;
    if constexpr (!PARTIALS && !STEP) {
      // Eq. (5) with a running reference: the row holds sum_r exp(m_r - mref) o_r
      if (m > mref) {
        const float f = expf(mref - m);   // 0 for the first chunk
#pragma unroll
        for (int c = 0; c < DMAX; ++c)
          if (c < d) orow[c] = (r == 0 ? 0.f : orow[c] * f) + o[c];
        den = den * f + l;
        mref = m;
      } else {
        const float w = expf(m - mref);
#pragma unroll
        for (int c = 0; c < DMAX; ++c)
          if (c < d) orow[c] = __builtin_fmaf(w, o[c], orow[c]);
        den = __builtin_fmaf(w, l, den);
      }
      continue;
    }
    const float inv = 1.0f / l;
    const float lse_r = m + logf(l);
    if constexpr (PARTIALS) {
      float* po = part_out + (((int64_t)r * BH + bh) * Nq + qi) * d;
#pragma unroll
      for (int c = 0; c < DMAX; ++c)
        if (c < d) po[c] = o[c] * inv;
      part_lse[((int64_t)r * BH + bh) * Nq + qi] = lse_r;
    } else {
      // Eq. (5), streamed: fold (loc_out_r, loc_lse_r) into the merged row
      const float M = fmaxf(lse_m, lse_r);
      const float a = expf(lse_m - M);
      const float b = expf(lse_r - M);
      const float ab = a + b;
      const float wa = a / ab;
      const float wb = b * inv / ab;
#pragma unroll
      for (int c = 0; c < DMAX; ++c)
        if (c < d) orow[c] = (lse_m == -INFINITY ? 0.f : orow[c] * wa) + o[c] * wb;
      lse_m = M + logf(ab);
    }
  }
  if constexpr (STEP) {
    if (active) acc_lse[bh * Nq + qi] = lse_m;
  } else if constexpr (!PARTIALS) {
    if (active) {
      const float inv = 1.0f / den;
#pragma unroll
      for (int c = 0; c < DMAX; ++c)
        if (c < d) orow[c] *= inv;
      lse[bh * Nq + qi] = mref + logf(den);
    }
  }
}

template <int DMAX, int MODE>
hipError_t launch(const FwdArgs& a) {
  dim3 grid((uint32_t)((a.Nq + kF32Threads - 1) / kF32Threads), (uint32_t)a.BH);
  hipLaunchKernelGGL((fwd_f32_kernel<DMAX, MODE>), grid, dim3(kF32Threads), 0, a.stream,
                     (const float*)a.q, (const float*)a.k, (const float*)a.v, (float*)a.out,
                     a.lse, a.part_out, a.part_lse, a.acc_out, a.acc_lse, a.first ? 1 : 0, a.BH,
                     (int)a.H, (int)a.G, a.Nq, a.Nk, (int)a.R, (int)a.d, a.scale);
  return hipGetLastError();
}

template <int DMAX>
hipError_t launch_mode(const FwdArgs& a, FwdMode mode) {
  switch (mode) {
    case FwdMode::kPartials: return launch<DMAX, (int)FwdMode::kPartials>(a);
    case FwdMode::kStep: return launch<DMAX, (int)FwdMode::kStep>(a);
    default: return launch<DMAX, (int)FwdMode::kFused>(a);
  }
}

}  // namespace

hipError_t launch_fwd_f32(const FwdArgs& a, FwdMode mode) {
  if (a.d <= 32) return launch_mode<32>(a, mode);
  if (a.d <= 64) return launch_mode<64>(a, mode);
  return launch_mode<128>(a, mode);
}

}  // namespace ringx
