// Backward preprocess, per query row: D_i = sum_c dout_ic * out_ic (fp32), and the row's
// log-sum-exp in the base-2 exponent form the recompute uses, nl_i = -lse_i * log2(e).
//
// The recompute backward needs D_i for dS_ij = P_ij (dP_ij - D_i), and forms
// P_ij = exp2(scale * log2(e) * q_i.k_j + nl_i); with nl_i stored once here the key-stationary
// kernel, which meets 16 different query rows per lane and block, needs no multiply per score
// element for it.  HBM-bound: reads out, dout and lse once, writes D and nl once.

#include "ringx_device.h"
#include "ringx_kernels.h"

namespace ringx {
namespace {

constexpr int kPreThreads = 256;

// bf16: D/8 threads per row, 16-byte loads, shuffle reduction inside the row's lanes.
template <int D>
__global__ __launch_bounds__(kPreThreads) void bwd_pre_bf16_kernel(
    const __bf16* __restrict__ out, const __bf16* __restrict__ dout,
    const float* __restrict__ lse, float* __restrict__ delta, float* __restrict__ nl,
    int64_t rows) {
  constexpr int kTpr = D / 8;
  const int64_t idx = (int64_t)blockIdx.x * kPreThreads + threadIdx.x;
  const int64_t row = idx / kTpr;
  const int part = (int)(idx % kTpr);
  float s = 0.f;
  if (row < rows) {
    const u32x4 o = *reinterpret_cast<const u32x4*>(out + row * D + part * 8);
    const u32x4 g = *reinterpret_cast<const u32x4*>(dout + row * D + part * 8);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      s = __builtin_fmaf(bf16_lo(o[w]), bf16_lo(g[w]), s);
      s = __builtin_fmaf(bf16_hi(o[w]), bf16_hi(g[w]), s);
    }
  }
#pragma unroll
  for (int off = kTpr / 2; off > 0; off >>= 1) s += __shfl_xor(s, off, kTpr);
  if (row < rows && part == 0) {
    delta[row] = s;
    nl[row] = lse[row] * -kLog2e;
  }
}

__global__ __launch_bounds__(kPreThreads) void bwd_pre_f32_kernel(
    const float* __restrict__ out, const float* __restrict__ dout, const float* __restrict__ lse,
    float* __restrict__ delta, float* __restrict__ nl, int64_t rows, int d) {
  const int64_t row = (int64_t)blockIdx.x * kPreThreads + threadIdx.x;
  if (row >= rows) return;
  float s = 0.f;
  for (int c = 0; c < d; ++c) s = __builtin_fmaf(out[row * d + c], dout[row * d + c], s);
  delta[row] = s;
  nl[row] = lse[row] * -kLog2e;
}

}  // namespace

hipError_t launch_bwd_pre(const BwdArgs& a, bool bf16) {
  const int64_t rows = a.BH * a.Nq;
  if (bf16) {
    const int64_t n = rows * (a.d / 8);
    const dim3 grid((uint32_t)((n + kPreThreads - 1) / kPreThreads));
    if (a.d == 128)
      hipLaunchKernelGGL(bwd_pre_bf16_kernel<128>, grid, dim3(kPreThreads), 0, a.stream,
                         (const __bf16*)a.out, (const __bf16*)a.dout, a.lse, a.delta, a.nl,
                         rows);
    else
      hipLaunchKernelGGL(bwd_pre_bf16_kernel<64>, grid, dim3(kPreThreads), 0, a.stream,
                         (const __bf16*)a.out, (const __bf16*)a.dout, a.lse, a.delta, a.nl,
                         rows);
  } else {
    const dim3 grid((uint32_t)((rows + kPreThreads - 1) / kPreThreads));
    hipLaunchKernelGGL(bwd_pre_f32_kernel, grid, dim3(kPreThreads), 0, a.stream,
                       (const float*)a.out, (const float*)a.dout, a.lse, a.delta, a.nl, rows,
                       (int)a.d);
  }
  return hipGetLastError();
}

}  // namespace ringx
