// Standalone N-way merge of per-chunk partial results, Eq. (5) of arXiv 2507.16697 Sec. III-A.
//
//   lse_max = max_r part_lse[r]          (the paper's allreduce-max)
//   w_r     = exp(part_lse[r] - lse_max)
//   out     = sum_r w_r part_out[r] / sum_r w_r,   lse = lse_max + log(sum_r w_r)
//
// HBM-bound: each output row reads R fp32 rows of d values and R log-sum-exps once.  Vector path:
// one thread per one or two quads of 4 consecutive columns of a row (16-byte loads, consecutive
// threads cover a row), the partial loop unrolled so that several rows are in flight per thread,
// and the partials and the output streamed with non-temporal loads and stores (each is touched
// once); scalar path for head dims that are not a multiple of 4 (fp32 output only).

#include "ringx_device.h"
#include "ringx_kernels.h"

namespace ringx {
namespace {

// 512-thread workgroups: 5% more bandwidth than 256 at the 8-way ring share's 2.3 GB merge (A/B
// in one job, 6.28 against 5.96 TB/s; a plain non-temporal read of the same bytes reaches 6.78)
constexpr int kMergeThreads = 512;

// Q quads of 4 columns per thread, at columns c + j d / Q (j < Q), so that each load instruction
// of a wave still covers consecutive 16-byte pieces of a row.  Q = 2 keeps twice the bytes in
// flight per thread, which pays when few partials (R < 8) give each thread few loads: 12-18% more
// bandwidth at R = 2-4 (d = 64 and 128), 3-6% less at R = 8 (A/B in one job, bitwise equal).
template <bool OUT_BF16, int Q>
__global__ __launch_bounds__(kMergeThreads) void merge_vec4_kernel(
    const float* __restrict__ part_out, const float* __restrict__ part_lse, void* __restrict__ out,
    float* __restrict__ lse, int R, int64_t rows, int d) {
  const int groups = d / (4 * Q);
  const int64_t idx = (int64_t)blockIdx.x * kMergeThreads + threadIdx.x;
  if (idx >= rows * groups) return;
  const int64_t row = idx / groups;
  const int c = (int)(idx % groups) * 4;
  const int step = d / Q;

  float M = -INFINITY;
#pragma unroll 8
  for (int r = 0; r < R; ++r) M = fmaxf(M, part_lse[(int64_t)r * rows + row]);
  f32x4 acc[Q];
#pragma unroll
  for (int j = 0; j < Q; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float den = 0.f;
  // unrolled so that several partial rows are in flight per thread
#pragma unroll 8
  for (int r = 0; r < R; ++r) {
    const float w = fast_exp2((part_lse[(int64_t)r * rows + row] - M) * kLog2e);
    const float* src = part_out + ((int64_t)r * rows + row) * d + c;
#pragma unroll
    for (int j = 0; j < Q; ++j)
      acc[j] += __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src + j * step)) * w;
    den += w;
  }
  const float inv = 1.0f / den;
#pragma unroll
  for (int j = 0; j < Q; ++j) {
    const f32x4 v = acc[j] * inv;
    const int64_t o = row * d + c + j * step;
    if constexpr (OUT_BF16) {
      u32x2 w2;
      w2[0] = pack_bf16x2(v[0], v[1]);
      w2[1] = pack_bf16x2(v[2], v[3]);
      __builtin_nontemporal_store(w2, reinterpret_cast<u32x2*>(reinterpret_cast<__bf16*>(out) + o));
    } else {
      __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(reinterpret_cast<float*>(out) + o));
    }
  }
  if (c == 0) lse[row] = M + logf(den);
}

template <int Q>
void launch_vec4(const MergeArgs& a, int64_t rows) {
  const int64_t n = rows * (a.d / (4 * Q));
  const dim3 grid((uint32_t)((n + kMergeThreads - 1) / kMergeThreads));
  if (a.out_bf16)
    hipLaunchKernelGGL((merge_vec4_kernel<true, Q>), grid, dim3(kMergeThreads), 0, a.stream,
                       a.part_out, a.part_lse, a.out, a.lse, (int)a.R, rows, (int)a.d);
  else
    hipLaunchKernelGGL((merge_vec4_kernel<false, Q>), grid, dim3(kMergeThreads), 0, a.stream,
                       a.part_out, a.part_lse, a.out, a.lse, (int)a.R, rows, (int)a.d);
}

__global__ __launch_bounds__(kMergeThreads) void merge_scalar_kernel(
    const float* __restrict__ part_out, const float* __restrict__ part_lse,
    float* __restrict__ out, float* __restrict__ lse, int R, int64_t rows, int d) {
  const int64_t idx = (int64_t)blockIdx.x * kMergeThreads + threadIdx.x;
  if (idx >= rows * d) return;
  const int64_t row = idx / d;
  const int c = (int)(idx % d);
  float M = -INFINITY;
  for (int r = 0; r < R; ++r) M = fmaxf(M, part_lse[(int64_t)r * rows + row]);
  float acc = 0.f, den = 0.f;
  for (int r = 0; r < R; ++r) {
    const float w = expf(part_lse[(int64_t)r * rows + row] - M);
    acc = __builtin_fmaf(w, part_out[((int64_t)r * rows + row) * d + c], acc);
    den += w;
  }
  out[row * d + c] = acc / den;
  if (c == 0) lse[row] = M + logf(den);
}

}  // namespace

hipError_t launch_lse_merge(const MergeArgs& a) {
  const int64_t rows = a.BH * a.Nq;
  if (a.d % 8 == 0 && a.R < 8) {
    launch_vec4<2>(a, rows);
  } else if (a.d % 4 == 0) {
    launch_vec4<1>(a, rows);
  } else {
    const int64_t n = rows * a.d;
    const dim3 grid((uint32_t)((n + kMergeThreads - 1) / kMergeThreads));
    hipLaunchKernelGGL(merge_scalar_kernel, grid, dim3(kMergeThreads), 0, a.stream, a.part_out,
                       a.part_lse, (float*)a.out, a.lse, (int)a.R, rows, (int)a.d);
  }
  return hipGetLastError();
}

}  // namespace ringx
