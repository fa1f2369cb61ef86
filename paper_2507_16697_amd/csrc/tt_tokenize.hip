// Multi-fidelity tokenizer of the Turbulence Transformer (arXiv 2507.16697 Sec. III-B; the
// filter / mode-size pairs of Table III): one fidelity mode of a field Y[c, z, y, x] is the
// periodic subdomain selection C(Y) of D/ratio x H/ratio x W/ratio cells around a centre, the k^3
// Gaussian filter F(.) applied with stride k (the D/k x H/k x W/k grid the paper gives for F(Y)),
// and patchify with patch p into tokens [L, C p^3] (token index x fastest, feature
// ((c p + iz) p + iy) p + ix).
//
// HBM-bound: the filter windows do not overlap, so every subdomain cell is read once and every
// token feature written once.  The unfiltered crop with patch 1 (Table III's filter 1) is a copy
// with one thread per cell and contiguous per-token stores.  For k a power of two a wave streams
// 256 consecutive cells of a row, 4 per lane, through the k^2 rows of its windows and accumulates
// in registers; the k cells of a window are then summed within the lane (k <= 4) or across k/4
// lanes by butterfly shuffles.  Other k take a plain kernel with one thread per filtered cell.
// The separable weights w_i w_j w_l come in as kernel arguments (computed on the host,
// normalised to sum 1).

#include "ringx_device.h"
#include "ringx_kernels.h"

namespace ringx {
namespace {

constexpr int kTokThreads = 256;
// four fp32 cells at 4-byte alignment
typedef float f32x4u __attribute__((ext_vector_type(4), aligned(4)));

__global__ __launch_bounds__(kTokThreads) void tt_tokenize_kernel(
    const float* __restrict__ field, void* __restrict__ tokens, int C, int D, int H, int W, int k,
    int gz, int gy, int gx, int z0, int y0, int x0, int p, TokWeights w, int out_bf16) {
  const int64_t n_out = (int64_t)C * gz * gy * gx;
  const int64_t idx = (int64_t)blockIdx.x * kTokThreads + threadIdx.x;
  if (idx >= n_out) return;
  const int e = (int)(idx % gx);
  int64_t r = idx / gx;
  const int b = (int)(r % gy);
  r /= gy;
  const int a = (int)(r % gz);
  const int c = (int)(r / gz);

  // first cell of the window in the (periodic) field; z0, y0, x0 are already in [0, D) etc.
  int zb = z0 + k * a;
  zb -= zb >= D ? D : 0;
  int yb = y0 + k * b;
  yb -= yb >= H ? H : 0;
  int xb = x0 + k * e;
  xb -= xb >= W ? W : 0;

  const float* fc = field + (int64_t)c * D * H * W;
  float acc = 0.f;
  for (int i = 0; i < k; ++i) {
    int z = zb + i;
    z -= z >= D ? D : 0;
    float accy = 0.f;
    for (int j = 0; j < k; ++j) {
      int y = yb + j;
      y -= y >= H ? H : 0;
      const float* row = fc + ((int64_t)z * H + y) * W;
      float accx = 0.f;
      for (int l = 0; l < k; ++l) {
        int x = xb + l;
        x -= x >= W ? W : 0;
        accx = __builtin_fmaf(w.w[l], row[x], accx);
      }
      accy = __builtin_fmaf(w.w[j], accx, accy);
    }
    acc = __builtin_fmaf(w.w[i], accy, acc);
  }

  // token (patch) index, x fastest, and feature within the token
  const int Py = gy / p, Px = gx / p;
  const int64_t t = ((int64_t)(a / p) * Py + b / p) * Px + e / p;
  const int f = ((c * p + a % p) * p + b % p) * p + e % p;
  const int64_t o = t * ((int64_t)C * p * p * p) + f;
  if (out_bf16) {
    reinterpret_cast<__bf16*>(tokens)[o] = (__bf16)acc;
  } else {
    reinterpret_cast<float*>(tokens)[o] = acc;
  }
}

// Row-streaming variant, K a power of two.  One wave = one (c, a, b) filtered row segment of 256
// subdomain cells along x (64 lanes x 4 cells); blockIdx.y picks the segment.
template <int K>
__global__ __launch_bounds__(kTokThreads) void tt_tokenize_rows_kernel(
    const float* __restrict__ field, void* __restrict__ tokens, int C, int D, int H, int W, int sx,
    int gz, int gy, int gx, int z0, int y0, int x0, int p, TokWeights w, int out_bf16) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (kTokThreads / 64) + (threadIdx.x >> 6);
  if (row >= (int64_t)C * gz * gy) return;
  const int b = (int)(row % gy);
  const int a = (int)((row / gy) % gz);
  const int c = (int)(row / ((int64_t)gy * gz));
  const int pos = blockIdx.y * 256 + 4 * lane;      // first of this lane's 4 subdomain cells
  const bool active = pos < sx;                     // sx is a multiple of K and of 4 when K >= 4

  int xs = x0 + pos;
  xs -= xs >= W ? W : 0;
  // one 16-byte load when the 4 cells do not wrap (4-byte alignment is all a multi-dword global
  // load needs, so a subdomain that starts off a 16-byte boundary streams the same way)
  const bool contiguous = active && xs + 4 <= W;
  const float* fc = field + (int64_t)c * D * H * W;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < K; ++i) {
    int z = z0 + K * a + i;
    z -= z >= D ? D : 0;
    z -= z >= D ? D : 0;
    for (int j = 0; j < K; ++j) {
      int y = y0 + K * b + j;
      y -= y >= H ? H : 0;
      y -= y >= H ? H : 0;
      const float wij = w.w[i] * w.w[j];
      const float* rowp = fc + ((int64_t)z * H + y) * W;
      if (contiguous) {
        // the field is streamed once: non-temporal loads, except for the unfiltered crop (k = 1),
        // whose short row segments are latency-bound
        const f32x4u* vp = reinterpret_cast<const f32x4u*>(rowp + xs);
        const f32x4 v = K > 1 ? __builtin_nontemporal_load(vp) : *vp;
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] = __builtin_fmaf(wij, v[e], acc[e]);
      } else if (active) {
        cold_path();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          int x = xs + e;
          x -= x >= W ? W : 0;
          acc[e] = __builtin_fmaf(wij, rowp[x], acc[e]);
        }
      }
    }
  }
  // x weights, then the window sums: within the lane for K <= 4, across K/4 lanes otherwise
  float part[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) part[e] = acc[e] * w.w[(pos + e) & (K - 1)];
  constexpr int kPerLane = K < 4 ? 4 / K : 1;      // windows completed inside one lane
  float win[kPerLane];
#pragma unroll
  for (int q = 0; q < kPerLane; ++q) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < (K < 4 ? K : 4); ++e) s += part[q * (K < 4 ? K : 4) + e];
    win[q] = s;
  }
  if constexpr (K > 4) {
#pragma unroll
    for (int m = 1; m < K / 4; m <<= 1) win[0] += __shfl_xor(win[0], m);
    if ((lane & (K / 4 - 1)) != 0) return;
  }
  if (!active) return;
  const int Py = gy / p, Px = gx / p;
  const int64_t feat = (int64_t)C * p * p * p;
#pragma unroll
  for (int q = 0; q < kPerLane; ++q) {
    const int e = pos / K + q;                       // filtered cell along x
    const int64_t t = ((int64_t)(a / p) * Py + b / p) * Px + e / p;
    const int f = ((c * p + a % p) * p + b % p) * p + e % p;
    if (out_bf16) reinterpret_cast<__bf16*>(tokens)[t * feat + f] = (__bf16)win[q];
    else reinterpret_cast<float*>(tokens)[t * feat + f] = win[q];
  }
}

// The unfiltered crop (k = 1) with patch 1: token t = subdomain cell (z, y, x), x fastest, and its
// C features are the C channels of that cell.  One thread per cell: the channel loads of
// consecutive threads are consecutive cells of a row (coalesced), and each thread writes its C
// features as one contiguous run (16-byte stores of 4 channels when C is a multiple of 4), so
// every output line is written whole by neighbouring threads.
template <bool OUT_BF16>
__global__ __launch_bounds__(kTokThreads) void tt_crop_kernel(
    const float* __restrict__ field, void* __restrict__ tokens, int C, int D, int H, int W,
    int sz, int sy, int sx, int z0, int y0, int x0) {
  const int64_t n = (int64_t)sz * sy * sx;
  const int64_t i = (int64_t)blockIdx.x * kTokThreads + threadIdx.x;
  if (i >= n) return;
  const int x = (int)(i % sx);
  const int64_t r = i / sx;
  const int y = (int)(r % sy);
  const int z = (int)(r / sy);
  int zz = z0 + z, yy = y0 + y, xx = x0 + x;
  zz -= zz >= D ? D : 0;
  yy -= yy >= H ? H : 0;
  xx -= xx >= W ? W : 0;
  const int64_t plane = (int64_t)D * H * W;
  const float* src = field + ((int64_t)zz * H + yy) * W + xx;
  if ((C & 3) == 0) {
    for (int c = 0; c < C; c += 4) {
      const f32x4 v = {src[c * plane], src[(c + 1) * plane], src[(c + 2) * plane],
                       src[(c + 3) * plane]};
      if constexpr (OUT_BF16) {
        u32x2 w2;
        w2[0] = pack_bf16x2(v[0], v[1]);
        w2[1] = pack_bf16x2(v[2], v[3]);
        *reinterpret_cast<u32x2*>(reinterpret_cast<__bf16*>(tokens) + i * C + c) = w2;
      } else {
        *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(tokens) + i * C + c) = v;
      }
    }
  } else {
    for (int c = 0; c < C; ++c) {
      const float v = src[c * plane];
      if constexpr (OUT_BF16) reinterpret_cast<__bf16*>(tokens)[i * C + c] = (__bf16)v;
      else reinterpret_cast<float*>(tokens)[i * C + c] = v;
    }
  }
}

template <int K>
hipError_t launch_rows(const TokArgs& a) {
  const int64_t rows = a.C * a.gz * a.gy;
  const int sx = (int)(a.gx * K);
  dim3 grid((uint32_t)((rows + kTokThreads / 64 - 1) / (kTokThreads / 64)),
            (uint32_t)((sx + 255) / 256));
  hipLaunchKernelGGL((tt_tokenize_rows_kernel<K>), grid, dim3(kTokThreads), 0, a.stream, a.field,
                     a.tokens, (int)a.C, (int)a.D, (int)a.H, (int)a.W, sx, (int)a.gz, (int)a.gy,
                     (int)a.gx, (int)a.z0, (int)a.y0, (int)a.x0, (int)a.p, a.w,
                     a.out_bf16 ? 1 : 0);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tt_tokenize(const TokArgs& a) {
  if (a.k == 1 && a.p == 1) {
    // the unfiltered crop: one thread per subdomain cell (the weight of a 1-cell window is 1)
    const int64_t n = a.gz * a.gy * a.gx;
    const dim3 grid((uint32_t)((n + kTokThreads - 1) / kTokThreads));
    if (a.out_bf16)
      hipLaunchKernelGGL(tt_crop_kernel<true>, grid, dim3(kTokThreads), 0, a.stream, a.field,
                         a.tokens, (int)a.C, (int)a.D, (int)a.H, (int)a.W, (int)a.gz, (int)a.gy,
                         (int)a.gx, (int)a.z0, (int)a.y0, (int)a.x0);
    else
      hipLaunchKernelGGL(tt_crop_kernel<false>, grid, dim3(kTokThreads), 0, a.stream, a.field,
                         a.tokens, (int)a.C, (int)a.D, (int)a.H, (int)a.W, (int)a.gz, (int)a.gy,
                         (int)a.gx, (int)a.z0, (int)a.y0, (int)a.x0);
    return hipGetLastError();
  }
  // the row kernel needs 4-cell lane groups inside the subdomain row: sx % 4 == 0
  const int64_t sx = a.gx * a.k;
  const int64_t rows = a.C * a.gz * a.gy;
  if (sx % 4 == 0 && (sx + 255) / 256 <= 65535 && (rows + 3) / 4 <= 0xffffffffll) {
    switch (a.k) {
      case 1: return launch_rows<1>(a);
      case 2: return launch_rows<2>(a);
      case 4: return launch_rows<4>(a);
      case 8: return launch_rows<8>(a);
      case 16: return launch_rows<16>(a);
      case 32: return launch_rows<32>(a);
      default: break;
    }
  }
  const int64_t n_out = a.C * a.gz * a.gy * a.gx;
  const int64_t blocks = (n_out + kTokThreads - 1) / kTokThreads;
  hipLaunchKernelGGL(tt_tokenize_kernel, dim3((uint32_t)blocks), dim3(kTokThreads), 0, a.stream,
                     a.field, a.tokens, (int)a.C, (int)a.D, (int)a.H, (int)a.W, (int)a.k,
                     (int)a.gz, (int)a.gy, (int)a.gx, (int)a.z0, (int)a.y0, (int)a.x0, (int)a.p,
                     a.w, a.out_bf16 ? 1 : 0);
  return hipGetLastError();
}

}  // namespace ringx
