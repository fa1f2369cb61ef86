// Host-side launch interface between the C ABI layer (ringx_api.cpp) and the kernel files.
// Arguments arrive here already validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ringx {

// What the forward does with each chunk's local result (loc_out_r, loc_lse_r).
enum class FwdMode {
  kFused = 0,     // Eq. (5) merge of all R chunks in registers -> out, lse
  kPartials = 1,  // write every chunk's result -> part_out, part_lse
  kStep = 2,      // R = 1: merge the one chunk into the running fp32 acc_out, acc_lse
};

struct FwdArgs {
  const void* q = nullptr;
  const void* k = nullptr;
  const void* v = nullptr;
  void* out = nullptr;          // merged output (fused mode)
  float* lse = nullptr;         // merged lse (fused mode)
  float* part_out = nullptr;    // [R,B,H,Nq,d] (partials mode)
  float* part_lse = nullptr;    // [R,B,H,Nq]   (partials mode)
  float* acc_out = nullptr;     // [B,H,Nq,d] running merged output (step mode)
  float* acc_lse = nullptr;     // [B,H,Nq]   running merged lse (step mode)
  bool first = false;           // step mode: the accumulator holds nothing yet
  int64_t BH = 0, Nq = 0, Nk = 0, d = 0, R = 1;
  int64_t H = 1, G = 1;         // query heads per batch; query heads per K/V head (GQA)
  float scale = 1.f;
  hipStream_t stream = nullptr;
};

struct MergeArgs {
  const float* part_out = nullptr;
  const float* part_lse = nullptr;
  void* out = nullptr;
  float* lse = nullptr;
  int64_t R = 1, BH = 0, Nq = 0, d = 0;
  bool out_bf16 = false;
  hipStream_t stream = nullptr;
};

struct BwdArgs {
  const void* q = nullptr;
  const void* k = nullptr;
  const void* v = nullptr;
  const void* out = nullptr;
  const void* dout = nullptr;
  const float* lse = nullptr;
  float* dq = nullptr;
  float* dk = nullptr;
  float* dv = nullptr;
  float* delta = nullptr;       // D_i = dout_i . out_i, [B,H,Nq]
  float* nl = nullptr;          // -lse_i * log2(e), [B,H,Nq] (the exponent's offset, base 2)
  int64_t BH = 0, Nq = 0, Nk = 0, d = 0, R = 1;   // BH = B * H query heads
  int64_t H = 1, G = 1;         // query heads per batch; query heads per K/V head (GQA)
  float scale = 1.f;
  bool accumulate_dkv = false;  // dk, dv += instead of =
  bool accumulate_dq = false;   // dq += instead of =
  char* ds = nullptr;           // store mode of the dK/dV kernel: -dS of every score, bf16
  hipStream_t stream = nullptr;
};

// Stored dS (written by the dK/dV kernel in store mode, read by bwd_dq_ds.hip): per query head j,
// 32-key block kb of the padded key axis (chunk r, 128-key tile t, block w: kb = 4 (r tpc + t) + w,
// nkb = 4 R tpc blocks), 128-query group qg and 32-query block qs of the group, one unit of
// kDsUnitBytes.  The query axis runs fastest, so that each wave of the writer, which owns one key
// block and sweeps the queries, writes one contiguous stream.
constexpr int64_t kDsUnitBytes = 2048;
__host__ __device__ inline int64_t ds_unit_offset(int64_t j, int64_t qg, int64_t kb, int64_t qs,
                                                  int64_t nqg, int64_t nkb) {
  return (((j * nkb + kb) * nqg + qg) * 4 + qs) * kDsUnitBytes;
}
// 128-key tiles per chunk (the longest chunk, ceil(Nk / R) keys, rounded up)
__host__ __device__ inline int64_t ds_tiles_per_chunk(int64_t Nk, int64_t R) {
  return ((Nk + R - 1) / R + 127) / 128;
}
// bytes of stored dS for nh query heads
inline int64_t ds_bytes(int64_t nh, int64_t Nq, int64_t Nk, int64_t R) {
  return nh * ((Nq + 127) / 128) * 4 * R * ds_tiles_per_chunk(Nk, R) * 4 * kDsUnitBytes;
}

struct DsArgs {
  const void* ds = nullptr;     // stored -dS of nh query heads
  const void* k = nullptr;      // K of the nh / G K/V heads, [nh / G, Nk, 128] bf16
  float* dq = nullptr;          // [nh, Nq, 128] fp32, overwritten
  int64_t nh = 0, G = 1, Nq = 0, Nk = 0, R = 1, tpc = 1;
  float scale = 1.f;
  hipStream_t stream = nullptr;
};

// One fidelity mode of the multi-fidelity tokenizer (tt_tokenize.hip).
constexpr int kMaxTokFilter = 32;
struct TokWeights {
  float w[kMaxTokFilter];       // normalised 1D Gaussian weights, w[0 .. k-1]
};
struct TokArgs {
  const float* field = nullptr;  // [C, D, H, W] fp32
  void* tokens = nullptr;        // [L, C p^3], fp32 or bf16
  int64_t C = 0, D = 0, H = 0, W = 0, k = 1, p = 1;
  int64_t gz = 0, gy = 0, gx = 0;   // filtered grid: subdomain size / k
  int64_t z0 = 0, y0 = 0, x0 = 0;   // first subdomain cell, in [0, D) x [0, H) x [0, W)
  TokWeights w{};
  bool out_bf16 = false;
  hipStream_t stream = nullptr;
};

hipError_t launch_fwd_bf16(const FwdArgs& a, FwdMode mode);
hipError_t launch_fwd_f32(const FwdArgs& a, FwdMode mode);
hipError_t launch_lse_merge(const MergeArgs& a);
hipError_t launch_bwd_pre(const BwdArgs& a, bool bf16);
hipError_t launch_bwd_dkdv_bf16(const BwdArgs& a);
hipError_t launch_bwd_dkdv_bf16_d64(const BwdArgs& a);   // d = 64 (bwd_bf16_d64.hip)
hipError_t launch_bwd_dq_bf16(const BwdArgs& a);
hipError_t launch_bwd_dq_bf16_d64(const BwdArgs& a);   // d = 64 (bwd_dq_bf16_d64.hip)
hipError_t launch_bwd_dkdv_f32(const BwdArgs& a);
hipError_t launch_bwd_dq_f32(const BwdArgs& a);
hipError_t launch_bwd_dq_ds(const DsArgs& a);   // d = 128, bf16 dS (bwd_dq_ds.hip)

hipError_t launch_tt_tokenize(const TokArgs& a);

int64_t fwd_bf16_workgroups(int64_t BH, int64_t Nq, int64_t d);

}  // namespace ringx
