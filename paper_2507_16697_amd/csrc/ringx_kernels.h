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

hipError_t launch_tt_tokenize(const TokArgs& a);

int64_t fwd_bf16_workgroups(int64_t BH, int64_t Nq, int64_t d);

}  // namespace ringx
