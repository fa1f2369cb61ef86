// Host-side launch interface between the C ABI layer (ringx_api.cpp) and the kernel files.
// Arguments arrive here already validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ringx {

struct FwdArgs {
  const void* q;
  const void* k;
  const void* v;
  void* out;          // merged output (fused mode)
  float* lse;         // merged lse (fused mode)
  float* part_out;    // [R,B,H,Nq,d] (partials mode)
  float* part_lse;    // [R,B,H,Nq]   (partials mode)
  int64_t BH, Nq, Nk, d, R;
  float scale;
  hipStream_t stream;
};

struct MergeArgs {
  const float* part_out;
  const float* part_lse;
  void* out;
  float* lse;
  int64_t R, BH, Nq, d;
  bool out_bf16;
  hipStream_t stream;
};

struct BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* out;
  const void* dout;
  const float* lse;
  float* dq;
  float* dk;
  float* dv;
  float* delta;       // D_i = dout_i . out_i, [B,H,Nq]
  int64_t BH, Nq, Nk, d, R;
  float scale;
  bool accumulate_dkv;
  hipStream_t stream;
};

hipError_t launch_fwd_bf16(const FwdArgs& a, bool partials);
hipError_t launch_fwd_f32(const FwdArgs& a, bool partials);
hipError_t launch_lse_merge(const MergeArgs& a);
hipError_t launch_bwd_pre(const BwdArgs& a, bool bf16);
hipError_t launch_bwd_dkdv_bf16(const BwdArgs& a);
hipError_t launch_bwd_dq_bf16(const BwdArgs& a);
hipError_t launch_bwd_dkdv_f32(const BwdArgs& a);
hipError_t launch_bwd_dq_f32(const BwdArgs& a);

int64_t fwd_bf16_workgroups(int64_t BH, int64_t Nq, int64_t d);

}  // namespace ringx
