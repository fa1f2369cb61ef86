// C ABI of libringx (declared in include/ringx.h): host-side validation, workspace sizing and
// kernel dispatch.  Every check runs before the first HIP call, so an error status means nothing
// was enqueued and no output was touched.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <climits>
#include <initializer_list>
#include <mutex>

#include "ringx.h"
#include "ringx_kernels.h"

namespace {

constexpr int64_t kMaxElems = int64_t(1) << 40;   // per tensor; keeps every index product in int64
constexpr int64_t kMaxRowsF32 = 65535;            // fp32 kernels put B*H on grid.y
constexpr int64_t kMaxKeys = int64_t(1) << 31;    // keeps r * Nk (chunk bounds) inside int64
// queries per head: the kernels keep query positions in 32 bits, with a tile of headroom
constexpr int64_t kMaxQueries = (int64_t(1) << 31) - 128;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Span {
  uintptr_t lo, hi;
};
Span span(const void* p, int64_t bytes) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  return Span{a, a + static_cast<uintptr_t>(bytes)};
}
bool overlap(Span a, Span b) { return a.lo < b.hi && b.lo < a.hi; }

int64_t esize(ringx_dtype t) { return t == RINGX_BF16 ? 2 : 4; }

bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a < 0 || b < 0) return false;
  if (a != 0 && b > kMaxElems / a) return false;
  *out = a * b;
  return *out <= kMaxElems;
}

ringx_status check_dims(int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t d, int64_t R,
                        float scale, ringx_dtype dtype) {
  if (B < 1 || H < 1 || Nq < 1 || Nk < 1 || Nk > kMaxKeys || Nq > kMaxQueries) return RINGX_E_SHAPE;
  if (!(std::isfinite(scale) && scale > 0.f)) return RINGX_E_SHAPE;
  if (dtype != RINGX_BF16 && dtype != RINGX_FP32) return RINGX_E_UNSUPPORTED;
  if (dtype == RINGX_BF16 && d != 64 && d != 128) return RINGX_E_UNSUPPORTED;
  if (dtype == RINGX_FP32 && (d < 1 || d > 128)) return RINGX_E_UNSUPPORTED;
  if (R < 1 || R > Nk) return RINGX_E_CHUNKS;
  int64_t bh, x;
  if (!mul_ok(B, H, &bh)) return RINGX_E_SHAPE;
  if (dtype == RINGX_FP32 && bh > kMaxRowsF32) return RINGX_E_SHAPE;
  if (!mul_ok(bh, Nq, &x) || !mul_ok(x, d, &x) || !mul_ok(x, R, &x)) return RINGX_E_SHAPE;
  if (!mul_ok(bh, Nk, &x) || !mul_ok(x, d, &x)) return RINGX_E_SHAPE;
  if (dtype == RINGX_BF16 && ringx::fwd_bf16_workgroups(bh, Nq, d) > 0xffffffffll)
    return RINGX_E_SHAPE;
  // the backward grid: one workgroup per (b, h, chunk, 128-key tile)
  if (dtype == RINGX_BF16) {
    const int64_t tpc = ((Nk + R - 1) / R + 127) / 128;
    if (!mul_ok(bh, R, &x) || !mul_ok(x, tpc, &x) || x > 0xffffffffll) return RINGX_E_SHAPE;
  }
  return RINGX_OK;
}

ringx_status hip_status(hipError_t e) { return e == hipSuccess ? RINGX_OK : RINGX_E_HIP; }

}  // namespace

extern "C" {

const char* ringx_status_str(int status) {
  // an int, not the enum: a C caller may pass any value, and an out-of-range enum is undefined
  switch (status) {
    case RINGX_OK: return "ok";
    case RINGX_E_NULLPTR: return "a required pointer is NULL";
    case RINGX_E_SHAPE: return "invalid shape, size overflow or scale";
    case RINGX_E_CHUNKS: return "chunk count or index out of range (need 1 <= R <= Nk)";
    case RINGX_E_UNSUPPORTED: return "unsupported dtype or head dim";
    case RINGX_E_ALIGN: return "tensor pointer not 16-byte aligned";
    case RINGX_E_WORKSPACE: return "backward workspace missing or too small";
    case RINGX_E_HIP: return "HIP launch failed";
    case RINGX_E_ALIAS: return "an output overlaps an input";
    case RINGX_E_SCRATCH:
      return "B * H * Nq exceeds the fixed scratch of ringx_attn_bwd_noalloc "
             "(RINGX_NOALLOC_MAX_ROWS rows)";
  }
  return "unknown status";
}

ringx_status ringx_chunk_bounds(int64_t Nk, int64_t R, int64_t r, int64_t* lo, int64_t* hi) {
  if (!lo || !hi) return RINGX_E_NULLPTR;
  if (Nk < 1 || Nk > kMaxElems) return RINGX_E_SHAPE;
  if (R < 1 || R > Nk || r < 0 || r >= R) return RINGX_E_CHUNKS;
  // r * Nk < 2^40 * 2^40 would overflow int64 for extreme inputs; split the product
  const int64_t qn = Nk / R, rn = Nk % R;
  *lo = r * qn + (r * rn) / R;
  *hi = (r + 1) * qn + ((r + 1) * rn) / R;
  return RINGX_OK;
}

}  // extern "C"

namespace {

// Forward with Hkv K/V heads serving H query heads (Hkv divides H; Hkv = H is plain MHA).
ringx_status fwd_impl(const void* q, const void* k, const void* v, void* out, float* lse,
                      int64_t B, int64_t H, int64_t Hkv, int64_t Nq, int64_t Nk, int64_t d,
                      int64_t R, float scale, ringx_dtype dtype, hipStream_t stream) {
  if (!q || !k || !v || !out || !lse) return RINGX_E_NULLPTR;
  if (Hkv < 1 || H < 1 || H % Hkv != 0) return RINGX_E_SHAPE;
  ringx_status st = check_dims(B, H, Nq, Nk, d, R, scale, dtype);
  if (st != RINGX_OK) return st;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) || !aligned16(lse))
    return RINGX_E_ALIGN;
  const int64_t es = esize(dtype), bh = B * H, bkv = B * Hkv;
  const Span sq = span(q, bh * Nq * d * es), sk = span(k, bkv * Nk * d * es),
             sv = span(v, bkv * Nk * d * es);
  const Span so = span(out, bh * Nq * d * es), sl = span(lse, bh * Nq * 4);
  for (Span o : {so, sl})
    for (Span i : {sq, sk, sv})
      if (overlap(o, i)) return RINGX_E_ALIAS;
  if (overlap(so, sl)) return RINGX_E_ALIAS;
  ringx::FwdArgs a;
  a.q = q, a.k = k, a.v = v, a.out = out, a.lse = lse;
  a.BH = bh, a.Nq = Nq, a.Nk = Nk, a.d = d, a.R = R, a.scale = scale, a.stream = stream;
  a.H = H, a.G = H / Hkv;
  return hip_status(dtype == RINGX_BF16 ? ringx::launch_fwd_bf16(a, ringx::FwdMode::kFused)
                                        : ringx::launch_fwd_f32(a, ringx::FwdMode::kFused));
}

}  // namespace

extern "C" {

ringx_status ringx_attn_fwd(const void* q, const void* k, const void* v, void* out, float* lse,
                            int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t d, int64_t R,
                            float scale, ringx_dtype dtype, hipStream_t stream) {
  return fwd_impl(q, k, v, out, lse, B, H, H, Nq, Nk, d, R, scale, dtype, stream);
}

ringx_status ringx_attn_fwd_gqa(const void* q, const void* k, const void* v, void* out,
                                float* lse, int64_t B, int64_t H, int64_t Hkv, int64_t Nq,
                                int64_t Nk, int64_t d, int64_t R, float scale, ringx_dtype dtype,
                                hipStream_t stream) {
  return fwd_impl(q, k, v, out, lse, B, H, Hkv, Nq, Nk, d, R, scale, dtype, stream);
}

ringx_status ringx_attn_fwd_partials(const void* q, const void* k, const void* v, float* part_out,
                                     float* part_lse, int64_t B, int64_t H, int64_t Nq, int64_t Nk,
                                     int64_t d, int64_t R, float scale, ringx_dtype dtype,
                                     hipStream_t stream) {
  if (!q || !k || !v || !part_out || !part_lse) return RINGX_E_NULLPTR;
  ringx_status st = check_dims(B, H, Nq, Nk, d, R, scale, dtype);
  if (st != RINGX_OK) return st;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(part_out) ||
      !aligned16(part_lse))
    return RINGX_E_ALIGN;
  const int64_t es = esize(dtype), bh = B * H;
  const Span sq = span(q, bh * Nq * d * es), sk = span(k, bh * Nk * d * es),
             sv = span(v, bh * Nk * d * es);
  const Span so = span(part_out, R * bh * Nq * d * 4), sl = span(part_lse, R * bh * Nq * 4);
  for (Span o : {so, sl})
    for (Span i : {sq, sk, sv})
      if (overlap(o, i)) return RINGX_E_ALIAS;
  if (overlap(so, sl)) return RINGX_E_ALIAS;
  ringx::FwdArgs a;
  a.q = q, a.k = k, a.v = v, a.part_out = part_out, a.part_lse = part_lse;
  a.BH = bh, a.Nq = Nq, a.Nk = Nk, a.d = d, a.R = R, a.scale = scale, a.stream = stream;
  a.H = H, a.G = 1;
  return hip_status(dtype == RINGX_BF16 ? ringx::launch_fwd_bf16(a, ringx::FwdMode::kPartials)
                                        : ringx::launch_fwd_f32(a, ringx::FwdMode::kPartials));
}

ringx_status ringx_lse_merge(const float* part_out, const float* part_lse, void* out, float* lse,
                             int64_t R, int64_t B, int64_t H, int64_t Nq, int64_t d,
                             ringx_dtype out_dtype, hipStream_t stream) {
  if (!part_out || !part_lse || !out || !lse) return RINGX_E_NULLPTR;
  if (B < 1 || H < 1 || Nq < 1) return RINGX_E_SHAPE;
  if (R < 1) return RINGX_E_CHUNKS;
  if (out_dtype != RINGX_BF16 && out_dtype != RINGX_FP32) return RINGX_E_UNSUPPORTED;
  if (d < 1 || d > 128 || (out_dtype == RINGX_BF16 && d % 4 != 0)) return RINGX_E_UNSUPPORTED;
  int64_t bh, x;
  if (!mul_ok(B, H, &bh) || !mul_ok(bh, Nq, &x) || !mul_ok(x, d, &x) || !mul_ok(x, R, &x))
    return RINGX_E_SHAPE;
  if ((bh * Nq * d + 255) / 256 > 0xffffffffll) return RINGX_E_SHAPE;
  if (!aligned16(part_out) || !aligned16(part_lse) || !aligned16(out) || !aligned16(lse))
    return RINGX_E_ALIGN;
  const Span si = span(part_out, R * bh * Nq * d * 4), sil = span(part_lse, R * bh * Nq * 4);
  const Span so = span(out, bh * Nq * d * esize(out_dtype)), sl = span(lse, bh * Nq * 4);
  for (Span o : {so, sl})
    for (Span i : {si, sil})
      if (overlap(o, i)) return RINGX_E_ALIAS;
  if (overlap(so, sl)) return RINGX_E_ALIAS;
  ringx::MergeArgs a;
  a.part_out = part_out, a.part_lse = part_lse, a.out = out, a.lse = lse;
  a.R = R, a.BH = bh, a.Nq = Nq, a.d = d, a.out_bf16 = out_dtype == RINGX_BF16, a.stream = stream;
  return hip_status(ringx::launch_lse_merge(a));
}


ringx_status ringx_bwd_preprocess(const void* out, const void* dout, const float* lse,
                                  float* delta, int64_t B, int64_t H, int64_t Nq, int64_t d,
                                  ringx_dtype dtype, hipStream_t stream) {
  if (!out || !dout || !lse || !delta) return RINGX_E_NULLPTR;
  ringx_status st = check_dims(B, H, Nq, 1, d, 1, 1.0f, dtype);
  if (st != RINGX_OK) return st;
  for (const void* p : {out, dout, (const void*)lse, (const void*)delta})
    if (!aligned16(p)) return RINGX_E_ALIGN;
  const int64_t es = esize(dtype), bh = B * H;
  const Span sd = span(delta, 2 * bh * Nq * 4);
  if (overlap(sd, span(out, bh * Nq * d * es)) || overlap(sd, span(dout, bh * Nq * d * es)) ||
      overlap(sd, span(lse, bh * Nq * 4)))
    return RINGX_E_ALIAS;
  ringx::BwdArgs a;
  a.out = out, a.dout = dout, a.lse = lse, a.delta = delta, a.nl = delta + bh * Nq;
  a.BH = bh, a.Nq = Nq, a.Nk = 1, a.d = d, a.R = 1, a.stream = stream, a.H = H, a.G = 1;
  return hip_status(ringx::launch_bwd_pre(a, dtype == RINGX_BF16));
}

namespace {

// Shared validation of the two gradient stages; `outs` are the fp32 outputs being written.
ringx_status check_bwd_stage(const void* q, const void* k, const void* v, const void* dout,
                             const float* lse, const float* delta,
                             std::initializer_list<Span> outs, int64_t B, int64_t H, int64_t Nq,
                             int64_t Nk, int64_t d, int64_t R, float scale, ringx_dtype dtype) {
  if (!q || !k || !v || !dout || !lse || !delta) return RINGX_E_NULLPTR;
  ringx_status st = check_dims(B, H, Nq, Nk, d, R, scale, dtype);
  if (st != RINGX_OK) return st;
  for (const void* p : {q, k, v, dout, (const void*)lse, (const void*)delta})
    if (!aligned16(p)) return RINGX_E_ALIGN;
  for (const Span& o : outs)
    if ((o.lo & 15u) != 0) return RINGX_E_ALIGN;
  const int64_t es = esize(dtype), bh = B * H;
  const Span ins[] = {span(q, bh * Nq * d * es), span(k, bh * Nk * d * es),
                      span(v, bh * Nk * d * es), span(dout, bh * Nq * d * es),
                      span(lse, bh * Nq * 4), span(delta, 2 * bh * Nq * 4)};
  for (auto oi = outs.begin(); oi != outs.end(); ++oi) {
    for (const Span& i : ins)
      if (overlap(*oi, i)) return RINGX_E_ALIAS;
    for (auto oj = oi + 1; oj != outs.end(); ++oj)
      if (overlap(*oi, *oj)) return RINGX_E_ALIAS;
  }
  return RINGX_OK;
}

}  // namespace

ringx_status ringx_attn_bwd_dkdv(const void* q, const void* k, const void* v, const void* dout,
                                 const float* lse, const float* delta, float* dk, float* dv,
                                 int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t d,
                                 int64_t R, float scale, ringx_dtype dtype, int accumulate_dkv,
                                 hipStream_t stream) {
  if (!dk || !dv) return RINGX_E_NULLPTR;
  const int64_t bh = B * H;
  ringx_status st = check_bwd_stage(q, k, v, dout, lse, delta,
                                    {span(dk, bh * Nk * d * 4), span(dv, bh * Nk * d * 4)}, B, H,
                                    Nq, Nk, d, R, scale, dtype);
  if (st != RINGX_OK) return st;
  ringx::BwdArgs a;
  a.q = q, a.k = k, a.v = v, a.dout = dout, a.lse = lse, a.dk = dk, a.dv = dv;
  a.delta = const_cast<float*>(delta), a.nl = const_cast<float*>(delta) + bh * Nq;
  a.BH = bh, a.Nq = Nq, a.Nk = Nk, a.d = d, a.R = R, a.scale = scale, a.H = H, a.G = 1;
  a.accumulate_dkv = accumulate_dkv != 0, a.stream = stream;
  return hip_status(dtype == RINGX_BF16 ? ringx::launch_bwd_dkdv_bf16(a)
                                        : ringx::launch_bwd_dkdv_f32(a));
}

ringx_status ringx_attn_bwd_dq(const void* q, const void* k, const void* v, const void* dout,
                               const float* lse, const float* delta, float* dq, int64_t B,
                               int64_t H, int64_t Nq, int64_t Nk, int64_t d, int64_t R,
                               float scale, ringx_dtype dtype, hipStream_t stream) {
  if (!dq) return RINGX_E_NULLPTR;
  const int64_t bh = B * H;
  ringx_status st = check_bwd_stage(q, k, v, dout, lse, delta, {span(dq, bh * Nq * d * 4)}, B, H,
                                    Nq, Nk, d, R, scale, dtype);
  if (st != RINGX_OK) return st;
  ringx::BwdArgs a;
  a.q = q, a.k = k, a.v = v, a.dout = dout, a.lse = lse, a.dq = dq;
  a.delta = const_cast<float*>(delta), a.nl = const_cast<float*>(delta) + bh * Nq;
  a.BH = bh, a.Nq = Nq, a.Nk = Nk, a.d = d, a.R = R, a.scale = scale, a.stream = stream;
  a.H = H, a.G = 1;
  return hip_status(dtype == RINGX_BF16 ? ringx::launch_bwd_dq_bf16(a)
                                        : ringx::launch_bwd_dq_f32(a));
}

size_t ringx_bwd_workspace_bytes(int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t d,
                                 int64_t R, ringx_dtype dtype) {
  if (check_dims(B, H, Nq, Nk, d, R, 1.0f, dtype) != RINGX_OK) return 0;
  const int64_t stats = 2 * B * H * Nq * 4;   // D and nl of every query row
  return static_cast<size_t>((stats + 255) / 256 * 256);
}

}  // extern "C"

namespace {

ringx_status bwd_impl(const void* q, const void* k, const void* v, const void* out,
                      const void* dout, const float* lse, float* dq, float* dk, float* dv,
                      int64_t B, int64_t H, int64_t Hkv, int64_t Nq, int64_t Nk, int64_t d,
                      int64_t R, float scale, ringx_dtype dtype, int accumulate_dkv,
                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!q || !k || !v || !out || !dout || !lse || !dq || !dk || !dv) return RINGX_E_NULLPTR;
  if (Hkv < 1 || H < 1 || H % Hkv != 0) return RINGX_E_SHAPE;
  ringx_status st = check_dims(B, H, Nq, Nk, d, R, scale, dtype);
  if (st != RINGX_OK) return st;
  const size_t need = ringx_bwd_workspace_bytes(B, H, Nq, Nk, d, R, dtype);
  if (!workspace || workspace_bytes < need) return RINGX_E_WORKSPACE;
  for (const void* p : {q, k, v, out, dout, (const void*)lse, (const void*)dq, (const void*)dk,
                        (const void*)dv, (const void*)workspace})
    if (!aligned16(p)) return RINGX_E_ALIGN;
  const int64_t es = esize(dtype), bh = B * H, bkv = B * Hkv;
  const Span ins[] = {span(q, bh * Nq * d * es),    span(k, bkv * Nk * d * es),
                      span(v, bkv * Nk * d * es),   span(out, bh * Nq * d * es),
                      span(dout, bh * Nq * d * es), span(lse, bh * Nq * 4)};
  const Span outs[] = {span(dq, bh * Nq * d * 4), span(dk, bkv * Nk * d * 4),
                       span(dv, bkv * Nk * d * 4), span(workspace, (int64_t)need)};
  for (int i = 0; i < 4; ++i) {
    for (const Span& s : ins)
      if (overlap(outs[i], s)) return RINGX_E_ALIAS;
    for (int j = i + 1; j < 4; ++j)
      if (overlap(outs[i], outs[j])) return RINGX_E_ALIAS;
  }
  float* delta = static_cast<float*>(workspace);
  ringx::BwdArgs a;
  a.q = q, a.k = k, a.v = v, a.out = out, a.dout = dout, a.lse = lse;
  a.dq = dq, a.dk = dk, a.dv = dv, a.delta = delta, a.nl = delta + bh * Nq;
  a.BH = bh, a.Nq = Nq, a.Nk = Nk, a.d = d, a.R = R, a.scale = scale;
  a.H = H, a.G = H / Hkv;
  a.accumulate_dkv = accumulate_dkv != 0, a.stream = stream;
  const bool bf16 = dtype == RINGX_BF16;
  if (ringx::launch_bwd_pre(a, bf16) != hipSuccess) return RINGX_E_HIP;
  if ((bf16 ? ringx::launch_bwd_dkdv_bf16(a) : ringx::launch_bwd_dkdv_f32(a)) != hipSuccess)
    return RINGX_E_HIP;
  return hip_status(bf16 ? ringx::launch_bwd_dq_bf16(a) : ringx::launch_bwd_dq_f32(a));
}

}  // namespace

extern "C" {

ringx_status ringx_attn_bwd(const void* q, const void* k, const void* v, const void* out,
                            const void* dout, const float* lse, float* dq, float* dk, float* dv,
                            int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t d, int64_t R,
                            float scale, ringx_dtype dtype, int accumulate_dkv, void* workspace,
                            size_t workspace_bytes, hipStream_t stream) {
  return bwd_impl(q, k, v, out, dout, lse, dq, dk, dv, B, H, H, Nq, Nk, d, R, scale, dtype,
                  accumulate_dkv, workspace, workspace_bytes, stream);
}

ringx_status ringx_attn_bwd_gqa(const void* q, const void* k, const void* v, const void* out,
                                const void* dout, const float* lse, float* dq, float* dk,
                                float* dv, int64_t B, int64_t H, int64_t Hkv, int64_t Nq,
                                int64_t Nk, int64_t d, int64_t R, float scale, ringx_dtype dtype,
                                int accumulate_dkv, void* workspace, size_t workspace_bytes,
                                hipStream_t stream) {
  return bwd_impl(q, k, v, out, dout, lse, dq, dk, dv, B, H, Hkv, Nq, Nk, d, R, scale, dtype,
                  accumulate_dkv, workspace, workspace_bytes, stream);
}

size_t ringx_bwd_ds_bytes(int64_t H, int64_t Hkv, int64_t Nq, int64_t Nk, int64_t d, int64_t R,
                          int64_t kv_count) {
  if (Hkv < 1 || H < 1 || H % Hkv != 0 || kv_count < 1) return 0;
  if (check_dims(1, H, Nq, Nk, d, R, 1.0f, RINGX_BF16) != RINGX_OK || d != 128) return 0;
  int64_t nh, x;
  if (!mul_ok(kv_count, H / Hkv, &nh)) return 0;
  // nh query heads x ceil(Nq/128) groups x 4 R tpc key blocks x 4 units of 2 KiB
  const int64_t tpc = ringx::ds_tiles_per_chunk(Nk, R);
  if (!mul_ok(nh, (Nq + 127) / 128, &x) || !mul_ok(x, 16 * R, &x) || !mul_ok(x, tpc, &x))
    return 0;
  if (x > (int64_t(1) << 62) / ringx::kDsUnitBytes) return 0;
  return static_cast<size_t>(ringx::ds_bytes(nh, Nq, Nk, R));
}

size_t ringx_bwd_ds_workspace_bytes(int64_t B, int64_t H, int64_t Hkv, int64_t Nq, int64_t Nk,
                                    int64_t d, int64_t R, int64_t kv_per_slab) {
  if (B < 1 || Hkv < 1 || kv_per_slab < 1 || kv_per_slab > B * Hkv) return 0;
  const size_t stats = ringx_bwd_workspace_bytes(B, H, Nq, Nk, d, R, RINGX_BF16);
  const size_t ds = ringx_bwd_ds_bytes(H, Hkv, Nq, Nk, d, R, kv_per_slab);
  if (stats == 0 || ds == 0) return 0;
  return stats + ds;
}

}  // extern "C"

namespace {

// Validation shared by the two stored-dS stages: shapes, the slab [kv_begin, kv_begin +
// kv_count) of the B * Hkv K/V heads, and the stored-dS buffer.
ringx_status check_ds_common(const void* ds, size_t ds_bytes, int64_t B, int64_t H, int64_t Hkv,
                             int64_t Nq, int64_t Nk, int64_t d, int64_t R, float scale,
                             ringx_dtype dtype, int64_t kv_begin, int64_t kv_count) {
  if (Hkv < 1 || H < 1 || H % Hkv != 0) return RINGX_E_SHAPE;
  ringx_status st = check_dims(B, H, Nq, Nk, d, R, scale, dtype);
  if (st != RINGX_OK) return st;
  if (dtype != RINGX_BF16 || d != 128) return RINGX_E_UNSUPPORTED;
  if (kv_begin < 0 || kv_count < 1 || kv_begin > B * Hkv - kv_count) return RINGX_E_SHAPE;
  const size_t need = ringx_bwd_ds_bytes(H, Hkv, Nq, Nk, d, R, kv_count);
  if (need == 0) return RINGX_E_SHAPE;
  if (!ds || ds_bytes < need) return RINGX_E_WORKSPACE;
  if (!aligned16(ds)) return RINGX_E_ALIGN;
  // the dQ grid: one workgroup per (query head, 128 queries)
  if (kv_count * (H / Hkv) * ((Nq + 127) / 128) > 0xffffffffll) return RINGX_E_SHAPE;
  return RINGX_OK;
}

}  // namespace

extern "C" {

ringx_status ringx_attn_bwd_dkdv_ds(const void* q, const void* k, const void* v, const void* dout,
                                    const float* lse, const float* delta, float* dk, float* dv,
                                    void* ds, size_t ds_bytes, int64_t B, int64_t H, int64_t Hkv,
                                    int64_t Nq, int64_t Nk, int64_t d, int64_t R, float scale,
                                    ringx_dtype dtype, int accumulate_dkv, int64_t kv_begin,
                                    int64_t kv_count, hipStream_t stream) {
  if (!q || !k || !v || !dout || !lse || !delta || !dk || !dv) return RINGX_E_NULLPTR;
  ringx_status st = check_ds_common(ds, ds_bytes, B, H, Hkv, Nq, Nk, d, R, scale, dtype,
                                    kv_begin, kv_count);
  if (st != RINGX_OK) return st;
  for (const void* p : {q, k, v, dout, (const void*)lse, (const void*)delta, (const void*)dk,
                        (const void*)dv})
    if (!aligned16(p)) return RINGX_E_ALIGN;
  const int64_t bh = B * H, bkv = B * Hkv, G = H / Hkv;
  const size_t need = ringx_bwd_ds_bytes(H, Hkv, Nq, Nk, d, R, kv_count);
  const Span ins[] = {span(q, bh * Nq * d * 2),    span(k, bkv * Nk * d * 2),
                      span(v, bkv * Nk * d * 2),   span(dout, bh * Nq * d * 2),
                      span(lse, bh * Nq * 4),      span(delta, 2 * bh * Nq * 4)};
  const Span outs[] = {span(dk, bkv * Nk * d * 4), span(dv, bkv * Nk * d * 4),
                       span(ds, (int64_t)need)};
  for (int i = 0; i < 3; ++i) {
    for (const Span& s : ins)
      if (overlap(outs[i], s)) return RINGX_E_ALIAS;
    for (int j = i + 1; j < 3; ++j)
      if (overlap(outs[i], outs[j])) return RINGX_E_ALIAS;
  }
  // the slab as a batch of kv_count K/V heads with G query heads each (query head h of K/V head
  // m is m G + h in batch-major order)
  const int64_t q0 = kv_begin * G;
  ringx::BwdArgs a;
  a.q = static_cast<const char*>(q) + q0 * Nq * d * 2;
  a.dout = static_cast<const char*>(dout) + q0 * Nq * d * 2;
  a.k = static_cast<const char*>(k) + kv_begin * Nk * d * 2;
  a.v = static_cast<const char*>(v) + kv_begin * Nk * d * 2;
  a.dk = dk + kv_begin * Nk * d, a.dv = dv + kv_begin * Nk * d;
  a.delta = const_cast<float*>(delta) + q0 * Nq;
  a.nl = const_cast<float*>(delta) + bh * Nq + q0 * Nq;
  a.ds = static_cast<char*>(ds);
  a.BH = kv_count * G, a.Nq = Nq, a.Nk = Nk, a.d = d, a.R = R, a.scale = scale;
  a.H = G, a.G = G;
  a.accumulate_dkv = accumulate_dkv != 0, a.stream = stream;
  return hip_status(ringx::launch_bwd_dkdv_bf16(a));
}

ringx_status ringx_attn_bwd_dq_ds(const void* ds, size_t ds_bytes, const void* k, float* dq,
                                  int64_t B, int64_t H, int64_t Hkv, int64_t Nq, int64_t Nk,
                                  int64_t d, int64_t R, float scale, ringx_dtype dtype,
                                  int64_t kv_begin, int64_t kv_count, hipStream_t stream) {
  if (!k || !dq) return RINGX_E_NULLPTR;
  ringx_status st = check_ds_common(ds, ds_bytes, B, H, Hkv, Nq, Nk, d, R, scale, dtype,
                                    kv_begin, kv_count);
  if (st != RINGX_OK) return st;
  if (!aligned16(k) || !aligned16(dq)) return RINGX_E_ALIGN;
  const int64_t bh = B * H, bkv = B * Hkv, G = H / Hkv;
  const size_t need = ringx_bwd_ds_bytes(H, Hkv, Nq, Nk, d, R, kv_count);
  const Span so = span(dq, bh * Nq * d * 4);
  if (overlap(so, span(ds, (int64_t)need)) || overlap(so, span(k, bkv * Nk * d * 2)))
    return RINGX_E_ALIAS;
  ringx::DsArgs a;
  a.ds = ds;
  a.k = static_cast<const char*>(k) + kv_begin * Nk * d * 2;
  a.dq = dq + kv_begin * G * Nq * d;
  a.nh = kv_count * G, a.G = G, a.Nq = Nq, a.Nk = Nk, a.R = R;
  a.tpc = ringx::ds_tiles_per_chunk(Nk, R), a.scale = scale, a.stream = stream;
  return hip_status(ringx::launch_bwd_dq_ds(a));
}

ringx_status ringx_attn_bwd_ds(const void* q, const void* k, const void* v, const void* out,
                               const void* dout, const float* lse, float* dq, float* dk,
                               float* dv, int64_t B, int64_t H, int64_t Hkv, int64_t Nq,
                               int64_t Nk, int64_t d, int64_t R, float scale, ringx_dtype dtype,
                               int accumulate_dkv, void* workspace, size_t workspace_bytes,
                               hipStream_t stream) {
  if (!q || !k || !v || !out || !dout || !lse || !dq || !dk || !dv) return RINGX_E_NULLPTR;
  if (Hkv < 1 || H < 1 || H % Hkv != 0) return RINGX_E_SHAPE;
  ringx_status st = check_dims(B, H, Nq, Nk, d, R, scale, dtype);
  if (st != RINGX_OK) return st;
  if (dtype != RINGX_BF16 || d != 128) return RINGX_E_UNSUPPORTED;
  const size_t stats = ringx_bwd_workspace_bytes(B, H, Nq, Nk, d, R, dtype);
  const size_t per_kv = ringx_bwd_ds_bytes(H, Hkv, Nq, Nk, d, R, 1);
  if (stats == 0 || per_kv == 0) return RINGX_E_SHAPE;
  if (!workspace || workspace_bytes < stats + per_kv) return RINGX_E_WORKSPACE;
  for (const void* p : {q, k, v, out, dout, (const void*)lse, (const void*)dq, (const void*)dk,
                        (const void*)dv, (const void*)workspace})
    if (!aligned16(p)) return RINGX_E_ALIGN;
  const int64_t bh = B * H, bkv = B * Hkv;
  // as many K/V heads per slab as the workspace holds (and the dQ grid allows)
  const int64_t wg_per_kv = (H / Hkv) * ((Nq + 127) / 128);
  if (wg_per_kv > 0xffffffffll) return RINGX_E_SHAPE;
  int64_t per_slab = (int64_t)((workspace_bytes - stats) / per_kv);
  if (per_slab > bkv) per_slab = bkv;
  if (per_slab > 0xffffffffll / wg_per_kv) per_slab = 0xffffffffll / wg_per_kv;
  while (per_slab > 1 && ringx_bwd_ds_bytes(H, Hkv, Nq, Nk, d, R, per_slab) == 0) --per_slab;
  const size_t used = stats + ringx_bwd_ds_bytes(H, Hkv, Nq, Nk, d, R, per_slab);
  const Span ins[] = {span(q, bh * Nq * d * 2),    span(k, bkv * Nk * d * 2),
                      span(v, bkv * Nk * d * 2),   span(out, bh * Nq * d * 2),
                      span(dout, bh * Nq * d * 2), span(lse, bh * Nq * 4)};
  const Span outs[] = {span(dq, bh * Nq * d * 4), span(dk, bkv * Nk * d * 4),
                       span(dv, bkv * Nk * d * 4), span(workspace, (int64_t)used)};
  for (int i = 0; i < 4; ++i) {
    for (const Span& s : ins)
      if (overlap(outs[i], s)) return RINGX_E_ALIAS;
    for (int j = i + 1; j < 4; ++j)
      if (overlap(outs[i], outs[j])) return RINGX_E_ALIAS;
  }
  float* delta = static_cast<float*>(workspace);
  char* ds = static_cast<char*>(workspace) + stats;
  const size_t ds_cap = workspace_bytes - stats;
  {
    ringx::BwdArgs a;
    a.out = out, a.dout = dout, a.lse = lse, a.delta = delta, a.nl = delta + bh * Nq;
    a.BH = bh, a.Nq = Nq, a.Nk = 1, a.d = d, a.R = 1, a.stream = stream, a.H = H, a.G = 1;
    if (ringx::launch_bwd_pre(a, true) != hipSuccess) return RINGX_E_HIP;
  }
  for (int64_t kv0 = 0; kv0 < bkv; kv0 += per_slab) {
    const int64_t cnt = kv0 + per_slab <= bkv ? per_slab : bkv - kv0;
    st = ringx_attn_bwd_dkdv_ds(q, k, v, dout, lse, delta, dk, dv, ds, ds_cap, B, H, Hkv, Nq, Nk,
                                d, R, scale, dtype, accumulate_dkv, kv0, cnt, stream);
    if (st != RINGX_OK) return st == RINGX_E_HIP ? st : RINGX_E_HIP;
    st = ringx_attn_bwd_dq_ds(ds, ds_cap, k, dq, B, H, Hkv, Nq, Nk, d, R, scale, dtype, kv0, cnt,
                              stream);
    if (st != RINGX_OK) return st == RINGX_E_HIP ? st : RINGX_E_HIP;
  }
  return RINGX_OK;
}

ringx_status ringx_attn_fwd_step(const void* q, const void* k, const void* v, float* out_acc,
                                 float* lse_acc, int64_t B, int64_t H, int64_t Nq, int64_t Nk,
                                 int64_t d, float scale, ringx_dtype dtype, int first,
                                 hipStream_t stream) {
  if (!q || !k || !v || !out_acc || !lse_acc) return RINGX_E_NULLPTR;
  ringx_status st = check_dims(B, H, Nq, Nk, d, 1, scale, dtype);
  if (st != RINGX_OK) return st;
  for (const void* p : {q, k, v, (const void*)out_acc, (const void*)lse_acc})
    if (!aligned16(p)) return RINGX_E_ALIGN;
  const int64_t es = esize(dtype), bh = B * H;
  const Span sq = span(q, bh * Nq * d * es), sk = span(k, bh * Nk * d * es),
             sv = span(v, bh * Nk * d * es);
  const Span so = span(out_acc, bh * Nq * d * 4), sl = span(lse_acc, bh * Nq * 4);
  for (Span o : {so, sl})
    for (Span i : {sq, sk, sv})
      if (overlap(o, i)) return RINGX_E_ALIAS;
  if (overlap(so, sl)) return RINGX_E_ALIAS;
  ringx::FwdArgs a;
  a.q = q, a.k = k, a.v = v, a.acc_out = out_acc, a.acc_lse = lse_acc, a.first = first != 0;
  a.BH = bh, a.Nq = Nq, a.Nk = Nk, a.d = d, a.R = 1, a.scale = scale, a.stream = stream;
  a.H = H, a.G = 1;
  return hip_status(dtype == RINGX_BF16 ? ringx::launch_fwd_bf16(a, ringx::FwdMode::kStep)
                                        : ringx::launch_fwd_f32(a, ringx::FwdMode::kStep));
}

ringx_status ringx_attn_bwd_step(const void* q, const void* k, const void* v, const void* dout,
                                 const float* lse, const float* delta, float* dq_acc, float* dk,
                                 float* dv, int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t d,
                                 float scale, ringx_dtype dtype, int accumulate_dq,
                                 int accumulate_dkv, hipStream_t stream) {
  if (!dq_acc || !dk || !dv) return RINGX_E_NULLPTR;
  const int64_t bh = B * H;
  ringx_status st = check_bwd_stage(
      q, k, v, dout, lse, delta,
      {span(dq_acc, bh * Nq * d * 4), span(dk, bh * Nk * d * 4), span(dv, bh * Nk * d * 4)}, B, H,
      Nq, Nk, d, 1, scale, dtype);
  if (st != RINGX_OK) return st;
  ringx::BwdArgs a;
  a.q = q, a.k = k, a.v = v, a.dout = dout, a.lse = lse, a.delta = const_cast<float*>(delta);
  a.nl = const_cast<float*>(delta) + bh * Nq;
  a.dq = dq_acc, a.dk = dk, a.dv = dv;
  a.BH = bh, a.Nq = Nq, a.Nk = Nk, a.d = d, a.R = 1, a.scale = scale, a.H = H, a.G = 1;
  a.accumulate_dkv = accumulate_dkv != 0, a.accumulate_dq = accumulate_dq != 0, a.stream = stream;
  const bool bf16 = dtype == RINGX_BF16;
  if ((bf16 ? ringx::launch_bwd_dkdv_bf16(a) : ringx::launch_bwd_dkdv_f32(a)) != hipSuccess)
    return RINGX_E_HIP;
  return hip_status(bf16 ? ringx::launch_bwd_dq_bf16(a) : ringx::launch_bwd_dq_f32(a));
}

ringx_status ringx_tt_tokenize(const float* field, void* tokens, int64_t C, int64_t D, int64_t H,
                               int64_t W, int64_t k, int64_t ratio, int64_t cz, int64_t cy,
                               int64_t cx, int64_t p, float sigma, ringx_dtype out_dtype,
                               hipStream_t stream) {
  if (!field || !tokens) return RINGX_E_NULLPTR;
  if (C < 1 || D < 1 || H < 1 || W < 1 || k < 1 || ratio < 1 || p < 1) return RINGX_E_SHAPE;
  if (k > ringx::kMaxTokFilter) return RINGX_E_UNSUPPORTED;
  if (out_dtype != RINGX_BF16 && out_dtype != RINGX_FP32) return RINGX_E_UNSUPPORTED;
  if (!(std::isfinite(sigma) && sigma > 0.f)) return RINGX_E_SHAPE;
  if (D % ratio || H % ratio || W % ratio) return RINGX_E_SHAPE;
  const int64_t sz = D / ratio, sy = H / ratio, sx = W / ratio;   // subdomain
  if (sz % (k * p) || sy % (k * p) || sx % (k * p)) return RINGX_E_SHAPE;
  if (cz < 0 || cz >= D || cy < 0 || cy >= H || cx < 0 || cx >= W) return RINGX_E_SHAPE;
  int64_t n_in, n_out;
  if (!mul_ok(C, D, &n_in) || !mul_ok(n_in, H, &n_in) || !mul_ok(n_in, W, &n_in))
    return RINGX_E_SHAPE;
  if (D > INT32_MAX / 2 || H > INT32_MAX / 2 || W > INT32_MAX / 2) return RINGX_E_SHAPE;
  const int64_t gz = sz / k, gy = sy / k, gx = sx / k;
  if (!mul_ok(C, gz, &n_out) || !mul_ok(n_out, gy, &n_out) || !mul_ok(n_out, gx, &n_out))
    return RINGX_E_SHAPE;
  if ((n_out + 255) / 256 > 0xffffffffll) return RINGX_E_SHAPE;
  if (!aligned16(field) || !aligned16(tokens)) return RINGX_E_ALIGN;
  if (overlap(span(field, n_in * 4), span(tokens, n_out * esize(out_dtype))))
    return RINGX_E_ALIAS;
  ringx::TokArgs a;
  a.field = field, a.tokens = tokens, a.out_bf16 = out_dtype == RINGX_BF16, a.stream = stream;
  a.C = C, a.D = D, a.H = H, a.W = W, a.k = k, a.p = p, a.gz = gz, a.gy = gy, a.gx = gx;
  // first cell of the subdomain, size // 2 cells before the centre, taken periodically
  a.z0 = ((cz - sz / 2) % D + D) % D;
  a.y0 = ((cy - sy / 2) % H + H) % H;
  a.x0 = ((cx - sx / 2) % W + W) % W;
  double wd[ringx::kMaxTokFilter], total = 0.0;
  for (int64_t i = 0; i < k; ++i) {
    const double u = (double)i - (double)(k - 1) / 2.0;
    wd[i] = std::exp(-u * u / (2.0 * (double)sigma * (double)sigma));
    total += wd[i];
  }
  for (int64_t i = 0; i < k; ++i) a.w.w[i] = (float)(wd[i] / total);
  return hip_status(ringx::launch_tt_tokenize(a));
}

}  // extern "C"

// ------------------------------------------------------------------------------------------------
// ringx_attn_bwd_noalloc: ringx_attn_bwd with its per-row statistics (D and nl, two fp32 per query
// row) in a fixed, file-scope device array instead of a caller workspace.  Every GPU the library
// runs on holds its own copy of the array (RINGX_NOALLOC_MAX_ROWS * 8 bytes = 16 MiB) until the
// process ends.  In host code the
// array's name is only a host-side stand-in: its device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and only that address is ever passed to kernels.

namespace {

__device__ __align__(256) float scratch[2 * RINGX_NOALLOC_MAX_ROWS];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the device that runs `stream` (the current device for the null
// stream).  The first call for a device makes that device current for the lookup and restores the
// caller's device afterwards.
ringx_status scratch_address(hipStream_t stream, float** out) {
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return RINGX_E_HIP;
  int dev = cur;
  if (stream != nullptr && hipStreamGetDevice(stream, &dev) != hipSuccess) return RINGX_E_HIP;
  if (dev < 0 || dev >= kMaxDevices) return RINGX_E_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    if (dev != cur && hipSetDevice(dev) != hipSuccess) return RINGX_E_HIP;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur && hipSetDevice(cur) != hipSuccess) return RINGX_E_HIP;
    if (e != hipSuccess || p == nullptr) return RINGX_E_HIP;
    g_scratch_ptr[dev] = static_cast<float*>(p);
  }
  *out = g_scratch_ptr[dev];
  return RINGX_OK;
}

}  // namespace

extern "C" {

ringx_status ringx_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* out,
                                    const void* dout, const float* lse, float* dq, float* dk,
                                    float* dv, int64_t B, int64_t H, int64_t Nq, int64_t Nk,
                                    int64_t d, int64_t R, float scale, ringx_dtype dtype,
                                    int accumulate_dkv, hipStream_t stream) {
  if (!q || !k || !v || !out || !dout || !lse || !dq || !dk || !dv) return RINGX_E_NULLPTR;
  ringx_status st = check_dims(B, H, Nq, Nk, d, R, scale, dtype);
  if (st != RINGX_OK) return st;
  if (B * H * Nq > RINGX_NOALLOC_MAX_ROWS) return RINGX_E_SCRATCH;
  float* ws = nullptr;
  st = scratch_address(stream, &ws);
  if (st != RINGX_OK) return st;
  static_assert(RINGX_NOALLOC_MAX_ROWS % 64 == 0, "whole 256-byte blocks");
  return bwd_impl(q, k, v, out, dout, lse, dq, dk, dv, B, H, H, Nq, Nk, d, R, scale, dtype,
                  accumulate_dkv, ws, sizeof(float) * 2 * (size_t)RINGX_NOALLOC_MAX_ROWS, stream);
}

}  // extern "C"
