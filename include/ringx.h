/*
 * ringx.h -- C ABI of libringx: ring-chunked, non-causal multi-head attention on one MI355X
 * (gfx950), i.e. one GPU's share of RingX sequence parallelism (arXiv 2507.16697, Sec. III-A).
 *
 * One query shard attends to the full key/value sequence, which arrives as R ring-step chunks.
 * Each chunk yields a partial output loc_out_r and log-sum-exp loc_lse_r (Sec. III-A, text after
 * Eq. (5)); the partials are merged exactly by Eq. (5).  The backward recomputes the softmax from
 * the merged log-sum-exp.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  Layout     Tensors are contiguous [B, H, N, d] (d fastest), the scaled_dot_product_attention
 *             convention (Sec. VI calls RingX a drop-in for it).  lse and part_lse are fp32
 *             [.., B, H, Nq], natural logarithm of sum_j exp(scale * q_i . k_j).
 *  Semantics  Non-causal, no mask, no dropout.  Scores are scale * q . k (scale is an explicit
 *             argument; the paper's Eqs. (1)/(4) print no scale).
 *  dtype      RINGX_BF16: q, k, v, out, dout are bf16; products on bf16 MFMA with fp32
 *             accumulation; softmax statistics, merge, lse and gradients in fp32.
 *             RINGX_FP32: every tensor fp32, fp32 arithmetic throughout.
 *  Chunks     Chunk r of R covers keys [floor(r*Nk/R), floor((r+1)*Nk/R)); 1 <= R <= Nk.
 *  Memory     Every tensor pointer is caller-owned device memory, 16-byte aligned; outputs must
 *             not overlap inputs.  The library never allocates, frees or keeps a pointer after
 *             returning.  Scratch memory needed by the backward is passed in by the caller, except
 *             for ringx_attn_bwd_noalloc, which uses a fixed device array of the library's own.
 *  Ordering   Work is enqueued on `stream` (0 = the null stream) and the call returns without
 *             synchronising.  Apart from that fixed array there is no global mutable state; calls
 *             are thread-safe.
 *  Errors     Arguments are checked on the host before any HIP call.  On an error status nothing
 *             has been enqueued and no output has been written.  RINGX_E_HIP reports a launch
 *             failure (hipGetLastError) after validation passed; outputs are then undefined.
 *             No C++ exception crosses the ABI.
 */
#ifndef RINGX_H
#define RINGX_H

#include <stddef.h>
#include <stdint.h>

/* hipStream_t: from the HIP runtime when hipcc compiles the includer; otherwise the same opaque
   handle type, so that plain C and C++ callers need no HIP headers (a repeated identical typedef
   is valid in C11 and C++). */
#ifdef __HIPCC__
#include <hip/hip_runtime_api.h>
#else
typedef struct ihipStream_t* hipStream_t;
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* In C++ both enums are given int as their fixed underlying type, so that any int a C caller
   passes (the ABI type of both) is a valid value of the enum on the library's side. */
#ifdef __cplusplus
#define RINGX_ENUM_BASE : int
#else
#define RINGX_ENUM_BASE
#endif

typedef enum ringx_status RINGX_ENUM_BASE {
  RINGX_OK = 0,
  RINGX_E_NULLPTR = 1,     /* a required pointer is NULL                                     */
  RINGX_E_SHAPE = 2,       /* B, H, Nq, Nk < 1, a size overflows, or scale not finite and > 0 */
                           /* (also Nk > 2^31 or Nq > 2^31 - 128 per head)                   */
  RINGX_E_CHUNKS = 3,      /* R < 1 or R > Nk, or chunk index out of range                   */
  RINGX_E_UNSUPPORTED = 4, /* dtype or head dim not supported (bf16: d in {64,128}; fp32: 1..128) */
  RINGX_E_ALIGN = 5,       /* a tensor pointer is not 16-byte aligned                        */
  RINGX_E_WORKSPACE = 6,   /* backward workspace missing or smaller than required            */
  RINGX_E_HIP = 7,         /* a HIP launch failed                                            */
  RINGX_E_ALIAS = 8,       /* an output overlaps an input                                    */
  RINGX_E_SCRATCH = 9      /* B*H*Nq above RINGX_NOALLOC_MAX_ROWS (ringx_attn_bwd_noalloc)   */
} ringx_status;

typedef enum ringx_dtype RINGX_ENUM_BASE { RINGX_FP32 = 0, RINGX_BF16 = 1 } ringx_dtype;

/*
 * Ring-chunked forward with the Eq. (5) merge fused (Sec. III-A, Eqs. (1)-(5)).
 *   q [B,H,Nq,d], k [B,H,Nk,d], v [B,H,Nk,d] (dtype) -- inputs.
 *   out [B,H,Nq,d] (dtype)  -- softmax(scale q k^T) v over all Nk keys.
 *   lse [B,H,Nq] (fp32)     -- merged log-sum-exp, lse_max + log(den) of Eq. (5); the backward's
 *                              input.
 *   R -- number of ring-step chunks; each chunk's (loc_out, loc_lse) is formed and merged in
 *   registers, in chunk order.
 */
ringx_status ringx_attn_fwd(const void* q, const void* k, const void* v, void* out, float* lse,
                            int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t d, int64_t R,
                            float scale, ringx_dtype dtype, hipStream_t stream);

/*
 * Per-chunk forward without the merge: the R local results of Sec. III-A (loc_out_i, loc_lse_i
 * "on the sequence chunk S_i"), as another GPU of a RingX_a group would produce them.
 *   part_out [R,B,H,Nq,d] (fp32), part_lse [R,B,H,Nq] (fp32, natural log).
 */
ringx_status ringx_attn_fwd_partials(const void* q, const void* k, const void* v, float* part_out,
                                     float* part_lse, int64_t B, int64_t H, int64_t Nq, int64_t Nk,
                                     int64_t d, int64_t R, float scale, ringx_dtype dtype,
                                     hipStream_t stream);

/*
 * Standalone N-way merge of partial results, Eq. (5) (Sec. III-A: allreduce of lse_max, then the
 * reduction of num and den; num/den is the attention):
 *   lse_max = max_r part_lse[r];  w_r = exp(part_lse[r] - lse_max);
 *   out = sum_r w_r part_out[r] / sum_r w_r;  lse = lse_max + log(sum_r w_r).
 *   part_out [R,B,H,Nq,d] fp32, part_lse [R,B,H,Nq] fp32 -- inputs (a partial with lse = -inf
 *   contributes nothing; every row needs one finite partial).
 *   out [B,H,Nq,d] in out_dtype (bf16 or fp32), lse [B,H,Nq] fp32.
 */
ringx_status ringx_lse_merge(const float* part_out, const float* part_lse, void* out, float* lse,
                             int64_t R, int64_t B, int64_t H, int64_t Nq, int64_t d,
                             ringx_dtype out_dtype, hipStream_t stream);

/*
 * Recompute-based backward with the merged lse (Sec. III-A, "Communication scheme": the K/V
 * chunk gradients are computed per chunk, the gradient of Q accumulates over all N steps).
 * Softmax gradient:
 *   D_i = sum_c dout_ic out_ic;  P_ij = exp(scale q_i.k_j - lse_i);  dP_ij = dout_i . v_j;
 *   dS_ij = P_ij (dP_ij - D_i);  dV_j = sum_i P_ij dout_i;  dK_j = scale sum_i dS_ij q_i;
 *   dQ_i = scale sum_j dS_ij k_j.
 * Runs ringx_bwd_preprocess, ringx_attn_bwd_dkdv and ringx_attn_bwd_dq in that order.
 *   q, k, v, out, dout (dtype), lse [B,H,Nq] fp32 (from ringx_attn_fwd or ringx_lse_merge).
 *   dq [B,H,Nq,d] fp32 -- overwritten; accumulated over every chunk in fp32 registers.
 *   dk, dv [B,H,Nk,d] fp32 -- overwritten, or added to when accumulate_dkv != 0 (as dK/dV
 *   travelling around a ring collect the contributions of other query shards).
 *   workspace/workspace_bytes -- device scratch of at least ringx_bwd_workspace_bytes(...) bytes,
 *   16-byte aligned, owned by the caller; it receives the per-row statistics of
 *   ringx_bwd_preprocess (D and nl); contents on entry are ignored.
 *   R -- chunk count: no key tile straddles a chunk boundary; results do not depend on R beyond
 *   rounding.  dq, dk and dv are bitwise reproducible.
 */
ringx_status ringx_attn_bwd(const void* q, const void* k, const void* v, const void* out,
                            const void* dout, const float* lse, float* dq, float* dk, float* dv,
                            int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t d, int64_t R,
                            float scale, ringx_dtype dtype, int accumulate_dkv, void* workspace,
                            size_t workspace_bytes, hipStream_t stream);

/*
 * ringx_attn_bwd without a workspace argument, for callers that cannot allocate device memory
 * (code under HIP graph capture, allocation-free serving loops, harnesses that forbid hipMalloc).
 * The caller still passes every input and output, exactly as for ringx_attn_bwd; the per-row
 * statistics (D and nl, two fp32 per query row) go to a fixed device array that the library holds
 * on every GPU it runs on (RINGX_NOALLOC_MAX_ROWS * 8 bytes = 16 MiB, kept until the process ends).
 * Nothing is allocated or freed.
 *   RINGX_E_SCRATCH if B * H * Nq > RINGX_NOALLOC_MAX_ROWS (checked before any HIP call).
 *   RINGX_E_HIP if the array's device address cannot be looked up (first call on a device).
 * All calls on one GPU share that GPU's array and nothing in it survives from one call to the
 * next (the statistics are written in full before they are read), but calls that overlap in time on one GPU -- on
 * different streams, or from several threads without ordering -- race on it and give undefined
 * results; order them (one stream, or events).  Results are bitwise those of ringx_attn_bwd.
 */
#define RINGX_NOALLOC_MAX_ROWS 2097152
ringx_status ringx_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* out,
                                    const void* dout, const float* lse, float* dq, float* dk,
                                    float* dv, int64_t B, int64_t H, int64_t Nq, int64_t Nk,
                                    int64_t d, int64_t R, float scale, ringx_dtype dtype,
                                    int accumulate_dkv, hipStream_t stream);

/* Backward preprocess: the per-row statistics of the recompute backward, delta [2,B,H,Nq] fp32:
 *   delta[0] = D_i = sum_c dout_ic out_ic;
 *   delta[1] = nl_i = -lse_i * log2(e), the row's log-sum-exp as the offset of the base-2
 *              exponent the kernels form, P_ij = 2^(scale log2(e) q_i.k_j + nl_i) (stored once so
 *              that no kernel multiplies it per score element).
 *   out, dout [B,H,Nq,d] in dtype (d as for the forward); lse [B,H,Nq] fp32 (natural log, from
 *   ringx_attn_fwd or ringx_lse_merge).  delta is caller-owned and must not overlap the inputs. */
ringx_status ringx_bwd_preprocess(const void* out, const void* dout, const float* lse,
                                  float* delta, int64_t B, int64_t H, int64_t Nq, int64_t d,
                                  ringx_dtype dtype, hipStream_t stream);

/* Gradients of the keys and values (the part a RingX group reduces across ranks): for every key
 * j of every chunk, dV_j = sum_i P_ij dout_i and dK_j = scale sum_i dS_ij q_i over all Nq queries,
 * using lse and delta [2,B,H,Nq] from ringx_bwd_preprocess (with the same lse).  dk, dv [B,H,Nk,d]
 * fp32, overwritten or added to (accumulate_dkv != 0). */
ringx_status ringx_attn_bwd_dkdv(const void* q, const void* k, const void* v, const void* dout,
                                 const float* lse, const float* delta, float* dk, float* dv,
                                 int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t d,
                                 int64_t R, float scale, ringx_dtype dtype, int accumulate_dkv,
                                 hipStream_t stream);

/* Gradient of the queries (the part each rank accumulates over all ring steps):
 * dQ_i = scale sum_j dS_ij k_j over the keys of every chunk, with lse and delta [2,B,H,Nq] as for
 * ringx_attn_bwd_dkdv.  dq [B,H,Nq,d] fp32, overwritten. */
ringx_status ringx_attn_bwd_dq(const void* q, const void* k, const void* v, const void* dout,
                               const float* lse, const float* delta, float* dq, int64_t B,
                               int64_t H, int64_t Nq, int64_t Nk, int64_t d, int64_t R,
                               float scale, ringx_dtype dtype, hipStream_t stream);

/*
 * Backward through stored dS, bf16 with d = 128 (RINGX_E_UNSUPPORTED otherwise).  The same
 * gradients as the recompute backward above (Sec. III-A: K/V chunk gradients per chunk, dQ
 * accumulated over every chunk), computed in a different order: the dK/dV stage also writes every
 * -dS_ij it forms (the bf16 operand of its dK product) to a caller-owned buffer, and the dQ stage
 * forms dQ_i = scale sum_j dS_ij k_j from it instead of recomputing P and dP.  That is 7U of
 * matrix products per backward instead of 9U (U = 2 B H Nq Nk d), for 2 B H Nq Nk bytes of dS
 * written and read once.  Both stages work on a slab of consecutive K/V heads
 * [kv_begin, kv_begin + kv_count) of the B * Hkv (batch-major; K/V head m serves query heads
 * m G .. m G + G - 1, G = H / Hkv), so that the stored dS of one slab fits the buffer.  The layout
 * of the buffer is private to the library: only ringx_attn_bwd_dq_ds reads it.
 *
 * ringx_bwd_ds_bytes: bytes of stored dS for kv_count K/V heads (about 2 G Nq Nk each); 0 if the
 * arguments are invalid.  Host only.
 */
size_t ringx_bwd_ds_bytes(int64_t H, int64_t Hkv, int64_t Nq, int64_t Nk, int64_t d, int64_t R,
                          int64_t kv_count);

/* dK/dV of the slab's K/V heads, as ringx_attn_bwd_dkdv (with Hkv K/V heads) restricted to them:
 * rows of dk, dv [B,Hkv,Nk,d] fp32 outside the slab are not touched.  delta [2,B,H,Nq] from
 * ringx_bwd_preprocess.  ds/ds_bytes: at least ringx_bwd_ds_bytes(H, Hkv, Nq, Nk, d, R, kv_count)
 * bytes, 16-byte aligned; receives the slab's dS (previous contents ignored).
 * RINGX_E_SHAPE if kv_begin < 0, kv_count < 1 or the slab passes B * Hkv; RINGX_E_WORKSPACE if
 * ds is NULL or too small. */
ringx_status ringx_attn_bwd_dkdv_ds(const void* q, const void* k, const void* v, const void* dout,
                                    const float* lse, const float* delta, float* dk, float* dv,
                                    void* ds, size_t ds_bytes, int64_t B, int64_t H, int64_t Hkv,
                                    int64_t Nq, int64_t Nk, int64_t d, int64_t R, float scale,
                                    ringx_dtype dtype, int accumulate_dkv, int64_t kv_begin,
                                    int64_t kv_count, hipStream_t stream);

/* dQ of the query heads of the slab's K/V heads from ds as written by ringx_attn_bwd_dkdv_ds with
 * the same shapes and slab: dq [B,H,Nq,d] fp32, those rows overwritten, the others not touched.
 * k [B,Hkv,Nk,d] bf16.  Errors as ringx_attn_bwd_dkdv_ds. */
ringx_status ringx_attn_bwd_dq_ds(const void* ds, size_t ds_bytes, const void* k, float* dq,
                                  int64_t B, int64_t H, int64_t Hkv, int64_t Nq, int64_t Nk,
                                  int64_t d, int64_t R, float scale, ringx_dtype dtype,
                                  int64_t kv_begin, int64_t kv_count, hipStream_t stream);

/* The whole backward through stored dS: ringx_bwd_preprocess, then ringx_attn_bwd_dkdv_ds and
 * ringx_attn_bwd_dq_ds slab by slab, with as many K/V heads per slab as the workspace holds.
 * Arguments as ringx_attn_bwd_gqa (Hkv = H for multi-head attention); the workspace must hold at
 * least ringx_bwd_ds_workspace_bytes(B, H, Hkv, Nq, Nk, d, R, 1) bytes (the per-row statistics
 * and one K/V head's dS); more lets a slab hold more heads.  dq, dk, dv agree with ringx_attn_bwd
 * to rounding (dk, dv bitwise). */
ringx_status ringx_attn_bwd_ds(const void* q, const void* k, const void* v, const void* out,
                               const void* dout, const float* lse, float* dq, float* dk,
                               float* dv, int64_t B, int64_t H, int64_t Hkv, int64_t Nq,
                               int64_t Nk, int64_t d, int64_t R, float scale, ringx_dtype dtype,
                               int accumulate_dkv, void* workspace, size_t workspace_bytes,
                               hipStream_t stream);

/* Workspace of ringx_attn_bwd_ds for slabs of kv_per_slab K/V heads (0 if invalid).  Host only. */
size_t ringx_bwd_ds_workspace_bytes(int64_t B, int64_t H, int64_t Hkv, int64_t Nq, int64_t Nk,
                                    int64_t d, int64_t R, int64_t kv_per_slab);

/*
 * One ring step of the forward (Sec. III-A: at every step a GPU holds one K/V chunk of S/N tokens,
 * computes its local result, and the results are merged by Eq. (5); "Communication and
 * computation overlap": the next chunk arrives in a second buffer meanwhile).  Computes the local
 * result (loc_out, loc_lse) of q against the one chunk k, v [B,H,Nk,d] (Nk = the chunk's length)
 * and folds it into the running result by Eq. (5):
 *   M = max(lse_acc, loc_lse);  a = exp(lse_acc - M);  b = exp(loc_lse - M);
 *   out_acc <- (a out_acc + b loc_out) / (a + b);  lse_acc <- M + log(a + b).
 *   out_acc [B,H,Nq,d] fp32, lse_acc [B,H,Nq] fp32 -- caller-owned, read and written in place
 *   (normalised output and natural-log lse of every chunk merged so far).
 *   first != 0: the accumulator holds nothing yet; it is overwritten (its contents are ignored).
 * After the last step, ringx_lse_merge with R = 1 turns (out_acc, lse_acc) into the output dtype.
 * Steps on one accumulator must be ordered (same stream or synchronised); the chunks may come in
 * any order (the merge is exact up to rounding).
 */
ringx_status ringx_attn_fwd_step(const void* q, const void* k, const void* v, float* out_acc,
                                 float* lse_acc, int64_t B, int64_t H, int64_t Nq, int64_t Nk,
                                 int64_t d, float scale, ringx_dtype dtype, int first,
                                 hipStream_t stream);

/*
 * One ring step of the backward (Sec. III-A, "Communication scheme": the K/V chunk's gradients
 * are computed at the step that holds the chunk and sent back to its owner; dQ accumulates over
 * the N steps).  With lse and delta of the whole sequence (the merged lse, and delta [2,B,H,Nq]
 * from ringx_bwd_preprocess with it), for the one chunk k, v [B,H,Nk,d]:
 *   dk, dv [B,H,Nk,d] fp32 -- the chunk's gradients, overwritten or added to
 *   (accumulate_dkv != 0);
 *   dq_acc [B,H,Nq,d] fp32 -- the chunk's contribution to dQ, added to the running sum
 *   (accumulate_dq != 0) or overwriting it (the first step).
 * Steps that touch one dq_acc must be ordered.
 */
ringx_status ringx_attn_bwd_step(const void* q, const void* k, const void* v, const void* dout,
                                 const float* lse, const float* delta, float* dq_acc, float* dk,
                                 float* dv, int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t d,
                                 float scale, ringx_dtype dtype, int accumulate_dq,
                                 int accumulate_dkv, hipStream_t stream);

/*
 * Grouped-query attention (Sec. VI lists RingX as compatible with GQA): Hkv K/V heads serve the H
 * query heads, query head h reading K/V head h / (H / Hkv) (consecutive groups of G = H / Hkv;
 * Hkv = H is ringx_attn_fwd, Hkv = 1 is multi-query attention).
 *   q, out [B,H,Nq,d], k, v [B,Hkv,Nk,d] (dtype); lse [B,H,Nq] fp32.  Everything else as
 *   ringx_attn_fwd.  RINGX_E_SHAPE if Hkv < 1 or Hkv does not divide H.
 */
ringx_status ringx_attn_fwd_gqa(const void* q, const void* k, const void* v, void* out,
                                float* lse, int64_t B, int64_t H, int64_t Hkv, int64_t Nq,
                                int64_t Nk, int64_t d, int64_t R, float scale, ringx_dtype dtype,
                                hipStream_t stream);

/*
 * Backward of ringx_attn_fwd_gqa.  dq [B,H,Nq,d] fp32; dk, dv [B,Hkv,Nk,d] fp32 hold the sum of
 * the gradients over the G query heads of each group (overwritten, or added to when
 * accumulate_dkv != 0).  Workspace as ringx_attn_bwd (ringx_bwd_workspace_bytes with H query
 * heads).  Everything else as ringx_attn_bwd.
 */
ringx_status ringx_attn_bwd_gqa(const void* q, const void* k, const void* v, const void* out,
                                const void* dout, const float* lse, float* dq, float* dk,
                                float* dv, int64_t B, int64_t H, int64_t Hkv, int64_t Nq,
                                int64_t Nk, int64_t d, int64_t R, float scale, ringx_dtype dtype,
                                int accumulate_dkv, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/*
 * One fidelity mode of the Turbulence Transformer's multi-fidelity input (Sec. III-B: the
 * subdomain selection C_i, the Gaussian filter F_i of size k_i^3, the model's patches; Table III
 * pairs filter k with mode-size ratio D/D_i), as tokens for the attention above:
 *   field  [C, D, H, W] fp32 (x fastest) -- input, caller-owned device memory.
 *   subdomain: D/ratio x H/ratio x W/ratio cells centred at (cz, cy, cx), taken periodically
 *   (cells cz - (D/ratio)/2 ... along z, and likewise);
 *   filter: weights w_i = exp(-(i - (k-1)/2)^2 / (2 sigma^2)) / sum, i < k (k <= 32), applied as
 *   w_i w_j w_l over each k^3 window with stride k;
 *   tokens [L, C p^3] in out_dtype (fp32 or bf16, round to nearest even) with
 *   L = (D/(ratio k p)) (H/(ratio k p)) (W/(ratio k p)); token (pz, py, px) at px + Px (py + Py pz),
 *   feature ((c p + iz) p + iy) p + ix.
 * RINGX_E_SHAPE unless ratio divides D, H, W and k p divides each subdomain extent, the centre lies
 * in the field and sigma is finite and > 0; RINGX_E_UNSUPPORTED for k > 32.
 */
ringx_status ringx_tt_tokenize(const float* field, void* tokens, int64_t C, int64_t D, int64_t H,
                               int64_t W, int64_t k, int64_t ratio, int64_t cz, int64_t cy,
                               int64_t cx, int64_t p, float sigma, ringx_dtype out_dtype,
                               hipStream_t stream);

/* Bytes of backward workspace for these arguments (0 if the arguments are invalid).  Host only. */
size_t ringx_bwd_workspace_bytes(int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t d,
                                 int64_t R, ringx_dtype dtype);

/* Key range [*lo, *hi) of chunk r (lo = floor(r*Nk/R)).  Host only; no HIP call. */
ringx_status ringx_chunk_bounds(int64_t Nk, int64_t R, int64_t r, int64_t* lo, int64_t* hi);

/* Static, NUL-terminated description of a status code (any int: values that are not a
   ringx_status give "unknown status"). */
const char* ringx_status_str(int status);

#ifdef __cplusplus
}
#endif
#endif /* RINGX_H */
