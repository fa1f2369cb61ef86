"""Plain fp64 CPU oracle for ring-chunked, non-causal multi-head attention.

TEST INFRASTRUCTURE ONLY. This module is imported by the test suite, by the smoke check of the
graft entry point and by the CPU-baseline leg of the benchmark script -- nothing else.  The
product path (the HIP library and its Python binding) never imports, links or calls it, and it
shares no code with that path: no kernels, helpers, tables or constants.

What it computes (arXiv 2507.16697, Sec. III-A "RingX Parallel Attention"):

* exact softmax attention, Eq. (1), written with the log-sum-exp of Eqs. (2)-(4):
  s_ij = scale * q_i . k_j,  lse_i = log sum_j exp(s_ij),  O_i = sum_j exp(s_ij - lse_i) v_j;
* per-chunk partial results (loc_out_r, loc_lse_r) over key chunk r, and their exact merge by
  Eq. (5): lse_max = max_r loc_lse_r, num = sum_r loc_out_r exp(loc_lse_r - lse_max),
  den = sum_r exp(loc_lse_r - lse_max), O = num / den;
* the backward.  The paper only states its communication pattern (K/V chunk gradients computed
  per chunk and reduced, dQ accumulated over the N steps); the arithmetic is the exact-softmax
  gradient, evaluated with the merged (global) log-sum-exp so every chunk is independent.

Readings of points where the paper is silent or garbled (each is repeated where it is used):

R1  Eq. (2) as printed sums over the wrong index; it is read as
    A_s = sum_i exp(e_si - LSE_s) V_i, i.e. Eq. (1) with the log-sum-exp shift.
R2  Eqs. (1) and (4) carry no 1/sqrt(d); scores are scale * q.k with an explicit scale argument,
    and the log-sum-exp is taken of the scaled scores.
R3  Eq. (5) gives only num/den; the merged log-sum-exp is lse_max + log(den), which the backward
    needs and which lets merges chain.
R4  Natural logarithm throughout (Eq. (3) writes log/exp).
R5  Chunk r of R covers keys [floor(r*Nk/R), floor((r+1)*Nk/R)), 1 <= R <= Nk, so no chunk is empty.
R6  No causal mask, no dropout (the model is a bidirectional ViT).
R7  Backward: D_i = sum_c dO_ic O_ic (from this oracle's own O), P_ij = exp(s_ij - lse_i),
    dP_ij = dO_i . v_j, dS_ij = P_ij (dP_ij - D_i), dV_j = sum_i P_ij dO_i,
    dK_j = scale sum_i dS_ij q_i, dQ_i = scale sum_j dS_ij k_j.

Arithmetic: numpy float64.  numpy.matmul is the only library primitive; it evaluates the dot
products q_i . k_j, P @ V and the gradient contractions.  Query rows are independent in every
formula, so large heads are processed a block of rows at a time purely to bound memory; sums over
queries (dK, dV) add those blocks in ascending order.  Nothing is fused or reordered beyond that.

Layout of the batched helpers: [B, H, N, d], the scaled_dot_product_attention convention
(Sec. VI names RingX a drop-in for it).
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "chunk_bounds",
    "head_scores",
    "head_attention",
    "head_partials",
    "lse_merge",
    "head_bwd_preprocess",
    "head_attention_bwd",
    "attention",
    "attention_partials",
    "attention_chunked",
    "attention_bwd",
]

_ROW_BLOCK = 1024


def chunk_bounds(nk: int, R: int, r: int) -> tuple[int, int]:
    """Key range [lo, hi) of ring step r when Nk keys are split into R chunks (reading R5).

    Sec. III-A: each of the N participants holds a chunk of S/N keys; the paper does not say how
    a remainder is distributed.  lo = floor(r*Nk/R), hi = floor((r+1)*Nk/R).
    """
    nk, R, r = int(nk), int(R), int(r)
    if nk < 1 or R < 1 or R > nk:
        raise ValueError(f"need 1 <= R <= Nk, got R={R}, Nk={nk}")
    if r < 0 or r >= R:
        raise ValueError(f"chunk index {r} outside [0, {R})")
    return (r * nk) // R, ((r + 1) * nk) // R


def head_scores(q: np.ndarray, k: np.ndarray, scale: float) -> np.ndarray:
    """Eq. (4) with reading R2: s_ij = scale * sum_c q_ic k_jc, shape [Nq, Nk]."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    return float(scale) * (q @ k.T)


def head_attention(q, k, v, scale: float, row_block: int = _ROW_BLOCK):
    """Exact attention of one head, Eq. (1) via the log-sum-exp of Eqs. (2)-(3) (readings R1, R4).

    Two passes per query row, deliberately not an online softmax:
      m_i = max_j s_ij;  Z_i = sum_j exp(s_ij - m_i);  lse_i = m_i + log Z_i;
      O_i = sum_j exp(s_ij - lse_i) v_j.
    Returns (O [Nq, dv], lse [Nq]).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    nq = q.shape[0]
    out = np.empty((nq, v.shape[1]), dtype=np.float64)
    lse = np.empty(nq, dtype=np.float64)
    for i0 in range(0, nq, row_block):
        i1 = min(nq, i0 + row_block)
        s = head_scores(q[i0:i1], k, scale)
        m = s.max(axis=1)
        z = np.exp(s - m[:, None]).sum(axis=1)
        lse_blk = m + np.log(z)
        p = np.exp(s - lse_blk[:, None])
        out[i0:i1] = p @ v
        lse[i0:i1] = lse_blk
    return out, lse


def head_partials(q, k, v, scale: float, R: int, row_block: int = _ROW_BLOCK):
    """Per-chunk local results (loc_out_r, loc_lse_r) of Eq. (5) for one head.

    Chunk r is the key range of chunk_bounds(Nk, R, r); its local result is exact attention of
    the queries over those keys alone.  Returns (part_out [R, Nq, dv], part_lse [R, Nq]).
    """
    nk = np.asarray(k).shape[0]
    outs, lses = [], []
    for r in range(int(R)):
        lo, hi = chunk_bounds(nk, R, r)
        o_r, l_r = head_attention(q, np.asarray(k)[lo:hi], np.asarray(v)[lo:hi], scale, row_block)
        outs.append(o_r)
        lses.append(l_r)
    return np.stack(outs), np.stack(lses)


def lse_merge(part_out, part_lse):
    """Exact merge of R partial results, Eq. (5), with reading R3 for the merged log-sum-exp.

    part_out [R, ..., dv], part_lse [R, ...] (leading axis = chunk).
      lse_max = max_r loc_lse_r
      num     = sum_r loc_out_r * exp(loc_lse_r - lse_max)
      den     = sum_r exp(loc_lse_r - lse_max)
      O = num / den,  lse = lse_max + log(den).
    A partial with loc_lse = -inf contributes nothing.  At least one partial must be finite.
    """
    part_out = np.asarray(part_out, dtype=np.float64)
    part_lse = np.asarray(part_lse, dtype=np.float64)
    lse_max = part_lse.max(axis=0)
    if not np.all(np.isfinite(lse_max)):
        raise ValueError("every row needs at least one finite partial log-sum-exp")
    w = np.exp(part_lse - lse_max)
    den = w.sum(axis=0)
    num = (part_out * w[..., None]).sum(axis=0)
    return num / den[..., None], lse_max + np.log(den)


def head_bwd_preprocess(o, do) -> np.ndarray:
    """D_i = sum_c dO_ic O_ic for one head (reading R7)."""
    o = np.asarray(o, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    return (do * o).sum(axis=1)


def head_attention_bwd(q, k, v, do, lse, D, scale: float, row_block: int = _ROW_BLOCK):
    """Exact-softmax gradient of one head, with the merged log-sum-exp (reading R7).

      P_ij  = exp(s_ij - lse_i)           dP_ij = dO_i . v_j
      dS_ij = P_ij (dP_ij - D_i)
      dV_j  = sum_i P_ij dO_i   dK_j = scale sum_i dS_ij q_i   dQ_i = scale sum_j dS_ij k_j

    Every query row i depends only on (q_i, dO_i, lse_i, D_i) and all keys, and every key j only on
    (k_j, v_j) and all queries.  So passing a subset of queries yields their exact dQ (with dK, dV
    restricted to those queries' contributions), and passing a subset of keys yields those keys'
    exact dK, dV.  Returns (dq [Nq, d], dk [Nk, d], dv [Nk, dv]).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    lse = np.asarray(lse, dtype=np.float64)
    D = np.asarray(D, dtype=np.float64)
    scale = float(scale)
    nq = q.shape[0]
    dq = np.empty_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for i0 in range(0, nq, row_block):
        i1 = min(nq, i0 + row_block)
        s = head_scores(q[i0:i1], k, scale)
        p = np.exp(s - lse[i0:i1, None])
        dv += p.T @ do[i0:i1]
        dp = do[i0:i1] @ v.T
        ds = p * (dp - D[i0:i1, None])
        dk += scale * (ds.T @ q[i0:i1])
        dq[i0:i1] = scale * (ds @ k)
    return dq, dk, dv


# ----------------------------------------------------------------------------------------------
# Batched helpers over [B, H, N, d]


def _heads(x):
    x = np.asarray(x)
    if x.ndim != 4:
        raise ValueError(f"expected [B, H, N, d], got shape {x.shape}")
    return x


def attention(q, k, v, scale: float):
    """Eq. (1) for every (b, h).  Returns (O [B,H,Nq,dv], lse [B,H,Nq])."""
    q, k, v = _heads(q), _heads(k), _heads(v)
    B, H, nq, _ = q.shape
    out = np.empty((B, H, nq, v.shape[3]))
    lse = np.empty((B, H, nq))
    for b in range(B):
        for h in range(H):
            out[b, h], lse[b, h] = head_attention(q[b, h], k[b, h], v[b, h], scale)
    return out, lse


def attention_partials(q, k, v, scale: float, R: int):
    """Per-chunk local results for every (b, h): (part_out [R,B,H,Nq,dv], part_lse [R,B,H,Nq])."""
    q, k, v = _heads(q), _heads(k), _heads(v)
    B, H, nq, _ = q.shape
    part_out = np.empty((R, B, H, nq, v.shape[3]))
    part_lse = np.empty((R, B, H, nq))
    for b in range(B):
        for h in range(H):
            part_out[:, b, h], part_lse[:, b, h] = head_partials(q[b, h], k[b, h], v[b, h], scale, R)
    return part_out, part_lse


def attention_chunked(q, k, v, scale: float, R: int):
    """Ring-chunked attention: R per-chunk partials merged by Eq. (5).  Returns (O, lse)."""
    part_out, part_lse = attention_partials(q, k, v, scale, R)
    return lse_merge(part_out, part_lse)


def attention_bwd(q, k, v, o, do, lse, scale: float):
    """Backward for every (b, h) given this oracle's O and lse.  Returns (dq, dk, dv)."""
    q, k, v, o, do = _heads(q), _heads(k), _heads(v), _heads(o), _heads(do)
    lse = np.asarray(lse, dtype=np.float64)
    B, H = q.shape[:2]
    dq = np.empty(q.shape)
    dk = np.empty(k.shape)
    dv = np.empty(v.shape)
    for b in range(B):
        for h in range(H):
            D = head_bwd_preprocess(o[b, h], do[b, h])
            dq[b, h], dk[b, h], dv[b, h] = head_attention_bwd(
                q[b, h], k[b, h], v[b, h], do[b, h], lse[b, h], D, scale)
    return dq, dk, dv
