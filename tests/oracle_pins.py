"""Pins of the fp64 oracle against things other than itself.

Each check takes the implementation under test as arguments and raises AssertionError on a
mismatch, so the same checks run against the oracle (tests/test_oracle_pins.py) and against
copies of it with a planted mistake (tests/test_oracle_mutants.py, which must fail them).

What pins what (arXiv 2507.16697, Sec. III-A):
  forward  Eq. (1) -- pure-Python brute force with the textbook (unshifted) softmax; torch fp64
           scaled_dot_product_attention and logsumexp; closed forms (Q = 0 gives the mean of V and
           lse = ln Nk; Nk = 1; d = 1, Nk = 2 is a logistic weight; one dominant key);
           permutation equivariance/invariance.
  merge    Eq. (5) -- chunked equals unchunked attention for every R; R = 1 is the identity;
           R = Nk rebuilds the softmax from single-key partials (v_j, s_ij); order of partials
           and grouping (tree merges) do not matter; a -inf partial contributes nothing.
  backward exact-softmax gradient -- central finite differences of L = sum(dO * O) through the
           brute-force forward; torch fp64 autograd; sum_j dV_j = sum_i dO_i and sum_j dK_j = 0;
           closed forms at Q = 0 and Nk = 1; chunk additivity.
"""

from __future__ import annotations

import math

import numpy as np
import torch


def brute_force_head(q, k, v, scale):
    """Pure-Python loops, textbook softmax exp(s)/sum exp(s) (no shift; tiny inputs only)."""
    q, k, v = (np.asarray(x, dtype=np.float64).tolist() for x in (q, k, v))
    O, L = [], []
    for qi in q:
        s = [scale * sum(a * b for a, b in zip(qi, kj)) for kj in k]
        w = [math.exp(x) for x in s]
        z = sum(w)
        O.append([sum(w[j] * v[j][c] for j in range(len(k))) / z for c in range(len(v[0]))])
        L.append(math.log(z))
    return np.array(O), np.array(L)


def _close(a, b, rtol, atol=0.0, what=""):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    err = np.max(np.abs(a - b)) if a.size else 0.0
    ref = max(np.max(np.abs(b)) if b.size else 0.0, 1e-300)
    assert err <= rtol * ref + atol, f"{what}: max err {err:.3e} (ref max {ref:.3e})"


TINY_SHAPES = [(nq, nk, d) for nq in (1, 2, 3, 17) for nk in (1, 2, 5, 31) for d in (1, 2, 3, 8)]


# ----------------------------------------------------------------------------------------------
# forward


def check_forward(head_attention, shapes=TINY_SHAPES, seed=0):
    rng = np.random.default_rng(seed)
    for (nq, nk, d) in shapes:
        q, k, v = (rng.standard_normal((n, d)) for n in (nq, nk, nk))
        scale = 1.0 / math.sqrt(d)
        O, L = head_attention(q, k, v, scale)
        Ob, Lb = brute_force_head(q, k, v, scale)
        _close(O, Ob, 1e-12, 1e-14, f"O vs brute force {nq,nk,d}")
        _close(L, Lb, 1e-12, 1e-14, f"lse vs brute force {nq,nk,d}")
        # library routines
        tq, tk, tv = (torch.from_numpy(x)[None, None] for x in (q, k, v))
        Ot = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=scale)[0, 0]
        Lt = torch.logsumexp(scale * (tq @ tk.transpose(-1, -2)), dim=-1)[0, 0]
        _close(O, Ot.numpy(), 1e-12, 1e-14, f"O vs torch sdpa {nq,nk,d}")
        _close(L, Lt.numpy(), 1e-12, 1e-14, f"lse vs torch logsumexp {nq,nk,d}")


def check_forward_closed_forms(head_attention, seed=1):
    rng = np.random.default_rng(seed)
    # Q = 0: every score is 0, the weights are uniform.
    nq, nk, d = 7, 13, 5
    k, v = rng.standard_normal((nk, d)), rng.standard_normal((nk, d))
    O, L = head_attention(np.zeros((nq, d)), k, v, 0.3)
    _close(O, np.broadcast_to(v.mean(axis=0), (nq, d)), 1e-14, 1e-15, "Q=0: O = mean V")
    _close(L, np.full(nq, math.log(nk)), 1e-15, 1e-15, "Q=0: lse = ln Nk")
    # Nk = 1: O = v_0 and lse = s_i0.
    q, k1, v1 = rng.standard_normal((nq, d)), rng.standard_normal((1, d)), rng.standard_normal((1, d))
    O, L = head_attention(q, k1, v1, 0.7)
    _close(O, np.broadcast_to(v1[0], (nq, d)), 1e-15, 1e-15, "Nk=1: O = v_0")
    _close(L, 0.7 * (q @ k1[0]), 1e-14, 1e-15, "Nk=1: lse = s_i0")
    # d = 1, Nk = 2: O_i = sigma(s1 - s2) v1 + sigma(s2 - s1) v2.
    q, k2, v2 = rng.standard_normal((nq, 1)), rng.standard_normal((2, 1)), rng.standard_normal((2, 1))
    O, L = head_attention(q, k2, v2, 1.0)
    s1, s2 = q[:, 0] * k2[0, 0], q[:, 0] * k2[1, 0]
    sig = lambda x: 1.0 / (1.0 + np.exp(-x))  # noqa: E731
    _close(O[:, 0], sig(s1 - s2) * v2[0, 0] + sig(s2 - s1) * v2[1, 0], 1e-14, 1e-15, "d=1,Nk=2")
    _close(L, np.logaddexp(s1, s2), 1e-14, 1e-15, "d=1,Nk=2 lse")
    # One dominant key: q_i = a e_0, k_j* = a e_0, every other key orthogonal to e_0.
    nk, d, a, jstar, scale = 50, 4, 3.0, 17, 0.5
    k = rng.standard_normal((nk, d))
    k[:, 0] = 0.0
    k[jstar] = 0.0
    k[jstar, 0] = a
    v = rng.standard_normal((nk, d))
    q = np.zeros((3, d))
    q[:, 0] = a
    O, L = head_attention(q, k, v, scale)
    c = scale * a * a
    rest = v.sum(axis=0) - v[jstar]
    _close(O, np.broadcast_to((math.exp(c) * v[jstar] + rest) / (math.exp(c) + nk - 1), (3, d)),
           1e-13, 1e-15, "dominant key O")
    _close(L, np.full(3, math.log(math.exp(c) + nk - 1)), 1e-14, 1e-15, "dominant key lse")


def check_forward_permutation(head_attention, seed=2):
    rng = np.random.default_rng(seed)
    nq, nk, d = 23, 41, 6
    q, k, v = rng.standard_normal((nq, d)), rng.standard_normal((nk, d)), rng.standard_normal((nk, d))
    O, L = head_attention(q, k, v, 0.4)
    pq = rng.permutation(nq)
    Op, Lp = head_attention(q[pq], k, v, 0.4)
    _close(Op, O[pq], 1e-14, 1e-15, "Q-row permutation")
    _close(Lp, L[pq], 1e-14, 1e-15, "Q-row permutation lse")
    pk = rng.permutation(nk)
    Ok, Lk = head_attention(q, k[pk], v[pk], 0.4)
    _close(Ok, O, 1e-13, 1e-15, "joint K/V permutation")
    _close(Lk, L, 1e-13, 1e-15, "joint K/V permutation lse")


# ----------------------------------------------------------------------------------------------
# Eq. (5) merge


def check_merge(head_partials, lse_merge, head_attention, seed=3):
    rng = np.random.default_rng(seed)
    nq, nk, d = 9, 37, 5
    q, k, v = rng.standard_normal((nq, d)), rng.standard_normal((nk, d)), rng.standard_normal((nk, d))
    scale = 0.45
    O, L = head_attention(q, k, v, scale)
    Ob, Lb = brute_force_head(q, k, v, scale)
    for R in (1, 2, 3, 7, 36, nk):
        po, pl = head_partials(q, k, v, scale, R)
        assert po.shape == (R, nq, d) and pl.shape == (R, nq), "partials shape"
        Om, Lm = lse_merge(po, pl)
        _close(Om, O, 1e-13, 1e-15, f"chunked = unchunked, R={R}")
        _close(Lm, L, 1e-13, 1e-15, f"chunked = unchunked lse, R={R}")
        _close(Om, Ob, 1e-12, 1e-15, f"chunked = brute force, R={R}")
        # order of the partials does not matter
        perm = rng.permutation(R)
        Op, Lp = lse_merge(po[perm], pl[perm])
        _close(Op, Om, 1e-14, 1e-15, f"partials permuted, R={R}")
        _close(Lp, Lm, 1e-14, 1e-15, f"partials permuted lse, R={R}")
    # R = 1 is the identity, bit for bit.
    po, pl = head_partials(q, k, v, scale, 1)
    O1, L1 = lse_merge(po, pl)
    assert np.array_equal(O1, po[0]) and np.array_equal(L1, pl[0]), "R=1 merge is not the identity"
    # R = Nk: each partial is a single key, loc_out = v_j and loc_lse = s_ij; merging them is the
    # softmax of Eq. (1).
    po, pl = head_partials(q, k, v, scale, nk)
    _close(po, np.broadcast_to(v[:, None, :], (nk, nq, d)), 1e-15, 1e-15, "single-key loc_out = v_j")
    _close(pl, (scale * (q @ k.T)).T, 1e-14, 1e-15, "single-key loc_lse = s_ij")
    # grouping: a tree of merges equals the flat merge (associativity the paper relies on)
    po, pl = head_partials(q, k, v, scale, 6)
    a = lse_merge(po[:2], pl[:2])
    b = lse_merge(po[2:5], pl[2:5])
    c = lse_merge(po[5:], pl[5:])
    Ot, Lt = lse_merge(np.stack([a[0], b[0], c[0]]), np.stack([a[1], b[1], c[1]]))
    _close(Ot, O, 1e-13, 1e-15, "tree merge")
    _close(Lt, L, 1e-13, 1e-15, "tree merge lse")
    # a partial with lse = -inf contributes nothing
    po2 = np.concatenate([po, rng.standard_normal((1, nq, d))])
    pl2 = np.concatenate([pl, np.full((1, nq), -np.inf)])
    Oi, Li = lse_merge(po2, pl2)
    _close(Oi, O, 1e-13, 1e-15, "-inf partial")
    _close(Li, L, 1e-13, 1e-15, "-inf partial lse")


# ----------------------------------------------------------------------------------------------
# backward


def _loss(q, k, v, do, scale):
    O, _ = brute_force_head(q, k, v, scale)
    return float(np.sum(do * O))


def check_backward_fd(head_attention_bwd, head_attention, head_bwd_preprocess, seed=4):
    rng = np.random.default_rng(seed)
    for (nq, nk, d) in [(3, 5, 3), (2, 4, 2), (4, 1, 2)]:
        q, k, v = rng.standard_normal((nq, d)), rng.standard_normal((nk, d)), rng.standard_normal((nk, d))
        do = rng.standard_normal((nq, d))
        scale = 0.6
        O, L = head_attention(q, k, v, scale)
        D = head_bwd_preprocess(O, do)
        dq, dk, dv = head_attention_bwd(q, k, v, do, L, D, scale)
        for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
            num = np.zeros_like(x)
            for idx in np.ndindex(*x.shape):
                h = 1e-6 * max(1.0, abs(x[idx]))
                xp, xm = x.copy(), x.copy()
                xp[idx] += h
                xm[idx] -= h
                args_p = {"q": q, "k": k, "v": v}
                args_m = {"q": q, "k": k, "v": v}
                args_p[name], args_m[name] = xp, xm
                num[idx] = (_loss(args_p["q"], args_p["k"], args_p["v"], do, scale)
                            - _loss(args_m["q"], args_m["k"], args_m["v"], do, scale)) / (2 * h)
            _close(g, num, 1e-6, 1e-9, f"finite differences d{name} {nq,nk,d}")


def check_backward_autograd(head_attention_bwd, head_attention, head_bwd_preprocess, seed=5):
    rng = np.random.default_rng(seed)
    for (nq, nk, d) in [(17, 31, 8), (1, 2, 3), (33, 7, 4)]:
        q, k, v = rng.standard_normal((nq, d)), rng.standard_normal((nk, d)), rng.standard_normal((nk, d))
        do = rng.standard_normal((nq, d))
        scale = 1.0 / math.sqrt(d)
        O, L = head_attention(q, k, v, scale)
        dq, dk, dv = head_attention_bwd(q, k, v, do, L, head_bwd_preprocess(O, do), scale)
        tq, tk, tv = (torch.from_numpy(x.copy())[None, None].requires_grad_(True) for x in (q, k, v))
        Ot = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=scale)
        Ot.backward(torch.from_numpy(do)[None, None])
        _close(dq, tq.grad[0, 0].numpy(), 1e-11, 1e-13, f"dq vs autograd {nq,nk,d}")
        _close(dk, tk.grad[0, 0].numpy(), 1e-11, 1e-13, f"dk vs autograd {nq,nk,d}")
        _close(dv, tv.grad[0, 0].numpy(), 1e-11, 1e-13, f"dv vs autograd {nq,nk,d}")


def check_backward_invariants(head_attention_bwd, head_attention, head_bwd_preprocess, seed=6):
    rng = np.random.default_rng(seed)
    nq, nk, d = 19, 29, 6
    q, k, v = rng.standard_normal((nq, d)), rng.standard_normal((nk, d)), rng.standard_normal((nk, d))
    do = rng.standard_normal((nq, d))
    scale = 0.35
    O, L = head_attention(q, k, v, scale)
    D = head_bwd_preprocess(O, do)
    dq, dk, dv = head_attention_bwd(q, k, v, do, L, D, scale)
    # V -> V + c shifts every O_i by c: sum_j dV_j = sum_i dO_i.
    _close(dv.sum(axis=0), do.sum(axis=0), 1e-13, 1e-13, "sum dV = sum dO")
    # K -> K + c leaves every softmax unchanged: sum_j dK_j = 0.
    _close(dk.sum(axis=0), np.zeros(d), 0.0, 1e-13 * np.abs(dk).sum(), "sum dK = 0")
    # Q = 0 closed forms.
    q0 = np.zeros((nq, d))
    O0, L0 = head_attention(q0, k, v, scale)
    dq0, dk0, dv0 = head_attention_bwd(q0, k, v, do, L0, head_bwd_preprocess(O0, do), scale)
    vbar = v.mean(axis=0)
    _close(dk0, np.zeros_like(dk0), 0.0, 1e-14, "Q=0: dK = 0")
    _close(dv0, np.broadcast_to(do.sum(axis=0) / nk, (nk, d)), 1e-13, 1e-15, "Q=0: dV")
    ref_dq = (scale / nk) * ((do @ (v - vbar).T) @ k)
    _close(dq0, ref_dq, 1e-13, 1e-15, "Q=0: dQ")
    # Nk = 1 closed forms.
    k1, v1 = k[:1], v[:1]
    O1, L1 = head_attention(q, k1, v1, scale)
    dq1, dk1, dv1 = head_attention_bwd(q, k1, v1, do, L1, head_bwd_preprocess(O1, do), scale)
    _close(dq1, np.zeros_like(dq1), 0.0, 1e-14, "Nk=1: dQ = 0")
    _close(dk1, np.zeros_like(dk1), 0.0, 1e-14, "Nk=1: dK = 0")
    _close(dv1, do.sum(axis=0, keepdims=True), 1e-14, 1e-15, "Nk=1: dV = sum dO")


def check_backward_chunks(head_attention_bwd, head_attention, head_bwd_preprocess, chunk_bounds,
                          seed=7):
    rng = np.random.default_rng(seed)
    nq, nk, d, R = 13, 40, 5, 3
    q, k, v = rng.standard_normal((nq, d)), rng.standard_normal((nk, d)), rng.standard_normal((nk, d))
    do = rng.standard_normal((nq, d))
    scale = 0.5
    O, L = head_attention(q, k, v, scale)
    D = head_bwd_preprocess(O, do)
    dq, dk, dv = head_attention_bwd(q, k, v, do, L, D, scale)
    dq_sum = np.zeros_like(dq)
    for r in range(R):
        lo, hi = chunk_bounds(nk, R, r)
        dq_r, dk_r, dv_r = head_attention_bwd(q, k[lo:hi], v[lo:hi], do, L, D, scale)
        dq_sum += dq_r
        _close(dk_r, dk[lo:hi], 1e-13, 1e-15, f"chunk {r} dK")
        _close(dv_r, dv[lo:hi], 1e-13, 1e-15, f"chunk {r} dV")
    _close(dq_sum, dq, 1e-13, 1e-15, "dQ = sum over chunks")
    # sampled rows give the same dQ rows as the full call
    rows = np.array([0, 5, nq - 1])
    dq_rows, _, _ = head_attention_bwd(q[rows], k, v, do[rows], L[rows], D[rows], scale)
    _close(dq_rows, dq[rows], 1e-14, 1e-15, "row-sampled dQ")


def check_chunk_bounds(chunk_bounds, max_nk=120):
    for nk in range(1, max_nk + 1):
        for R in range(1, nk + 1):
            prev_hi = 0
            for r in range(R):
                lo, hi = chunk_bounds(nk, R, r)
                assert lo == prev_hi, "chunks must tile the keys contiguously"
                assert hi > lo, "no chunk may be empty"
                assert hi - lo in (nk // R, -(-nk // R)), "chunk sizes differ by at most one"
                prev_hi = hi
            assert prev_hi == nk, "chunks must cover every key"
