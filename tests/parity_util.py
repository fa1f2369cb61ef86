"""Shared helpers of the GPU parity tests: moving seeded inputs to the device and comparing."""

from __future__ import annotations

import concurrent.futures
import os

import numpy as np
import torch

import oracle

from paper_2507_16697_amd import inputs

# Tolerances of the parity bar: fp32 max abs error 1e-5; bf16 max abs error relative to the
# reference RMS 2e-2 (per tensor); lse (bf16 path) max abs 2e-2 (an lse error e scales the
# softmax weights by exp(e)); chunk and index bookkeeping exact.
TOL_F32 = 1e-5
TOL_BF16_REL_RMS = 2e-2
TOL_BF16_LSE = 2e-2


def to_device(arr: np.ndarray, store: str, device="cuda") -> torch.Tensor:
    if store == "fp32":
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)
    t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(device)
    return t.view(torch.bfloat16)


def to_host_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel_rms_err(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref)))
    return float(np.max(np.abs(got - ref))) / max(rms, 1e-300)


def max_abs_err(got, ref) -> float:
    return float(np.max(np.abs(np.asarray(got, np.float64) - np.asarray(ref, np.float64))))


def random_case(seed, B, H, Nq, Nk, d, store="bf16", std=1.0, do_std=1.0):
    """Seeded i.i.d. inputs (storage form) and their exact fp64 values."""
    t = inputs.make_iid(B, H, Nq, Nk, d, seed=seed, std=std, store=store, do_std=do_std)
    exact = {key: inputs.to_f64(val, store) for key, val in t.items()}
    return t, exact


def host_threads() -> int:
    """Host threads for the oracle: the cores this process may run on, at most 16."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def pool_map(fn, items, workers=None):
    """fn over items on host threads (numpy releases the GIL in its matmuls and ufuncs), with the
    BLAS library held to one thread per call so that the threads do not oversubscribe the cores."""
    from threadpoolctl import threadpool_limits
    items = list(items)
    workers = min(workers or host_threads(), max(1, len(items)))
    with threadpool_limits(limits=1, user_api="blas"):
        with concurrent.futures.ThreadPoolExecutor(workers) as ex:
            return list(ex.map(fn, items))


def oracle_head_stats(q, k, v, do, scale, block=128):
    """The oracle's O, lse and D of every query row of one head ([Nq, d], [Nq], [Nq]).  Rows are
    independent in every formula, so blocks of rows go to host threads; each block is the
    oracle's own head_attention over all keys.  Prints a line at every quarter (long runs)."""
    nq = q.shape[0]
    spans = [(i, min(nq, i + block)) for i in range(0, nq, block)]
    marks = {len(spans) * j // 4 for j in range(1, 4)}

    def one(idx_sp):
        idx, (i0, i1) = idx_sp
        r = oracle.head_attention(q[i0:i1], k, v, scale, row_block=128)
        if idx in marks:
            print(f"  oracle head pass: block {idx} of {len(spans)}", flush=True)
        return r

    res = pool_map(one, enumerate(spans))
    o = np.concatenate([r[0] for r in res])
    lse = np.concatenate([r[1] for r in res])
    return o, lse, oracle.head_bwd_preprocess(o, do)


def oracle_key_grads(q, k, v, do, lse, D, scale, keys, block=2048):
    """The oracle's dK and dV of the keys `keys` of one head, summed over every query (the keys'
    gradients need only those keys against all queries, given every row's lse and D).  Query
    blocks go to host threads; their contributions are added in ascending block order."""
    nq = q.shape[0]
    ks, vs = k[keys], v[keys]
    spans = [(i, min(nq, i + block)) for i in range(0, nq, block)]
    parts = pool_map(lambda sp: oracle.head_attention_bwd(
        q[sp[0]:sp[1]], ks, vs, do[sp[0]:sp[1]], lse[sp[0]:sp[1]], D[sp[0]:sp[1]], scale)[1:],
        spans)
    dk = np.zeros_like(ks)
    dv = np.zeros_like(vs)
    for pk, pv in parts:
        dk += pk
        dv += pv
    return dk, dv


def sample_rows(Nq, n=256, seed=0):
    """At least n query rows: the edges of query tiles of 32, 64, 128 and 256 rows at both ends and
    in the middle, plus seeded random rows."""
    rows = {0, 1, 31, 32, 63, 64, 127, 128, 255, 256, Nq // 2 - 1, Nq // 2, Nq // 2 + 17,
            Nq - 257, Nq - 256, Nq - 129, Nq - 128, Nq - 65, Nq - 64, Nq - 33, Nq - 2, Nq - 1}
    rows = {r for r in rows if 0 <= r < Nq}
    rng = np.random.default_rng([seed, 1])
    while len(rows) < min(n, Nq):
        rows.add(int(rng.integers(0, Nq)))
    return np.array(sorted(rows))


def sample_keys(Nk, R, n=256, seed=0):
    """At least n keys: in every chunk its first and last keys, the edges of the 32-key wave blocks
    and 64/128-key tiles at both ends of the chunk and around one seeded tile edge inside it, plus
    seeded random keys."""
    rng = np.random.default_rng([seed, 2])
    keys = set()
    for r in range(R):
        lo, hi = oracle.chunk_bounds(Nk, R, r)
        cand = [lo, lo + 1, lo + 31, lo + 32, lo + 63, lo + 64, lo + 127, lo + 128,
                hi - 129, hi - 128, hi - 65, hi - 64, hi - 2, hi - 1]
        if hi - lo > 256:
            m = lo + 128 * int(rng.integers(1, (hi - lo) // 128))
            cand += [m - 1, m]
        keys.update(x for x in cand if lo <= x < hi)
    while len(keys) < min(n, Nk):
        keys.add(int(rng.integers(0, Nk)))
    return np.array(sorted(keys))


def err_stats(got, ref):
    """max |got - ref|, the reference RMS and their ratio (the bf16 parity measure)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    mx = float(np.max(np.abs(got - ref)))
    rms = float(np.sqrt(np.mean(ref * ref)))
    return mx, rms, mx / max(rms, 1e-300)


def check_rows(name, w, t, res, heads, with_bwd=True, n_rows=256):
    """out, lse (and dQ) of at least n_rows seeded rows of every head in `heads` against the oracle,
    row by row (a row's out, lse and dQ depend on that row and all keys).  Heads go to host
    threads."""
    out = res["out"]

    def one(h):
        rows = sample_rows(w.Nq, n_rows, seed=1000 * w.seed + h)
        q = inputs.to_f64(t["q"][0, h, rows], "bf16")
        k = inputs.to_f64(t["k"][0, h], "bf16")
        v = inputs.to_f64(t["v"][0, h], "bf16")
        o, l = oracle.head_attention(q, k, v, w.scale, row_block=64)
        r = {"rows": rows, "out": o, "lse": l}
        if with_bwd:
            do = inputs.to_f64(t["do"][0, h, rows], "bf16")
            D = oracle.head_bwd_preprocess(o, do)
            r["dq"] = oracle.head_attention_bwd(q, k, v, do, l, D, w.scale, row_block=64)[0]
        return r

    refs = pool_map(one, heads)
    keys = ("out", "dq") if with_bwd else ("out",)
    got = {key: [] for key in keys + ("lse",)}
    for h, r in zip(heads, refs):
        idx = torch.as_tensor(r["rows"], device=out.device)
        got["out"].append(to_host_f64(out[0, h].index_select(0, idx)))
        got["lse"].append(to_host_f64(res["lse"][0, h].index_select(0, idx)))
        if with_bwd:
            got["dq"].append(to_host_f64(res["dq"][0, h].index_select(0, idx)))
    errs = {}
    for key in keys:
        errs[key] = err_stats(np.concatenate(got[key]), np.concatenate([r[key] for r in refs]))
    lse_err = max_abs_err(np.concatenate(got["lse"]), np.concatenate([r["lse"] for r in refs]))
    nrows = sum(len(r["rows"]) for r in refs)
    print(f"{name}: {nrows} rows over heads {list(heads)}",
          " ".join(f"{k}: max_abs={m:.3e} rms={s:.3e} ratio={e:.3e}" for k, (m, s, e) in
                   errs.items()), f"lse max_abs={lse_err:.3e}", flush=True)
    assert lse_err <= TOL_BF16_LSE
    for key, (_, _, e) in errs.items():
        assert e <= TOL_BF16_REL_RMS, (key, e)


def rounding_bounds(x, kr, vr, ro, rl, scale):
    """Element-wise bounds on the error of the bf16 path that come from its roundings alone: P and
    dS are rounded to bf16 (relative 2^-8) before their contractions, the output is stored in
    bf16 (another 2^-8), and D is formed from that rounded output.  Propagated with absolute
    values through each contraction, from the fp64 quantities of the definition."""
    u = 2.0 ** -8
    q, do = x["q"], x["do"]
    P = np.exp(scale * (q @ np.swapaxes(kr, -1, -2)) - rl[..., None])
    D = np.sum(do * ro, axis=-1)
    dS = P * (do @ np.swapaxes(vr, -1, -2) - D[..., None])
    av = oracle.attention(q, kr, np.abs(vr), scale)[0]       # sum_j P_ij |v_j|
    b_out = u * (av + np.abs(ro))
    dD = np.sum(np.abs(do) * b_out, axis=-1)                   # from the rounded output
    E = u * np.abs(dS) + P * dD[..., None]                     # |error of dS_ij|
    b_dq = scale * (E @ np.abs(kr))
    b_dk = scale * (np.swapaxes(E, -1, -2) @ np.abs(q))
    b_dv = u * (np.swapaxes(P, -1, -2) @ np.abs(do))
    return b_out, b_dq, b_dk, b_dv
