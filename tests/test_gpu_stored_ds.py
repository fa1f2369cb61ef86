"""The backward through stored dS (ringx_attn_bwd_ds, and its stages ringx_attn_bwd_dkdv_ds and
ringx_attn_bwd_dq_ds) against the fp64 oracle and against the recompute backward, through the C
ABI (needs an MI355X).

The stored path forms the same dS_ij as the recompute path (the dK/dV kernel is the same code
with stores added), so dK and dV must be bitwise those of ringx_attn_bwd, and dQ may differ from
the recompute dQ only by fp32 summation order and the occasional one-ulp bf16 rounding of a dS
that the two kernels form in a different order."""

import math

import numpy as np
import pytest
import torch

import oracle
from paper_2507_16697_amd import inputs, ringx

from parity_util import (TOL_BF16_LSE, TOL_BF16_REL_RMS, check_rows, max_abs_err, rel_rms_err,
                         to_device, to_host_f64)

pytestmark = pytest.mark.gpu

STD = 2 ** -0.5          # the ring-share workloads' input scale at d = 128
D = 128
# dQ of the two paths: relative RMS of the difference
TOL_PATHS = 1e-4


def _case(seed, B, H, Hkv, Nq, Nk):
    q = inputs.make_iid(B, H, Nq, 1, D, seed=seed, std=STD, store="bf16", do_std=STD,
                        with_do=True)
    kv = inputs.make_iid(B, Hkv, 1, Nk, D, seed=seed + 1000, std=STD, store="bf16",
                         with_do=False)
    t = {"q": q["q"], "do": q["do"], "k": kv["k"], "v": kv["v"]}
    x = {key: inputs.to_f64(val, "bf16") for key, val in t.items()}
    g = {key: to_device(val, "bf16") for key, val in t.items()}
    return x, g


def _rel_rms_diff(a, b):
    a, b = a.double(), b.double()
    return float((a - b).pow(2).mean().sqrt() / b.pow(2).mean().sqrt().clamp_min(1e-300))


# several query groups and key tiles with ragged tails, chunk boundaries off the tile grid,
# grouped-query and multi-query heads, one key per chunk (R = Nk), a single query
CASES = [(1, 2, 2, 300, 1000, 3), (1, 4, 2, 100, 700, 4), (2, 2, 1, 65, 129, 1),
         (1, 1, 1, 37, 300, 300), (1, 3, 3, 257, 2000, 5), (1, 2, 2, 1, 5, 2),
         (2, 4, 4, 130, 515, 2)]


@pytest.mark.parametrize("B,H,Hkv,Nq,Nk,R", CASES)
def test_stored_ds_backward_against_oracle(B, H, Hkv, Nq, Nk, R):
    G = H // Hkv
    x, g = _case(61, B, H, Hkv, Nq, Nk)
    scale = float(np.float32(1 / math.sqrt(D)))
    out, lse = ringx.ringx_attn_fwd_gqa(g["q"], g["k"], g["v"], R, scale=scale)
    dq, dk, dv = ringx.ringx_attn_bwd_ds(g["q"], g["k"], g["v"], out, g["do"], lse, R,
                                         scale=scale)
    rq_, rk_, rv_ = ringx.ringx_attn_bwd_gqa(g["q"], g["k"], g["v"], out, g["do"], lse, R,
                                             scale=scale)
    torch.cuda.synchronize()
    kr, vr = np.repeat(x["k"], G, axis=1), np.repeat(x["v"], G, axis=1)
    ro, rl = oracle.attention(x["q"], kr, vr, scale)
    rq, rk, rv = oracle.attention_bwd(x["q"], kr, vr, ro, x["do"], rl, scale)
    rk = rk.reshape(B, Hkv, G, Nk, D).sum(axis=2)
    rv = rv.reshape(B, Hkv, G, Nk, D).sum(axis=2)
    errs = dict(dq=rel_rms_err(to_host_f64(dq), rq), dk=rel_rms_err(to_host_f64(dk), rk),
                dv=rel_rms_err(to_host_f64(dv), rv))
    paths = _rel_rms_diff(dq, rq_)
    print(f"stored dS {(B, H, Hkv, Nq, Nk, R)}",
          " ".join(f"{k}={e:.3e}" for k, e in errs.items()), f"dq vs recompute {paths:.3e}",
          flush=True)
    assert max_abs_err(to_host_f64(lse), rl) <= TOL_BF16_LSE
    for key, e in errs.items():
        assert e <= TOL_BF16_REL_RMS, (key, e)
    assert torch.equal(dk, rk_) and torch.equal(dv, rv_)
    assert paths <= TOL_PATHS
    assert bool(torch.isfinite(dq).all())


def test_stored_ds_single_key():
    """Nk = 1: every P_ij is 1, so dQ = 0, dK = 0 and dV_0 = sum_i dO_i (closed forms; the zeros
    have no RMS scale, so they are checked in absolute terms against O(1) inputs)."""
    x, g = _case(65, 1, 2, 2, 77, 1)
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], 1)
    dq, dk, dv = ringx.ringx_attn_bwd_ds(g["q"], g["k"], g["v"], out, g["do"], lse, 1)
    torch.cuda.synchronize()
    assert float(torch.max(torch.abs(dq))) <= 1e-3
    assert float(torch.max(torch.abs(dk))) <= 1e-3
    assert rel_rms_err(to_host_f64(dv)[:, :, 0], x["do"].sum(axis=2)) <= TOL_BF16_REL_RMS


def test_stored_ds_stages_and_slabs():
    """ringx_attn_bwd_ds equals preprocess + per-slab ringx_attn_bwd_dkdv_ds / _dq_ds for any slab
    size, and each stage touches only its slab's rows (the others keep a sentinel)."""
    B, H, Hkv, Nq, Nk, R = 2, 6, 3, 200, 777, 3
    G = H // Hkv
    x, g = _case(62, B, H, Hkv, Nq, Nk)
    out, lse = ringx.ringx_attn_fwd_gqa(g["q"], g["k"], g["v"], R)
    dq0, dk0, dv0 = ringx.ringx_attn_bwd_ds(g["q"], g["k"], g["v"], out, g["do"], lse, R)
    delta = ringx.ringx_bwd_preprocess(out, g["do"], lse)
    for slab in (1, 2, 4, 6):
        nbytes = ringx.ringx_bwd_ds_bytes(H, Hkv, Nq, Nk, D, R, slab)
        ds = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        dq = torch.full((B, H, Nq, D), 7.0, device="cuda")
        dk = torch.full((B, Hkv, Nk, D), 7.0, device="cuda")
        dv = torch.full((B, Hkv, Nk, D), 7.0, device="cuda")
        for kv0 in range(0, B * Hkv, slab):
            n = min(slab, B * Hkv - kv0)
            ringx.ringx_attn_bwd_dkdv_ds(g["q"], g["k"], g["v"], g["do"], lse, delta, R, ds, kv0,
                                         n, dk=dk, dv=dv)
            ringx.ringx_attn_bwd_dq_ds(ds, g["k"], (B, H, Nq, D), R, kv0, n, dq=dq)
            torch.cuda.synchronize()
            # rows of the K/V heads after this slab (and their query heads) are still untouched
            done = kv0 + n
            assert bool((dk.view(B * Hkv, Nk, D)[done:] == 7.0).all())
            assert bool((dq.view(B * H, Nq, D)[done * G:] == 7.0).all())
        assert torch.equal(dk, dk0) and torch.equal(dv, dv0), slab
        assert _rel_rms_diff(dq, dq0) <= TOL_PATHS, slab
    # the full backward with a workspace that holds exactly one K/V head's dS (slabs of 1)
    ws = torch.empty(ringx.ringx_bwd_ds_workspace_bytes(B, H, Hkv, Nq, Nk, D, R, 1),
                     dtype=torch.uint8, device="cuda")
    dq1, dk1, dv1 = ringx.ringx_attn_bwd_ds(g["q"], g["k"], g["v"], out, g["do"], lse, R,
                                            workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(dk1, dk0) and torch.equal(dv1, dv0)
    assert _rel_rms_diff(dq1, dq0) <= TOL_PATHS


def test_stored_ds_accumulate_and_reproducible():
    B, H, Nq, Nk, R = 1, 2, 200, 600, 3
    _, g = _case(63, B, H, H, Nq, Nk)
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R)
    dq, dk, dv = ringx.ringx_attn_bwd_ds(g["q"], g["k"], g["v"], out, g["do"], lse, R)
    base_k, base_v = torch.randn_like(dk), torch.randn_like(dv)
    dk2, dv2 = base_k.clone(), base_v.clone()
    dq2, _, _ = ringx.ringx_attn_bwd_ds(g["q"], g["k"], g["v"], out, g["do"], lse, R, dk=dk2,
                                        dv=dv2, accumulate_dkv=True)
    torch.cuda.synchronize()
    assert torch.allclose(dk2 - base_k, dk, rtol=0, atol=1e-5)
    assert torch.allclose(dv2 - base_v, dv, rtol=0, atol=1e-5)
    assert torch.equal(dq2, dq)           # no atomics: bitwise reproducible


def test_stored_ds_scores_far_below_zero():
    """Scores shifted far below zero (lse about -200, where exp(-lse) overflows fp32) with chunk
    ends off the tile grid: the stored path stays finite and equals the recompute path."""
    B, H, Nq, Nk, R = 1, 2, 100, 333, 3
    x, g = _case(64, B, H, H, Nq, Nk)
    # q . k_j shifted by the same -c for every key: add a constant column pair to q and k
    q = g["q"].clone()
    k = g["k"].clone()
    q[..., 0] = 16.0
    k[..., 0] = -16.0 * 8        # scale 1/sqrt(128): shift of -16*128/sqrt(128) ~ -181 per score
    out, lse = ringx.ringx_attn_fwd(q, k, g["v"], R)
    torch.cuda.synchronize()
    assert float(lse.max()) < -100
    a = ringx.ringx_attn_bwd_ds(q, k, g["v"], out, g["do"], lse, R)
    b = ringx.ringx_attn_bwd(q, k, g["v"], out, g["do"], lse, R)
    torch.cuda.synchronize()
    for u in a:
        assert bool(torch.isfinite(u).all())
    assert torch.equal(a[1], b[1]) and torch.equal(a[2], b[2])
    assert _rel_rms_diff(a[0], b[0]) <= TOL_PATHS


@pytest.mark.slow
def test_stored_ds_ring8_full_size():
    """The 8-way ring share (Nq = 32768, Nk = 262144, R = 8) through the stored path with slabs of
    two heads: out/lse/dQ of 256 seeded rows of every head against the oracle, and dK/dV bitwise
    those of the recompute path (whose sampled keys the workload tests check against the
    oracle)."""
    w = inputs.WORKLOADS["ring8_nk262k_d128"]
    t = inputs.make_workload(w.name)
    g = {key: to_device(val, "bf16") for key, val in t.items()}
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], w.R, scale=w.scale)
    dq, dk, dv = ringx.ringx_attn_bwd_ds(g["q"], g["k"], g["v"], out, g["do"], lse, w.R,
                                         scale=w.scale, kv_per_slab=2)
    torch.cuda.synchronize()
    res = {"out": out, "lse": lse, "dq": dq}
    check_rows(w.name + " (stored dS)", w, t, res, heads=range(w.H))
    rq, rk, rv = ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], out, g["do"], lse, w.R,
                                      scale=w.scale)
    torch.cuda.synchronize()
    assert torch.equal(dk, rk) and torch.equal(dv, rv)
    diff = _rel_rms_diff(dq, rq)
    print(f"{w.name}: stored-dS dq vs recompute rel-rms {diff:.3e}", flush=True)
    assert diff <= TOL_PATHS
