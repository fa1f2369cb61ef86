"""HIP path against the fp64 oracle, through the C ABI (needs an MI355X).

Sizes span several tiles with ragged tails (query tiles of 128, key tiles of 64/128 inside every
chunk, chunk boundaries that are not tile aligned), plus the degenerate cases (one query, one key,
R = 1, R = Nk).
"""

import math

import numpy as np
import pytest
import torch

import oracle
from oracle import attention_fp64 as oa
from paper_2507_16697_amd import inputs, ringx

from parity_util import (TOL_BF16_LSE, TOL_BF16_REL_RMS, TOL_F32, max_abs_err, random_case,
                         rel_rms_err, to_device, to_host_f64)

pytestmark = pytest.mark.gpu


def _dev(t, store):
    return {k: to_device(v, store) for k, v in t.items()}


def _report(name, **errs):
    print(name, " ".join(f"{k}={v:.3e}" for k, v in errs.items()), flush=True)


# ----------------------------------------------------------------------------------------------
# fp32 exactness path


def test_fp32_exact_workload():
    """1024 queries x 1024 keys, H=2, d=64, R=4, fp32 i.i.d. N(0,1) from seed 0."""
    w = inputs.WORKLOADS["exact_fp32_n1k"]
    t = inputs.make_workload(w.name, use_cache=False)
    x = {k: inputs.to_f64(v, "fp32") for k, v in t.items()}
    g = _dev(t, "fp32")
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], w.R, scale=w.scale)
    po, pl = ringx.ringx_attn_fwd_partials(g["q"], g["k"], g["v"], w.R, scale=w.scale)
    mo, ml = ringx.ringx_lse_merge(po, pl, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref_po, ref_pl = oracle.attention_partials(x["q"], x["k"], x["v"], w.scale, w.R)
    ref_o, ref_l = oa.lse_merge(ref_po, ref_pl)
    errs = dict(out=max_abs_err(to_host_f64(out), ref_o), lse=max_abs_err(to_host_f64(lse), ref_l),
                part_out=max_abs_err(to_host_f64(po), ref_po),
                part_lse=max_abs_err(to_host_f64(pl), ref_pl),
                merged_out=max_abs_err(to_host_f64(mo), ref_o),
                merged_lse=max_abs_err(to_host_f64(ml), ref_l))
    _report("exact_fp32_n1k", **errs)
    for k, e in errs.items():
        assert e <= TOL_F32, (k, e)


@pytest.mark.parametrize("B,H,Nq,Nk,d,R", [(1, 1, 1, 1, 1, 1), (2, 3, 37, 101, 3, 5),
                                           (1, 2, 130, 65, 128, 65), (1, 1, 300, 200, 100, 3),
                                           (2, 1, 129, 33, 64, 1)])
def test_fp32_shapes(B, H, Nq, Nk, d, R):
    t, x = random_case(7, B, H, Nq, Nk, d, store="fp32")
    g = _dev(t, "fp32")
    scale = float(np.float32(1 / math.sqrt(d)))
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    torch.cuda.synchronize()
    ref_o, ref_l = oracle.attention_chunked(x["q"], x["k"], x["v"], scale, R)
    assert max_abs_err(to_host_f64(out), ref_o) <= TOL_F32
    assert max_abs_err(to_host_f64(lse), ref_l) <= TOL_F32


def test_fp32_backward():
    B, H, Nq, Nk, d, R = 1, 2, 70, 90, 16, 3
    t, x = random_case(8, B, H, Nq, Nk, d, store="fp32")
    g = _dev(t, "fp32")
    scale = 0.25
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    dq, dk, dv = ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], out, g["do"], lse, R, scale=scale)
    torch.cuda.synchronize()
    ref_o, ref_l = oracle.attention(x["q"], x["k"], x["v"], scale)
    rq, rk, rv = oracle.attention_bwd(x["q"], x["k"], x["v"], ref_o, x["do"], ref_l, scale)
    for name, got, ref in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        e = max_abs_err(to_host_f64(got), ref)
        _report("fp32 bwd " + name, err=e)
        assert e <= TOL_F32, (name, e)


# ----------------------------------------------------------------------------------------------
# chunk bookkeeping: exact


def test_chunk_coverage_probe_fp32():
    """Q = 0, v_j = (j, 1): chunk r's local result is the mean key index of [lo_r, hi_r) and
    lse = ln(hi_r - lo_r), which identifies the key range exactly."""
    Nq, Nk, d = 5, 1000, 2
    for R in (1, 3, 7, 64):
        q = torch.zeros((1, 1, Nq, d), device="cuda")
        k = torch.randn((1, 1, Nk, d), device="cuda")
        v = torch.stack([torch.arange(Nk, dtype=torch.float32), torch.ones(Nk)], dim=-1)
        v = v.reshape(1, 1, Nk, d).cuda()
        po, pl = ringx.ringx_attn_fwd_partials(q, k, v, R, scale=1.0)
        po, pl = po.cpu().numpy(), pl.cpu().numpy()
        for r in range(R):
            n = int(round(math.exp(float(pl[r, 0, 0, 0]))))
            lo = int(round(float(po[r, 0, 0, 0, 0]) - (n - 1) / 2))
            assert (lo, lo + n) == oa.chunk_bounds(Nk, R, r), (R, r)
            assert np.all(po[r, 0, 0, :, 1] == 1.0)


@pytest.mark.parametrize("d", [64, 128])
def test_chunk_coverage_probe_bf16(d):
    """bf16 variant: with Q = 0 every probability is exactly 1, V carries j % 256 and j // 256
    (exact in bf16), so the fp32 partials give the sum of key indices of each chunk."""
    Nq, Nk = 3, 4000
    j = torch.arange(Nk, dtype=torch.float32)
    v = torch.zeros((1, 1, Nk, d))
    v[0, 0, :, 0] = j % 256
    v[0, 0, :, 1] = torch.div(j, 256, rounding_mode="floor")
    v[0, 0, :, 2] = 1.0
    v = v.to(torch.bfloat16).cuda()
    q = torch.zeros((1, 1, Nq, d), dtype=torch.bfloat16, device="cuda")
    k = torch.randn((1, 1, Nk, d), device="cuda").to(torch.bfloat16)
    for R in (1, 3, 8, 61):
        po, pl = ringx.ringx_attn_fwd_partials(q, k, v, R, scale=0.1)
        po, pl = po.double().cpu().numpy(), pl.double().cpu().numpy()
        for r in range(R):
            n = int(round(math.exp(pl[r, 0, 0, 0])))
            s = round(po[r, 0, 0, 0, 0] * n) + 256 * round(po[r, 0, 0, 0, 1] * n)
            lo = (s - n * (n - 1) // 2) // n
            assert (lo, lo + n) == oa.chunk_bounds(Nk, R, r), (d, R, r)
            assert np.allclose(po[r, 0, 0, :, 2], 1.0, rtol=0, atol=1e-6)


# ----------------------------------------------------------------------------------------------
# bf16 MFMA path


BF16_SHAPES = [
    # B, H, Nq, Nk, d, R
    (1, 2, 300, 1000, 64, 3),
    (2, 1, 129, 517, 128, 4),
    (1, 1, 1, 1, 64, 1),
    (1, 1, 1, 1, 128, 1),
    (1, 3, 200, 777, 128, 7),
    (1, 1, 257, 64, 64, 64),
    (1, 2, 128, 2048, 128, 8),
]


def _bf16_forward_case(B, H, Nq, Nk, d, R, seed=11, std=1.0):
    t, x = random_case(seed, B, H, Nq, Nk, d, store="bf16", std=std)
    g = _dev(t, "bf16")
    scale = float(np.float32(1 / math.sqrt(d)))
    return t, x, g, scale


@pytest.mark.parametrize("B,H,Nq,Nk,d,R", BF16_SHAPES)
def test_bf16_forward(B, H, Nq, Nk, d, R):
    t, x, g, scale = _bf16_forward_case(B, H, Nq, Nk, d, R)
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    po, pl = ringx.ringx_attn_fwd_partials(g["q"], g["k"], g["v"], R, scale=scale)
    torch.cuda.synchronize()
    ref_po, ref_pl = oracle.attention_partials(x["q"], x["k"], x["v"], scale, R)
    ref_o, ref_l = oa.lse_merge(ref_po, ref_pl)
    errs = dict(out=rel_rms_err(to_host_f64(out), ref_o), lse=max_abs_err(to_host_f64(lse), ref_l),
                part_out=rel_rms_err(to_host_f64(po), ref_po),
                part_lse=max_abs_err(to_host_f64(pl), ref_pl))
    _report(f"bf16 fwd {(B, H, Nq, Nk, d, R)}", **errs)
    assert errs["out"] <= TOL_BF16_REL_RMS and errs["part_out"] <= TOL_BF16_REL_RMS
    assert errs["lse"] <= TOL_BF16_LSE and errs["part_lse"] <= TOL_BF16_LSE


@pytest.mark.parametrize("d", [64, 128])
def test_bf16_fused_equals_partials_plus_merge(d):
    B, H, Nq, Nk, R = 1, 2, 200, 1500, 5
    t, x, g, scale = _bf16_forward_case(B, H, Nq, Nk, d, R, seed=12)
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    po, pl = ringx.ringx_attn_fwd_partials(g["q"], g["k"], g["v"], R, scale=scale)
    mo, ml = ringx.ringx_lse_merge(po, pl, out_dtype=torch.bfloat16)
    mo32, ml32 = ringx.ringx_lse_merge(po, pl, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref_o, ref_l = oa.lse_merge(*oracle.attention_partials(x["q"], x["k"], x["v"], scale, R))
    # the same partials, merged in the kernel's registers or by the standalone merge
    assert rel_rms_err(to_host_f64(mo), to_host_f64(out)) <= 2 * 2.0 ** -8 * 8
    assert max_abs_err(to_host_f64(ml), to_host_f64(lse)) <= 1e-5
    assert max_abs_err(to_host_f64(ml32), to_host_f64(ml)) == 0.0
    assert rel_rms_err(to_host_f64(mo32), ref_o) <= TOL_BF16_REL_RMS
    # standalone merge of exact partials (fp32 in, fp32 out) is fp32-accurate
    ref_po, ref_pl = oracle.attention_partials(x["q"], x["k"], x["v"], scale, R)
    po_t = torch.from_numpy(ref_po.astype(np.float32)).cuda()
    pl_t = torch.from_numpy(ref_pl.astype(np.float32)).cuda()
    eo, el = ringx.ringx_lse_merge(po_t, pl_t, out_dtype=torch.float32)
    ref_mo, ref_ml = oa.lse_merge(ref_po.astype(np.float32).astype(np.float64),
                                  ref_pl.astype(np.float32).astype(np.float64))
    assert max_abs_err(to_host_f64(eo), ref_mo) <= TOL_F32
    assert max_abs_err(to_host_f64(el), ref_ml) <= TOL_F32


def test_merge_ignores_minus_inf_partials():
    R, B, H, Nq, d = 3, 1, 1, 10, 64
    rng = np.random.default_rng(3)
    po = rng.standard_normal((R, B, H, Nq, d)).astype(np.float32)
    pl = rng.standard_normal((R, B, H, Nq)).astype(np.float32)
    pl[1] = -np.inf
    po[1] = 1e30
    eo, el = ringx.ringx_lse_merge(torch.from_numpy(po).cuda(), torch.from_numpy(pl).cuda(),
                                   out_dtype=torch.float32)
    ro, rl = oa.lse_merge(po.astype(np.float64), pl.astype(np.float64))
    assert max_abs_err(to_host_f64(eo), ro) <= TOL_F32
    assert max_abs_err(to_host_f64(el), rl) <= TOL_F32


@pytest.mark.parametrize("d", [4, 12, 64, 72, 128])
@pytest.mark.parametrize("R", [2, 7, 8, 9])
def test_merge_vector_paths(d, R):
    """Standalone Eq. (5) merge on every vector path: one or two 4-column quads per thread (two
    when d is a multiple of 8 and R < 8), fp32 and bf16 outputs, a row count that leaves a ragged
    last workgroup."""
    B, H, Nq = 1, 3, 37
    rng = np.random.default_rng(100 * d + R)
    po = rng.standard_normal((R, B, H, Nq, d)).astype(np.float32)
    pl = (3 * rng.standard_normal((R, B, H, Nq))).astype(np.float32)
    ro, rl = oa.lse_merge(po.astype(np.float64), pl.astype(np.float64))
    gpo, gpl = torch.from_numpy(po).cuda(), torch.from_numpy(pl).cuda()
    eo, el = ringx.ringx_lse_merge(gpo, gpl, out_dtype=torch.float32)
    assert max_abs_err(to_host_f64(eo), ro) <= TOL_F32
    assert max_abs_err(to_host_f64(el), rl) <= TOL_F32
    bo, bl = ringx.ringx_lse_merge(gpo, gpl, out_dtype=torch.bfloat16)
    got = to_host_f64(bo)
    # rounding to bf16 (nearest even) moves a value by at most half an ulp, 2^-9 of it; the fp32
    # sum before it may sit on the other side of a rounding boundary: one ulp
    assert np.all(np.abs(got - ro) <= 2.0 ** -8 * np.abs(ro) + TOL_F32)
    assert max_abs_err(to_host_f64(bl), rl) <= TOL_F32


def test_bf16_forward_independent_of_R():
    """The chunk count changes only the rounding: R = 1 and R = 8 both meet the oracle bar (two
    bf16 outputs may differ by one bf16 ulp from each other, so they are not compared directly)."""
    B, H, Nq, Nk, d = 1, 2, 150, 3000, 128
    t, x, g, scale = _bf16_forward_case(B, H, Nq, Nk, d, 1, seed=13, std=2 ** -0.5)
    ref_o, ref_l = oracle.attention(x["q"], x["k"], x["v"], scale)
    for R in (1, 2, 8, 3000):
        o, l = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
        torch.cuda.synchronize()
        assert rel_rms_err(to_host_f64(o), ref_o) <= TOL_BF16_REL_RMS, R
        assert max_abs_err(to_host_f64(l), ref_l) <= 1e-4, R


def test_bf16_forward_determinism_and_q_permutation():
    """Each query's arithmetic is independent of every other query: a permutation of the Q rows
    permutes out and lse bit for bit, and repeated runs are bitwise identical."""
    B, H, Nq, Nk, d, R = 1, 2, 256, 1200, 128, 3
    t, x, g, scale = _bf16_forward_case(B, H, Nq, Nk, d, R, seed=14)
    o1, l1 = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    o2, l2 = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    perm = torch.from_numpy(np.random.default_rng(5).permutation(Nq)).cuda()
    qp = g["q"][:, :, perm].contiguous()
    op, lp = ringx.ringx_attn_fwd(qp, g["k"], g["v"], R, scale=scale)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    assert torch.equal(op, o1[:, :, perm]) and torch.equal(lp, l1[:, :, perm])


# Input scales of the paper-shaped workloads: d=64 inputs ~0.5 N(0,1) with dO ~ N(0,1) (the
# single-shard 16k workload), d=128 inputs and dO ~ N(0,1)/sqrt(2) (the ring-share workloads).
def _workload_std(d):
    return (0.5, 1.0) if d == 64 else (2 ** -0.5, 2 ** -0.5)


@pytest.mark.parametrize("B,H,Nq,Nk,d,R", [(1, 2, 300, 1000, 64, 3), (1, 2, 100, 700, 128, 4),
                                           (2, 1, 65, 129, 128, 1), (1, 3, 257, 2000, 64, 5),
                                           (1, 1, 37, 300, 128, 300)])
def test_bf16_backward(B, H, Nq, Nk, d, R):
    std, do_std = _workload_std(d)
    t, x = random_case(21, B, H, Nq, Nk, d, store="bf16", std=std, do_std=do_std)
    g = _dev(t, "bf16")
    scale = float(np.float32(1 / math.sqrt(d)))
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    dq, dk, dv = ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], out, g["do"], lse, R, scale=scale)
    torch.cuda.synchronize()
    ref_o, ref_l = oracle.attention(x["q"], x["k"], x["v"], scale)
    rq, rk, rv = oracle.attention_bwd(x["q"], x["k"], x["v"], ref_o, x["do"], ref_l, scale)
    errs = dict(dq=rel_rms_err(to_host_f64(dq), rq), dk=rel_rms_err(to_host_f64(dk), rk),
                dv=rel_rms_err(to_host_f64(dv), rv))
    _report(f"bf16 bwd {(B, H, Nq, Nk, d, R)}", **errs)
    for k, e in errs.items():
        assert e <= TOL_BF16_REL_RMS, (k, e)


@pytest.mark.parametrize("d", [64, 128])
def test_bf16_backward_single_key(d):
    """Nk = 1: every P_ij is 1, so dQ = 0, dK = 0 and dV_0 = sum_i dO_i (closed forms; the exact
    zeros have no RMS scale, so they are checked in absolute terms against O(1) inputs)."""
    t, x = random_case(23, 1, 2, 77, 1, d, store="bf16", std=1.0)
    g = _dev(t, "bf16")
    scale = float(np.float32(1 / math.sqrt(d)))
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], 1, scale=scale)
    dq, dk, dv = ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], out, g["do"], lse, 1, scale=scale)
    torch.cuda.synchronize()
    assert float(torch.max(torch.abs(dq))) <= 1e-3
    assert float(torch.max(torch.abs(dk))) <= 1e-3
    assert rel_rms_err(to_host_f64(dv)[:, :, 0], x["do"].sum(axis=2)) <= TOL_BF16_REL_RMS


def test_bf16_backward_accumulate_and_invariants():
    B, H, Nq, Nk, d, R = 1, 2, 200, 600, 128, 3
    t, x = random_case(22, B, H, Nq, Nk, d, store="bf16", std=1.0)
    g = _dev(t, "bf16")
    scale = float(np.float32(1 / math.sqrt(d)))
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    dq, dk, dv = ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], out, g["do"], lse, R, scale=scale)
    base_k = torch.randn_like(dk)
    base_v = torch.randn_like(dv)
    dk2, dv2 = base_k.clone(), base_v.clone()
    ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], out, g["do"], lse, R, scale=scale, dk=dk2,
                         dv=dv2, accumulate_dkv=True)
    torch.cuda.synchronize()
    assert torch.allclose(dk2 - base_k, dk, rtol=0, atol=1e-5)
    assert torch.allclose(dv2 - base_v, dv, rtol=0, atol=1e-5)
    # no atomics anywhere: every gradient is bitwise reproducible
    dq3, dk3, dv3 = ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], out, g["do"], lse, R, scale=scale)
    torch.cuda.synchronize()
    assert torch.equal(dq3, dq) and torch.equal(dk3, dk) and torch.equal(dv3, dv)
    # sum_j dV_j = sum_i dO_i and sum_j dK_j = 0, per (b, h)
    sdv = dv.double().sum(dim=2)
    sdo = g["do"].double().sum(dim=2)
    assert torch.max(torch.abs(sdv - sdo)) <= 2e-2 * torch.max(torch.abs(dv.double()).sum(dim=2))
    sdk = dk.double().sum(dim=2)
    assert torch.max(torch.abs(sdk)) <= 2e-2 * torch.max(torch.abs(dk.double()).sum(dim=2))


@pytest.mark.parametrize("dtype,d", [(torch.bfloat16, 128), (torch.bfloat16, 64), (torch.float32, 24)])
def test_backward_stages_compose(dtype, d):
    """ringx_attn_bwd is exactly ringx_bwd_preprocess + ringx_attn_bwd_dkdv + ringx_attn_bwd_dq."""
    B, H, Nq, Nk, R = 1, 2, 130, 333, 3
    store = "bf16" if dtype == torch.bfloat16 else "fp32"
    t, x = random_case(24, B, H, Nq, Nk, d, store=store, std=0.6)
    g = _dev(t, store)
    scale = float(np.float32(1 / math.sqrt(d)))
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    dq, dk, dv = ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], out, g["do"], lse, R, scale=scale)
    delta = ringx.ringx_bwd_preprocess(out, g["do"], lse)
    dk2, dv2 = ringx.ringx_attn_bwd_dkdv(g["q"], g["k"], g["v"], g["do"], lse, delta, R, scale=scale)
    dq2 = ringx.ringx_attn_bwd_dq(g["q"], g["k"], g["v"], g["do"], lse, delta, R, scale=scale)
    torch.cuda.synchronize()
    assert torch.equal(dq, dq2) and torch.equal(dk, dk2) and torch.equal(dv, dv2)
    ref_d = (to_host_f64(out) * x["do"]).sum(axis=-1)
    assert max_abs_err(to_host_f64(delta[0]), ref_d) <= 1e-4 * max(1.0, float(np.abs(ref_d).max()))
    # the second row: the lse in the base-2 exponent form, -lse * log2(e), to fp32 rounding
    ref_nl = -to_host_f64(lse) / math.log(2.0)
    assert max_abs_err(to_host_f64(delta[1]), ref_nl) <= 2.0 ** -22 * max(1.0, float(np.abs(ref_nl).max()))


@pytest.mark.parametrize("H,Hkv", [(3, 3), (6, 3)])
def test_dkdv_launch_groups_match_per_head_calls(H, Hkv):
    """At a key length where ringx_attn_bwd_dkdv splits its launch into groups of K/V heads (two
    per launch at 262,144 keys in 8 chunks, the last group ragged), the gradients equal those of
    one call per K/V head (each a single launch) bitwise: the groups only move pointers."""
    B, Nq, Nk, d, R = 1, 128, 262144, 128, 8
    G = H // Hkv
    q = inputs.make_iid(B, H, Nq, 1, d, seed=31, std=2 ** -0.5, store="bf16", do_std=2 ** -0.5)
    kv = inputs.make_iid(B, Hkv, 1, Nk, d, seed=32, std=2 ** -0.5, store="bf16", with_do=False)
    g = {"q": to_device(q["q"], "bf16"), "do": to_device(q["do"], "bf16"),
         "k": to_device(kv["k"], "bf16"), "v": to_device(kv["v"], "bf16")}
    out, lse = ringx.ringx_attn_fwd_gqa(g["q"], g["k"], g["v"], R)
    delta = ringx.ringx_bwd_preprocess(out, g["do"], lse)
    if Hkv == H:
        dk, dv = ringx.ringx_attn_bwd_dkdv(g["q"], g["k"], g["v"], g["do"], lse, delta, R)
    else:
        _, dk, dv = ringx.ringx_attn_bwd_gqa(g["q"], g["k"], g["v"], out, g["do"], lse, R)
    for m in range(Hkv):
        hs = slice(m * G, (m + 1) * G)
        dl = delta[:, :, hs].contiguous()
        qs, dos, ls = g["q"][:, hs], g["do"][:, hs], lse[:, hs]
        ks, vs = g["k"][:, m:m + 1], g["v"][:, m:m + 1]
        if G == 1:
            dk1, dv1 = ringx.ringx_attn_bwd_dkdv(qs, ks, vs, dos, ls, dl, R)
        else:
            _, dk1, dv1 = ringx.ringx_attn_bwd_gqa(qs, ks, vs, out[:, hs], dos, ls, R)
        torch.cuda.synchronize()
        assert torch.equal(dk1[:, 0], dk[:, m]) and torch.equal(dv1[:, 0], dv[:, m]), m


def test_errors_leave_outputs_untouched():
    q = torch.randn((1, 1, 16, 64), device="cuda").to(torch.bfloat16)
    k = torch.randn((1, 1, 8, 64), device="cuda").to(torch.bfloat16)
    out = torch.full((1, 1, 16, 64), 7.0, device="cuda").to(torch.bfloat16)
    lse = torch.full((1, 1, 16), 3.0, device="cuda")
    with pytest.raises(ringx.RingxError):
        ringx.ringx_attn_fwd(q, k, k.clone(), 9, out=out, lse=lse)    # R > Nk
    with pytest.raises(ringx.RingxError):
        ringx.ringx_attn_fwd(q, k, k.clone(), 1, scale=float("nan"), out=out, lse=lse)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0) and torch.all(lse == 3.0)


def test_mismatched_buffers_are_refused_before_launch():
    """Every wrapper checks each tensor against the sizes the kernels derive from q and k; a
    mismatch raises on the host and nothing is launched (the outputs keep their contents)."""
    dev = "cuda"
    bf = dict(dtype=torch.bfloat16, device=dev)
    f32 = dict(dtype=torch.float32, device=dev)
    q = torch.randn((1, 2, 16, 64), **bf)
    k = torch.randn((1, 2, 40, 64), **bf)
    v = torch.randn((1, 2, 40, 64), **bf)
    out = torch.full((1, 2, 16, 64), 7.0, **bf)
    lse = torch.full((1, 2, 16), 3.0, **f32)
    with pytest.raises(ValueError, match="v: shape"):
        ringx.ringx_attn_fwd(q, k, v[:, :, :39].contiguous(), 2, out=out, lse=lse)
    with pytest.raises(ValueError, match="lse: shape"):
        ringx.ringx_attn_fwd(q, k, v, 2, out=out, lse=torch.zeros((1, 2, 15), **f32))
    with pytest.raises(TypeError, match="out: dtype"):
        ringx.ringx_attn_fwd(q, k, v, 2, out=torch.zeros((1, 2, 16, 64), **f32), lse=lse)
    do = torch.randn_like(q)
    with pytest.raises(TypeError, match="dk: dtype"):
        ringx.ringx_attn_bwd(q, k, v, out, do, lse, 2, dk=torch.zeros((1, 2, 40, 64), **bf))
    with pytest.raises(ValueError, match="dv: shape"):
        ringx.ringx_attn_bwd(q, k, v, out, do, lse, 2, dv=torch.zeros((1, 2, 39, 64), **f32))
    delta = torch.zeros((2, 1, 2, 16), **f32)
    with pytest.raises(ValueError, match="delta: shape"):
        ringx.ringx_attn_bwd_dq(q, k, v, do, lse, delta[0].contiguous(), 2)
    with pytest.raises(TypeError, match="out_acc: dtype"):
        ringx.ringx_attn_fwd_step(q, k, v, torch.zeros((1, 2, 16, 64), **bf), lse, True)
    with pytest.raises(ValueError, match="dk: shape"):
        ringx.ringx_attn_bwd_gqa(q, k[:, :1].contiguous(), v[:, :1].contiguous(), out, do, lse, 2,
                                 dk=torch.zeros((1, 2, 40, 64), **f32))
    with pytest.raises(ValueError, match="part_lse: shape"):
        ringx.ringx_lse_merge(torch.zeros((2, 1, 2, 16, 64), **f32), torch.zeros((2, 1, 2, 8), **f32))
    field = torch.zeros((2, 8, 8, 8), **f32)
    with pytest.raises(ValueError, match="tokens: shape"):
        ringx.ringx_tt_tokenize(field, 2, 1, (4, 4, 4), 1, tokens=torch.zeros((63, 2), **f32))
    torch.cuda.synchronize()
    assert torch.all(out == 7.0) and torch.all(lse == 3.0)
