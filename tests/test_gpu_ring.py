"""The ring-step path (one chunk per call, Eq. (5) into a running accumulator) and the ring driver
that overlaps chunk arrival with compute, against the fused entry points and the fp64 oracle."""

import math

import numpy as np
import pytest
import torch

import oracle
from oracle import attention_fp64 as oa
from paper_2507_16697_amd import inputs, ring, ringx

from parity_util import (TOL_BF16_LSE, TOL_BF16_REL_RMS, TOL_F32, check_rows, max_abs_err,
                         random_case, rel_rms_err, to_device, to_host_f64)

pytestmark = pytest.mark.gpu


def _chunks(t, bounds):
    return [t[:, :, lo:hi].contiguous() for lo, hi in bounds]


def _even_bounds(Nk, R):
    return [oa.chunk_bounds(Nk, R, r) for r in range(R)]


@pytest.mark.parametrize("d", [64, 128])
def test_ring_forward_matches_fused_and_oracle(d):
    B, H, Nq, Nk, R = 1, 2, 300, 1000, 3
    std = 0.5 if d == 64 else 2 ** -0.5
    t, x = random_case(41, B, H, Nq, Nk, d, store="bf16", std=std)
    g = {k: to_device(v, "bf16") for k, v in t.items()}
    scale = float(np.float32(1 / math.sqrt(d)))
    bounds = _even_bounds(Nk, R)
    out, lse = ring.ring_forward(g["q"], _chunks(g["k"], bounds), _chunks(g["v"], bounds),
                                 scale=scale)
    fo, fl = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    torch.cuda.synchronize()
    ref_o, ref_l = oracle.attention(x["q"], x["k"], x["v"], scale)
    assert rel_rms_err(to_host_f64(out), ref_o) <= TOL_BF16_REL_RMS
    assert max_abs_err(to_host_f64(lse), ref_l) <= TOL_BF16_LSE
    # same math as the fused path; P is rounded to bf16 against a different reference maximum
    # (per chunk here, running there), so the two agree to the parity bar, not bitwise
    assert rel_rms_err(to_host_f64(out), to_host_f64(fo)) <= TOL_BF16_REL_RMS
    assert max_abs_err(to_host_f64(lse), to_host_f64(fl)) <= 1e-4


def test_ring_forward_uneven_chunks_any_order():
    """Chunks of unequal length (down to one key), merged in two different orders."""
    B, H, Nq, Nk, d = 1, 2, 129, 700, 128
    t, x = random_case(42, B, H, Nq, Nk, d, store="bf16", std=2 ** -0.5)
    g = {k: to_device(v, "bf16") for k, v in t.items()}
    bounds = [(0, 100), (100, 101), (101, 163), (163, 700)]
    ks, vs = _chunks(g["k"], bounds), _chunks(g["v"], bounds)
    o1, l1 = ring.ring_forward(g["q"], ks, vs)
    o2, l2 = ring.ring_forward(g["q"], ks[::-1], vs[::-1])
    torch.cuda.synchronize()
    ref_o, ref_l = oracle.attention(x["q"], x["k"], x["v"], 1 / math.sqrt(d))
    for o, l in ((o1, l1), (o2, l2)):
        assert rel_rms_err(to_host_f64(o), ref_o) <= TOL_BF16_REL_RMS
        assert max_abs_err(to_host_f64(l), ref_l) <= TOL_BF16_LSE


def test_ring_forward_fp32_exact():
    B, H, Nq, Nk, d = 1, 2, 70, 257, 24
    t, x = random_case(43, B, H, Nq, Nk, d, store="fp32")
    g = {k: to_device(v, "fp32") for k, v in t.items()}
    bounds = _even_bounds(Nk, 4)
    scale = float(np.float32(1 / math.sqrt(d)))
    out, lse = ring.ring_forward(g["q"], _chunks(g["k"], bounds), _chunks(g["v"], bounds),
                                 scale=scale)
    torch.cuda.synchronize()
    ref_o, ref_l = oracle.attention(x["q"], x["k"], x["v"], scale)
    assert max_abs_err(to_host_f64(out), ref_o) <= TOL_F32
    assert max_abs_err(to_host_f64(lse), ref_l) <= TOL_F32


def test_fwd_step_first_ignores_accumulator_contents():
    B, H, Nq, Nk, d = 1, 1, 50, 90, 64
    t, _ = random_case(44, B, H, Nq, Nk, d, store="bf16", std=0.5)
    g = {k: to_device(v, "bf16") for k, v in t.items()}
    acc = torch.full((B, H, Nq, d), float("nan"), device="cuda")
    lacc = torch.full((B, H, Nq), float("nan"), device="cuda")
    ringx.ringx_attn_fwd_step(g["q"], g["k"], g["v"], acc, lacc, first=True)
    po, pl = ringx.ringx_attn_fwd_partials(g["q"], g["k"], g["v"], 1)
    torch.cuda.synchronize()
    assert torch.equal(acc, po[0]) and torch.equal(lacc, pl[0])


@pytest.mark.parametrize("d", [64, 128])
def test_ring_backward_matches_full_backward(d):
    """dK/dV of each chunk are bitwise the full backward's (same key tiles); dQ sums the chunks'
    contributions in fp32."""
    B, H, Nq, Nk, R = 1, 2, 200, 900, 3
    std, do_std = (0.5, 1.0) if d == 64 else (2 ** -0.5, 2 ** -0.5)
    t, x = random_case(45, B, H, Nq, Nk, d, store="bf16", std=std, do_std=do_std)
    g = {k: to_device(v, "bf16") for k, v in t.items()}
    scale = float(np.float32(1 / math.sqrt(d)))
    bounds = _even_bounds(Nk, R)
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    dq, dk, dv = ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], out, g["do"], lse, R, scale=scale)
    rq, rks, rvs = ring.ring_backward(g["q"], _chunks(g["k"], bounds), _chunks(g["v"], bounds),
                                      out, g["do"], lse, scale=scale)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat(rks, dim=2), dk) and torch.equal(torch.cat(rvs, dim=2), dv)
    assert rel_rms_err(to_host_f64(rq), to_host_f64(dq)) <= 1e-5
    ref_o, ref_l = oracle.attention(x["q"], x["k"], x["v"], scale)
    oq, _, _ = oracle.attention_bwd(x["q"], x["k"], x["v"], ref_o, x["do"], ref_l, scale)
    assert rel_rms_err(to_host_f64(rq), oq) <= TOL_BF16_REL_RMS


def test_bwd_step_accumulate_dkv():
    B, H, Nq, Nk, d = 1, 2, 64, 200, 128
    t, _ = random_case(46, B, H, Nq, Nk, d, store="bf16", std=2 ** -0.5)
    g = {k: to_device(v, "bf16") for k, v in t.items()}
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], 1)
    delta = ringx.ringx_bwd_preprocess(out, g["do"], lse)
    f32 = dict(dtype=torch.float32, device="cuda")
    dq, dk, dv = torch.empty((B, H, Nq, d), **f32), torch.empty((B, H, Nk, d), **f32), \
        torch.empty((B, H, Nk, d), **f32)
    ringx.ringx_attn_bwd_step(g["q"], g["k"], g["v"], g["do"], lse, delta, dq, dk, dv,
                              accumulate_dq=False)
    base_k, base_v = torch.randn_like(dk), torch.randn_like(dv)
    dk2, dv2, dq2 = base_k.clone(), base_v.clone(), dq.clone()
    ringx.ringx_attn_bwd_step(g["q"], g["k"], g["v"], g["do"], lse, delta, dq2, dk2, dv2,
                              accumulate_dq=True, accumulate_dkv=True)
    torch.cuda.synchronize()
    assert torch.allclose(dk2 - base_k, dk, rtol=0, atol=1e-5)
    assert torch.allclose(dv2 - base_v, dv, rtol=0, atol=1e-5)
    assert torch.allclose(dq2, 2 * dq, rtol=1e-6, atol=1e-6)


def test_ring_overlap_does_not_change_results():
    B, H, Nq, Nk, d = 1, 2, 150, 640, 128
    t, _ = random_case(47, B, H, Nq, Nk, d, store="bf16", std=2 ** -0.5)
    g = {k: to_device(v, "bf16") for k, v in t.items()}
    bounds = _even_bounds(Nk, 5)
    ks, vs = _chunks(g["k"], bounds), _chunks(g["v"], bounds)
    o1, l1 = ring.ring_forward(g["q"], ks, vs, overlap=True)
    o2, l2 = ring.ring_forward(g["q"], ks, vs, overlap=False)
    a = ring.ring_backward(g["q"], ks, vs, o1, g["do"], l1, overlap=True)
    b = ring.ring_backward(g["q"], ks, vs, o1, g["do"], l1, overlap=False)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2) and torch.equal(a[0], b[0])
    assert all(torch.equal(x, y) for x, y in zip(a[1] + a[2], b[1] + b[2]))


def test_ring_chunks_produced_just_before_the_call():
    """Chunks written by kernels on the current stream right before ring_forward/ring_backward
    (behind a long queue of other work there): the copy stream must wait for them, so the results
    equal those of chunks that were ready long before."""
    B, H, Nq, Nk, d = 1, 2, 150, 640, 128
    t, _ = random_case(48, B, H, Nq, Nk, d, store="bf16", std=2 ** -0.5)
    g = {k: to_device(v, "bf16") for k, v in t.items()}
    bounds = _even_bounds(Nk, 4)
    ref_ks, ref_vs = _chunks(g["k"], bounds), _chunks(g["v"], bounds)
    o_ref, l_ref = ring.ring_forward(g["q"], ref_ks, ref_vs)
    b_ref = ring.ring_backward(g["q"], ref_ks, ref_vs, o_ref, g["do"], l_ref)
    torch.cuda.synchronize()

    def busy():
        # a few milliseconds of fp32 work queued on the current stream
        x = torch.rand(4096, 4096, device="cuda")
        for _ in range(8):
            x = torch.sin(x @ x) * 0.01
        return x

    def produce(chunks):
        # each chunk comes out of an elementwise kernel on the current stream
        return [(c.float() * 1.0).to(torch.bfloat16) for c in chunks]

    busy()
    ks, vs = produce(ref_ks), produce(ref_vs)
    o, l = ring.ring_forward(g["q"], ks, vs)
    busy()
    ks2, vs2 = produce(ref_ks), produce(ref_vs)
    b = ring.ring_backward(g["q"], ks2, vs2, o_ref, g["do"], l_ref)
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref) and torch.equal(l, l_ref)
    assert torch.equal(b[0], b_ref[0])
    assert all(torch.equal(x, y) for x, y in zip(b[1] + b[2], b_ref[1] + b_ref[2]))


@pytest.mark.slow
def test_ring_steps_at_full_size():
    """The 8-way ring share (Nq=32768, Nk=262144 as 8 chunks of 32768) run step by step: the
    same result as the fused entry points (dK/dV bitwise)."""
    w = inputs.WORKLOADS["ring8_nk262k_d128"]
    t = inputs.make_workload(w.name)
    g = {k: to_device(v, "bf16") for k, v in t.items()}
    bounds = _even_bounds(w.Nk, w.R)
    ks, vs = _chunks(g["k"], bounds), _chunks(g["v"], bounds)
    out, lse = ring.ring_forward(g["q"], ks, vs, scale=w.scale)
    fo, fl = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], w.R, scale=w.scale)
    torch.cuda.synchronize()
    assert float(torch.max(torch.abs(lse - fl))) <= 1e-4
    check_rows("ring steps", w, t, {"out": out, "lse": lse}, heads=(0, 9), with_bwd=False)
    del ks, vs
    dq, dk, dv = ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], fo, g["do"], fl, w.R, scale=w.scale)
    rq, rks, rvs = ring.ring_backward(g["q"], _chunks(g["k"], bounds), _chunks(g["v"], bounds),
                                      fo, g["do"], fl, scale=w.scale)
    torch.cuda.synchronize()
    for r, (lo, hi) in enumerate(bounds):
        assert torch.equal(rks[r], dk[:, :, lo:hi]) and torch.equal(rvs[r], dv[:, :, lo:hi])
    assert float(torch.max(torch.abs(rq - dq))) <= 1e-4 * float(torch.max(torch.abs(dq)))
