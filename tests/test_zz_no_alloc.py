"""ringx_attn_bwd_noalloc (D in the library's fixed device array, no workspace argument) against
ringx_attn_bwd (caller workspace), through the C ABI, on the GPU.

Both run the same kernels on the same inputs, so their results must agree bit for bit: two calls
in a row, the second on a smaller problem (the array keeps the first call's contents), bf16 at
d = 128 and 64 and fp32, overwrite and accumulate modes, plus the oracle's parity bar on one case.
"""

import math

import numpy as np
import pytest
import torch

import oracle
from paper_2507_16697_amd import ringx

from parity_util import TOL_BF16_REL_RMS, TOL_F32, max_abs_err, random_case, rel_rms_err, \
    to_device, to_host_f64

pytestmark = pytest.mark.gpu


def _case(seed, B, H, Nq, Nk, d, store):
    std, do_std = ((0.5, 1.0) if d == 64 else (2 ** -0.5, 2 ** -0.5)) if store == "bf16" \
        else (1.0, 1.0)
    t, x = random_case(seed, B, H, Nq, Nk, d, store=store, std=std, do_std=do_std)
    g = {k: to_device(v, store) for k, v in t.items()}
    return g, x


def _both(g, R, scale, accumulate=False):
    """(reference via ringx_attn_bwd, result via ringx_attn_bwd_noalloc) on the same inputs."""
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    B, H, Nq, d = g["q"].shape
    Nk = g["k"].shape[2]
    f32 = dict(dtype=torch.float32, device="cuda")
    base_k = torch.randn((B, H, Nk, d), **f32) if accumulate else None
    base_v = torch.randn((B, H, Nk, d), **f32) if accumulate else None
    ref = ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], out, g["do"], lse, R, scale=scale,
                               dk=None if base_k is None else base_k.clone(),
                               dv=None if base_v is None else base_v.clone(),
                               accumulate_dkv=accumulate)
    dq = torch.full((B, H, Nq, d), float("nan"), **f32)
    dk = base_k.clone() if accumulate else torch.full((B, H, Nk, d), float("nan"), **f32)
    dv = base_v.clone() if accumulate else torch.full((B, H, Nk, d), float("nan"), **f32)
    got = ringx.ringx_attn_bwd_noalloc(g["q"], g["k"], g["v"], out, g["do"], lse, R, dq, dk, dv,
                                       scale=scale, accumulate_dkv=accumulate)
    torch.cuda.synchronize()
    return out, lse, ref, got


@pytest.mark.parametrize("store,d", [("bf16", 128), ("bf16", 64), ("fp32", 40)])
def test_noalloc_equals_workspace_backward_two_calls(store, d):
    # a larger problem, then a smaller one: the second call must not see the first call's D
    for i, (B, H, Nq, Nk, R) in enumerate([(2, 3, 700, 1500, 3), (1, 2, 130, 333, 2)]):
        g, _ = _case(60 + i, B, H, Nq, Nk, d, store)
        scale = float(np.float32(1 / math.sqrt(d)))
        _, _, ref, got = _both(g, R, scale)
        print(f"noalloc {store} d={d} call {i} shape B={B} H={H} Nq={Nq} Nk={Nk} R={R}",
              flush=True)
        for name, a, b in zip(("dq", "dk", "dv"), ref, got):
            assert torch.equal(a, b), (name, i)


def test_noalloc_accumulate_mode():
    g, _ = _case(63, 1, 2, 300, 640, 128, "bf16")
    _, _, ref, got = _both(g, 5, float(np.float32(1 / math.sqrt(128))), accumulate=True)
    for name, a, b in zip(("dq", "dk", "dv"), ref, got):
        assert torch.equal(a, b), name


@pytest.mark.parametrize("store,d", [("bf16", 128), ("fp32", 64)])
def test_noalloc_meets_the_oracle(store, d):
    B, H, Nq, Nk, R = 1, 2, 257, 900, 4
    g, x = _case(64, B, H, Nq, Nk, d, store)
    scale = float(np.float32(1 / math.sqrt(d)))
    out, lse, _, got = _both(g, R, scale)
    ref_o, ref_l = oracle.attention(x["q"], x["k"], x["v"], scale)
    oq, ok, ov = oracle.attention_bwd(x["q"], x["k"], x["v"], ref_o, x["do"], ref_l, scale)
    for name, a, b in zip(("dq", "dk", "dv"), got, (oq, ok, ov)):
        if store == "bf16":
            assert rel_rms_err(to_host_f64(a), b) <= TOL_BF16_REL_RMS, name
        else:
            assert max_abs_err(to_host_f64(a), b) <= TOL_F32, name


def test_noalloc_rejects_rows_beyond_the_array():
    g, _ = _case(65, 1, 1, 64, 128, 64, "bf16")
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], 1)
    f32 = dict(dtype=torch.float32, device="cuda")
    dq = torch.empty((1, 1, 64, 64), **f32)
    dk, dv = torch.empty((1, 1, 128, 64), **f32), torch.empty((1, 1, 128, 64), **f32)
    # a row count above the array, passed straight to the C entry point: rejected on the host
    # before any HIP call, so the small buffers are never touched
    st = ringx.lib().ringx_attn_bwd_noalloc(
        g["q"].data_ptr(), g["k"].data_ptr(), g["v"].data_ptr(), out.data_ptr(),
        g["do"].data_ptr(), lse.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), 1, 1,
        ringx.NOALLOC_MAX_ROWS + 1, 128, 64, 1, 0.125, ringx.RINGX_BF16, 0, None)
    assert st == 9 and "scratch" in ringx.ringx_status_str(st)
