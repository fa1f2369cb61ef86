"""Grouped-query attention (Hkv K/V heads shared by H query heads in consecutive groups) against
the oracle run on explicitly repeated K/V heads: forward outputs equal, dK/dV equal the sum of the
repeated heads' gradients over each group."""

import math

import numpy as np
import pytest
import torch

import oracle
from paper_2507_16697_amd import inputs, ringx

from parity_util import (TOL_BF16_LSE, TOL_BF16_REL_RMS, TOL_F32, max_abs_err, rel_rms_err,
                         to_device, to_host_f64)

pytestmark = pytest.mark.gpu


def _case(seed, B, H, Hkv, Nq, Nk, d, store, std):
    q = inputs.make_iid(B, H, Nq, 1, d, seed=seed, std=std, store=store, with_do=True)
    kv = inputs.make_iid(B, Hkv, 1, Nk, d, seed=seed + 1000, std=std, store=store, with_do=False)
    t = {"q": q["q"], "do": q["do"], "k": kv["k"], "v": kv["v"]}
    x = {key: inputs.to_f64(val, store) for key, val in t.items()}
    return t, x


@pytest.mark.parametrize("store,d,H,Hkv", [("bf16", 128, 4, 2), ("bf16", 64, 6, 1),
                                           ("bf16", 128, 3, 3), ("fp32", 24, 4, 2)])
def test_gqa_forward_backward(store, d, H, Hkv):
    B, Nq, Nk, R = 2, 300, 1000, 3
    G = H // Hkv
    std = 2 ** -0.5 if d == 128 else 0.5
    t, x = _case(51, B, H, Hkv, Nq, Nk, d, store, std)
    g = {key: to_device(val, store) for key, val in t.items()}
    scale = float(np.float32(1 / math.sqrt(d)))
    out, lse = ringx.ringx_attn_fwd_gqa(g["q"], g["k"], g["v"], R, scale=scale)
    dq, dk, dv = ringx.ringx_attn_bwd_gqa(g["q"], g["k"], g["v"], out, g["do"], lse, R,
                                          scale=scale)
    torch.cuda.synchronize()
    kr, vr = np.repeat(x["k"], G, axis=1), np.repeat(x["v"], G, axis=1)
    ro, rl = oracle.attention(x["q"], kr, vr, scale)
    rq, rk, rv = oracle.attention_bwd(x["q"], kr, vr, ro, x["do"], rl, scale)
    rk = rk.reshape(B, Hkv, G, Nk, d).sum(axis=2)
    rv = rv.reshape(B, Hkv, G, Nk, d).sum(axis=2)
    got = {"out": to_host_f64(out), "dq": to_host_f64(dq), "dk": to_host_f64(dk),
           "dv": to_host_f64(dv)}
    ref = {"out": ro, "dq": rq, "dk": rk, "dv": rv}
    if store == "fp32":
        assert max_abs_err(to_host_f64(lse), rl) <= TOL_F32
        assert max_abs_err(got["out"], ro) <= TOL_F32
        for key in ("dq", "dk", "dv"):
            assert max_abs_err(got[key], ref[key]) <= 1e-4 * max(1.0, np.abs(ref[key]).max()), key
    else:
        assert max_abs_err(to_host_f64(lse), rl) <= TOL_BF16_LSE
        for key in ("out", "dq", "dk", "dv"):
            assert rel_rms_err(got[key], ref[key]) <= TOL_BF16_REL_RMS, key


def test_gqa_with_one_group_is_mha_bitwise():
    B, H, Nq, Nk, d, R = 1, 3, 257, 700, 128, 4
    t, _ = _case(52, B, H, H, Nq, Nk, d, "bf16", 2 ** -0.5)
    g = {key: to_device(val, "bf16") for key, val in t.items()}
    o1, l1 = ringx.ringx_attn_fwd_gqa(g["q"], g["k"], g["v"], R)
    o2, l2 = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R)
    a = ringx.ringx_attn_bwd_gqa(g["q"], g["k"], g["v"], o1, g["do"], l1, R)
    b = ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], o1, g["do"], l1, R)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    assert all(torch.equal(u, w) for u, w in zip(a, b))
