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
            assert max_abs_err(got[key], ref[key]) <= TOL_F32, key
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


def _gqa_full_inputs(nq=None):
    """The headline workload with its first H/4 K/V heads shared by groups of 4 query heads (the
    grouped-query configuration bench.py times); optionally only the first `nq` query rows."""
    w = inputs.WORKLOADS["ring8_nk262k_d128"]
    t = inputs.make_workload(w.name)
    hkv = t["q"].shape[1] // 4
    q, do = (t["q"], t["do"]) if nq is None else (t["q"][:, :, :nq], t["do"][:, :, :nq])
    return w, {"q": q, "do": do, "k": t["k"][:, :hkv], "v": t["v"][:, :hkv]}


def _gqa_run(w, g):
    out, lse = ringx.ringx_attn_fwd_gqa(g["q"], g["k"], g["v"], w.R, scale=w.scale)
    dq, dk, dv = ringx.ringx_attn_bwd_gqa(g["q"], g["k"], g["v"], out, g["do"], lse, w.R,
                                          scale=w.scale)
    torch.cuda.synchronize()
    return {"out": out, "lse": lse, "dq": dq, "dk": dk, "dv": dv}


@pytest.mark.slow
def test_gqa_ring8_full_size():
    """H=16 query heads over Hkv=4 K/V heads at the full 8-way ring share (Nq=32768, Nk=262144,
    R=8, d=128): sampled query rows of heads in every group against the oracle (out, lse and dQ
    of a row depend on that row alone), and dK/dV through identities that hold at any size,
    summed over each group: sum_j dV_j = sum over the group's heads of sum_i dO_i, sum_j dK_j = 0."""
    w, t = _gqa_full_inputs()
    g = {key: to_device(val, "bf16") for key, val in t.items()}
    res = _gqa_run(w, g)
    H, hkv = t["q"].shape[1], t["k"].shape[1]
    grp = H // hkv
    for key in ("out", "lse", "dq", "dk", "dv"):
        assert bool(torch.isfinite(res[key]).all()), key
    dv, dk = res["dv"].double(), res["dk"].double()
    sdo = g["do"].double().sum(dim=2).reshape(1, hkv, grp, -1).sum(dim=2)
    ev = float(torch.max(torch.abs(dv.sum(dim=2) - sdo)) / torch.max(torch.abs(dv).sum(dim=2)))
    ek = float(torch.max(torch.abs(dk.sum(dim=2))) / torch.max(torch.abs(dk).sum(dim=2)))
    print(f"gqa full size invariants sum_dv_minus_sum_do={ev:.3e} sum_dk={ek:.3e}", flush=True)
    assert ev <= 2e-3 and ek <= 2e-3
    rows = np.array([0, 1, 63, 64, 255, 256, 16383, 16401, 32639, 32703, 32766, 32767])
    for h in (0, 5, 10, 15):
        hk = h // grp
        q = inputs.to_f64(t["q"][0, h, rows], "bf16")
        k = inputs.to_f64(t["k"][0, hk], "bf16")
        v = inputs.to_f64(t["v"][0, hk], "bf16")
        do = inputs.to_f64(t["do"][0, h, rows], "bf16")
        o, l = oracle.head_attention(q, k, v, w.scale)
        D = oracle.head_bwd_preprocess(o, do)
        dq, _, _ = oracle.head_attention_bwd(q, k, v, do, l, D, w.scale)
        errs = {"out": rel_rms_err(to_host_f64(res["out"][0, h, rows]), o),
                "lse": float(np.max(np.abs(to_host_f64(res["lse"][0, h, rows]) - l))),
                "dq": rel_rms_err(to_host_f64(res["dq"][0, h, rows]), dq)}
        print(f"gqa full size head {h} (kv head {hk})",
              " ".join(f"{k_}={v_:.3e}" for k_, v_ in errs.items()), flush=True)
        assert errs["lse"] <= TOL_BF16_LSE
        assert errs["out"] <= TOL_BF16_REL_RMS and errs["dq"] <= TOL_BF16_REL_RMS


@pytest.mark.slow
def test_gqa_ring8_full_key_length_dkdv():
    """Grouped dK and dV over the full 262,144-key sequence in 8 chunks, element by element for
    K/V head 1 (query heads 4..7), with the query shard cut to its first 256 rows so the oracle
    can afford it; out, lse and dQ of those four heads in full."""
    w, t = _gqa_full_inputs(nq=256)
    g = {key: to_device(val, "bf16") for key, val in t.items()}
    res = _gqa_run(w, g)
    grp = t["q"].shape[1] // t["k"].shape[1]
    hk = 1
    k = inputs.to_f64(t["k"][0, hk], "bf16")
    v = inputs.to_f64(t["v"][0, hk], "bf16")
    rdk, rdv = np.zeros_like(k), np.zeros_like(v)
    errs = {}
    for h in range(hk * grp, (hk + 1) * grp):
        q = inputs.to_f64(t["q"][0, h], "bf16")
        do = inputs.to_f64(t["do"][0, h], "bf16")
        o, l = oracle.head_attention(q, k, v, w.scale)
        D = oracle.head_bwd_preprocess(o, do)
        dq, dk, dv = oracle.head_attention_bwd(q, k, v, do, l, D, w.scale)
        rdk += dk
        rdv += dv
        errs[f"out{h}"] = rel_rms_err(to_host_f64(res["out"][0, h]), o)
        errs[f"lse{h}"] = float(np.max(np.abs(to_host_f64(res["lse"][0, h]) - l)))
        errs[f"dq{h}"] = rel_rms_err(to_host_f64(res["dq"][0, h]), dq)
    errs["dk"] = rel_rms_err(to_host_f64(res["dk"][0, hk]), rdk)
    errs["dv"] = rel_rms_err(to_host_f64(res["dv"][0, hk]), rdv)
    print("gqa Nq=256 kv head 1", " ".join(f"{k_}={v_:.3e}" for k_, v_ in errs.items()), flush=True)
    for key, e in errs.items():
        assert e <= (TOL_BF16_LSE if key.startswith("lse") else TOL_BF16_REL_RMS), (key, e)
