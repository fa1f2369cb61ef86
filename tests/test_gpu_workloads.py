"""The paper-shaped workloads at their full sizes, through the C ABI, against the fp64 oracle.

Every workload runs in the launch configuration bench.py times (ringx_attn_fwd, then
ringx_bwd_preprocess, ringx_attn_bwd_dkdv and ringx_attn_bwd_dq).  Where the oracle can afford
the whole tensor it checks all of it; otherwise it checks sampled query rows, which it computes
one by one against every key (out, lse and dQ of a row depend on that row alone), and the
gradients of K and V through identities that hold at any size:
  sum_j dV_j = sum_i dO_i           (each softmax row sums to 1)
  sum_j dK_j = 0                    (each row of dS sums to D_i - D_i = 0)
"""

import math

import numpy as np
import pytest
import torch

import oracle
from paper_2507_16697_amd import inputs, ringx

from parity_util import (TOL_BF16_LSE, TOL_BF16_REL_RMS, check_rows, rel_rms_err, to_device,
                         to_host_f64)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _report(name, **errs):
    print(name, " ".join(f"{k}={v:.3e}" for k, v in errs.items()), flush=True)


def _run(w, g, with_bwd=True):
    """The bench.py step on device tensors g; returns the device results."""
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], w.R, scale=w.scale)
    res = {"out": out, "lse": lse}
    if with_bwd:
        delta = ringx.ringx_bwd_preprocess(out, g["do"])
        res["dk"], res["dv"] = ringx.ringx_attn_bwd_dkdv(g["q"], g["k"], g["v"], g["do"], lse,
                                                         delta, w.R, scale=w.scale)
        res["dq"] = ringx.ringx_attn_bwd_dq(g["q"], g["k"], g["v"], g["do"], lse, delta, w.R,
                                            scale=w.scale)
    torch.cuda.synchronize()
    return res


def _check_invariants(name, g, res):
    dk, dv = res["dk"].double(), res["dv"].double()
    sdv, sdo = dv.sum(dim=2), g["do"].double().sum(dim=2)
    sdk = dk.sum(dim=2)
    ev = float(torch.max(torch.abs(sdv - sdo)) / torch.max(torch.abs(dv).sum(dim=2)))
    ek = float(torch.max(torch.abs(sdk)) / torch.max(torch.abs(dk).sum(dim=2)))
    _report(f"{name} invariants", sum_dv_minus_sum_do=ev, sum_dk=ek)
    assert ev <= 2e-3 and ek <= 2e-3
    for key in ("out", "lse", "dq", "dk", "dv"):
        assert bool(torch.isfinite(res[key]).all()), key


def test_ring8_nk262k_d128_full_size():
    """One GPU's share of an 8-way ring (Nq=32768, Nk=262144, R=8, d=128): the bench workload."""
    w = inputs.WORKLOADS["ring8_nk262k_d128"]
    t = inputs.make_workload(w.name)
    g = {key: to_device(val, "bf16") for key, val in t.items()}
    res = _run(w, g)
    _check_invariants(w.name, g, res)
    check_rows(w.name, w, t, res, heads=(0, 6, 15))


def test_ring8_full_key_length_dkdv():
    """dK and dV over the full 262,144-key sequence in 8 chunks, compared element by element for
    two heads, with the query shard cut to its first 1024 rows so the oracle can afford it."""
    w = inputs.WORKLOADS["ring8_nk262k_d128"]
    t = inputs.make_workload(w.name)
    nq = 1024
    t = {"q": t["q"][:, :, :nq], "k": t["k"], "v": t["v"], "do": t["do"][:, :, :nq]}
    g = {key: to_device(val, "bf16") for key, val in t.items()}
    res = _run(w, g)
    for h in (0, 11):
        x = {key: inputs.to_f64(t[key][0, h], "bf16") for key in t}
        o, l = oracle.head_attention(x["q"], x["k"], x["v"], w.scale)
        D = oracle.head_bwd_preprocess(o, x["do"])
        dq, dk, dv = oracle.head_attention_bwd(x["q"], x["k"], x["v"], x["do"], l, D, w.scale)
        errs = {"out": rel_rms_err(to_host_f64(res["out"][0, h]), o),
                "lse": float(np.max(np.abs(to_host_f64(res["lse"][0, h]) - l))),
                "dq": rel_rms_err(to_host_f64(res["dq"][0, h]), dq),
                "dk": rel_rms_err(to_host_f64(res["dk"][0, h]), dk),
                "dv": rel_rms_err(to_host_f64(res["dv"][0, h]), dv)}
        _report(f"ring8 Nq={nq} head {h}", **errs)
        assert errs["lse"] <= TOL_BF16_LSE
        for key in ("out", "dq", "dk", "dv"):
            assert errs[key] <= TOL_BF16_REL_RMS, (key, errs[key])


def test_shard_n16k_d64_full():
    """Single-shard bf16 case (Nq=Nk=16384, d=64, R=4): every element of three heads."""
    w = inputs.WORKLOADS["shard_n16k_d64"]
    t = inputs.make_workload(w.name)
    g = {key: to_device(val, "bf16") for key, val in t.items()}
    res = _run(w, g)
    _check_invariants(w.name, g, res)
    for h in (0, 7, 15):
        x = {key: inputs.to_f64(t[key][0, h], "bf16") for key in t}
        o, l = oracle.head_attention(x["q"], x["k"], x["v"], w.scale)
        D = oracle.head_bwd_preprocess(o, x["do"])
        dq, dk, dv = oracle.head_attention_bwd(x["q"], x["k"], x["v"], x["do"], l, D, w.scale)
        errs = {"out": rel_rms_err(to_host_f64(res["out"][0, h]), o),
                "lse": float(np.max(np.abs(to_host_f64(res["lse"][0, h]) - l))),
                "dq": rel_rms_err(to_host_f64(res["dq"][0, h]), dq),
                "dk": rel_rms_err(to_host_f64(res["dk"][0, h]), dk),
                "dv": rel_rms_err(to_host_f64(res["dv"][0, h]), dv)}
        _report(f"{w.name} head {h}", **errs)
        assert errs["lse"] <= TOL_BF16_LSE
        for key in ("out", "dq", "dk", "dv"):
            assert errs[key] <= TOL_BF16_REL_RMS, (key, errs[key])


def test_turbulence_tokens_forward():
    """Turbulence-shaped tokens (256^3 field, 4^3 patches, width 1024, 16 heads of 64), a query
    shard of 65536 against all 262144 keys in 4 chunks; forward only."""
    w = inputs.WORKLOADS["turbulence_nk262k_d64"]
    t = inputs.make_workload(w.name)
    g = {key: to_device(val, "bf16") for key, val in t.items()}
    res = _run(w, g, with_bwd=False)
    assert bool(torch.isfinite(res["out"].float()).all()) and bool(torch.isfinite(res["lse"]).all())
    check_rows(w.name, w, t, res, heads=(0, 3, 8, 15), with_bwd=False)


def test_long_nk524k_d128():
    """Long-context step (Nq=65536, Nk=524288, R=8, d=128): forward and backward."""
    w = inputs.WORKLOADS["long_nk524k_d128"]
    t = inputs.make_workload(w.name, use_cache=False)
    g = {key: to_device(val, "bf16") for key, val in t.items()}
    res = _run(w, g)
    _check_invariants(w.name, g, res)
    check_rows(w.name, w, t, res, heads=(0, 15))
