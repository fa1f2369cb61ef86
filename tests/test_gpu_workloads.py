"""The paper-shaped workloads at their full sizes, through the C ABI, against the fp64 oracle.

Every workload runs in the launch configuration bench.py times (ringx_attn_fwd, then
ringx_bwd_preprocess, ringx_attn_bwd_dkdv and ringx_attn_bwd_dq).  Where the oracle can afford
the whole tensor it checks all of it; otherwise it checks, element by element, 256 seeded query
rows of every head (out, lse and dQ of a row depend on that row and all keys) and 256 keys of
chosen heads over the full query shard (dK and dV of a key depend on that key and all queries,
given every row's lse and D from one full oracle pass of the head), and also the gradients of K
and V through identities that hold at any size:
  sum_j dV_j = sum_i dO_i           (each softmax row sums to 1)
  sum_j dK_j = 0                    (each row of dS sums to D_i - D_i = 0)
"""

import math

import numpy as np
import pytest
import torch

import oracle
from paper_2507_16697_amd import inputs, ringx

from parity_util import (TOL_BF16_LSE, TOL_BF16_REL_RMS, check_rows, err_stats, max_abs_err,
                         oracle_head_stats, oracle_key_grads, rel_rms_err, sample_keys, to_device,
                         to_host_f64)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _report(name, **errs):
    print(name, " ".join(f"{k}={v:.3e}" for k, v in errs.items()), flush=True)


def _run(w, g, with_bwd=True):
    """The bench.py step on device tensors g; returns the device results."""
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], w.R, scale=w.scale)
    res = {"out": out, "lse": lse}
    if with_bwd:
        delta = ringx.ringx_bwd_preprocess(out, g["do"], lse)
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


@pytest.fixture(scope="module")
def ring8():
    """The 8-way ring share (Nq=32768, Nk=262144, R=8, d=128) through the bench step, once."""
    w = inputs.WORKLOADS["ring8_nk262k_d128"]
    t = inputs.make_workload(w.name)
    g = {key: to_device(val, "bf16") for key, val in t.items()}
    res = _run(w, g)
    yield w, t, g, res
    del g, res
    torch.cuda.empty_cache()


def test_ring8_nk262k_d128_full_size(ring8):
    """The bench workload: invariants, and out/lse/dQ of 256 seeded rows of every head."""
    w, t, g, res = ring8
    _check_invariants(w.name, g, res)
    check_rows(w.name, w, t, res, heads=range(w.H))


def _check_sampled_keys(name, w, t, res, h):
    """dK and dV of >= 256 keys of head h (every chunk's first and last keys and the tile edges
    around them, plus seeded keys) over the full query shard, element by element against the
    oracle, which needs every row's lse and D (one full pass of the head) and then only those
    keys against all queries."""
    x = {key: inputs.to_f64(t[key][0, h], "bf16") for key in t}
    _, lse, D = oracle_head_stats(x["q"], x["k"], x["v"], x["do"], w.scale)
    keys = sample_keys(w.Nk, w.R, 256, seed=1000 * w.seed + h)
    dk, dv = oracle_key_grads(x["q"], x["k"], x["v"], x["do"], lse, D, w.scale, keys)
    idx = torch.as_tensor(keys, device=res["dk"].device)
    errs = {"dk": err_stats(to_host_f64(res["dk"][0, h].index_select(0, idx)), dk),
            "dv": err_stats(to_host_f64(res["dv"][0, h].index_select(0, idx)), dv),
            "lse": (max_abs_err(to_host_f64(res["lse"][0, h]), lse), 1.0, 0.0)}
    print(f"{name} head {h}: {len(keys)} keys x {w.Nq} queries",
          " ".join(f"{k}: max_abs={m:.3e} rms={r:.3e} ratio={e:.3e}"
                   for k, (m, r, e) in errs.items() if k != "lse"),
          f"lse (all {w.Nq} rows) max_abs={errs['lse'][0]:.3e}", flush=True)
    assert errs["lse"][0] <= TOL_BF16_LSE
    for key in ("dk", "dv"):
        assert errs[key][2] <= TOL_BF16_REL_RMS, (key, errs[key])


@pytest.mark.parametrize("h", [0, 15])
def test_ring8_dkdv_sampled_keys_full_queries(ring8, h):
    w, t, _, res = ring8
    _check_sampled_keys(w.name, w, t, res, h)


def test_ring8_full_key_length_dkdv():
    """dK and dV over the full 262,144-key sequence in 8 chunks, compared element by element for
    two heads, with the query shard cut to its first 1024 rows so the oracle can afford every
    key."""
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
    check_rows(w.name, w, t, res, heads=range(w.H), with_bwd=False)


@pytest.fixture(scope="module")
def long_step():
    """The long training step (Nq=65536, Nk=524288, R=8, d=128) through the bench step, once."""
    w = inputs.WORKLOADS["long_nk524k_d128"]
    t = inputs.make_workload(w.name, use_cache=False)
    g = {key: to_device(val, "bf16") for key, val in t.items()}
    res = _run(w, g)
    yield w, t, g, res
    del g, res
    torch.cuda.empty_cache()


def test_long_nk524k_d128(long_step):
    """Long-context step: invariants, and out/lse/dQ of 256 seeded rows of every head."""
    w, t, g, res = long_step
    _check_invariants(w.name, g, res)
    check_rows(w.name, w, t, res, heads=range(w.H))


def test_long_dkdv_sampled_keys_full_queries(long_step):
    """dK/dV of >= 256 keys of head 0 over all 65536 queries; the fp32 dK there spans 4 GiB."""
    w, t, _, res = long_step
    _check_sampled_keys(w.name, w, t, res, 0)
