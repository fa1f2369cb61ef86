"""Shared helpers of the GPU parity tests: moving seeded inputs to the device and comparing."""

from __future__ import annotations

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


def _sample_rows(Nq):
    """Rows at tile edges (query tiles of 128 and 64), the middle and the end."""
    rows = {0, 1, 63, 64, 127, 128, 129, Nq // 2 - 1, Nq // 2 + 17, Nq - 129, Nq - 65, Nq - 2,
            Nq - 1}
    return np.array(sorted(r for r in rows if 0 <= r < Nq))


def check_rows(name, w, t, res, heads, with_bwd=True):
    """out, lse (and dQ) of sampled rows of `heads` against the oracle, row by row."""
    rows = _sample_rows(w.Nq)
    got_o, ref_o, got_l, ref_l, got_dq, ref_dq = [], [], [], [], [], []
    out = res["out"]
    for h in heads:
        q = inputs.to_f64(t["q"][0, h, rows], "bf16")
        k = inputs.to_f64(t["k"][0, h], "bf16")
        v = inputs.to_f64(t["v"][0, h], "bf16")
        o, l = oracle.head_attention(q, k, v, w.scale)
        got_o.append(to_host_f64(out[0, h, rows]))
        ref_o.append(o)
        got_l.append(to_host_f64(res["lse"][0, h, rows]))
        ref_l.append(l)
        if with_bwd:
            do = inputs.to_f64(t["do"][0, h, rows], "bf16")
            D = oracle.head_bwd_preprocess(o, do)
            dq, _, _ = oracle.head_attention_bwd(q, k, v, do, l, D, w.scale)
            got_dq.append(to_host_f64(res["dq"][0, h, rows]))
            ref_dq.append(dq)
    errs = {"out": rel_rms_err(np.concatenate(got_o), np.concatenate(ref_o)),
            "lse": float(np.max(np.abs(np.concatenate(got_l) - np.concatenate(ref_l))))}
    if with_bwd:
        errs["dq"] = rel_rms_err(np.concatenate(got_dq), np.concatenate(ref_dq))
    print(f"{name} rows {list(rows)} heads {list(heads)}",
          " ".join(f"{k}={v:.3e}" for k, v in errs.items()), flush=True)
    assert errs["out"] <= TOL_BF16_REL_RMS and errs["lse"] <= TOL_BF16_LSE
    if with_bwd:
        assert errs["dq"] <= TOL_BF16_REL_RMS
