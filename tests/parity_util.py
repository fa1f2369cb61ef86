"""Shared helpers of the GPU parity tests: moving seeded inputs to the device and comparing."""

from __future__ import annotations

import numpy as np
import torch

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
