"""The bf16 backward on unit-variance inputs (Q, K, V, dO ~ N(0, 1), so the scaled scores have
standard deviation 1, twice that of the widest paper-shaped workload), against the fp64 oracle.

The parity measure (max abs error / reference RMS <= 2e-2) is met on the paper-shaped workloads,
whose scores have standard deviation 0.25-0.5.  With scores of standard deviation 1 the softmax
rows are more peaked, fewer terms average each gradient's rounding, and the bf16 rounding of P and
dS before the dV and dK contractions alone (the mixed-precision method itself, reproduced in
fp64 on the host) gives up to about 3.4e-2 on dK at d = 128.  So here every gradient element is
held to the error bound of the path's roundings (P and dS rounded to bf16, the output stored in
bf16, D formed from it; 1.5x margin), the output and lse to the usual bars, and the RMS measure of
each gradient is printed beside it; the RMS bar is asserted where the method meets it.
"""

import math

import numpy as np
import pytest
import torch

import oracle
from paper_2507_16697_amd import ringx

from parity_util import (TOL_BF16_LSE, TOL_BF16_REL_RMS, max_abs_err, random_case,
                         rel_rms_err, rounding_bounds, to_device, to_host_f64)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("d", [64, 128])
def test_unit_variance_backward(d):
    B, H, Nq, Nk, R = 1, 2, 1024, 4096, 4
    t, x = random_case(70 + d, B, H, Nq, Nk, d, store="bf16", std=1.0, do_std=1.0)
    g = {k: to_device(v, "bf16") for k, v in t.items()}
    scale = float(np.float32(1 / math.sqrt(d)))
    out, lse = ringx.ringx_attn_fwd(g["q"], g["k"], g["v"], R, scale=scale)
    dq, dk, dv = ringx.ringx_attn_bwd(g["q"], g["k"], g["v"], out, g["do"], lse, R, scale=scale)
    torch.cuda.synchronize()
    ro, rl = oracle.attention(x["q"], x["k"], x["v"], scale)
    rq, rk, rv = oracle.attention_bwd(x["q"], x["k"], x["v"], ro, x["do"], rl, scale)
    b_out, b_dq, b_dk, b_dv = rounding_bounds(x, x["k"], x["v"], ro, rl, scale)
    got = {"out": to_host_f64(out), "dq": to_host_f64(dq), "dk": to_host_f64(dk),
           "dv": to_host_f64(dv)}
    ref = {"out": ro, "dq": rq, "dk": rk, "dv": rv}
    bnd = {"out": b_out, "dq": b_dq, "dk": b_dk, "dv": b_dv}
    rms = {k: rel_rms_err(got[k], ref[k]) for k in got}
    frac = {}
    for k in got:
        lim = 1.5 * bnd[k] + 1e-5 * max(1.0, float(np.max(np.abs(ref[k]))))
        frac[k] = float(np.max(np.abs(got[k] - ref[k]) / lim))
    lse_err = max_abs_err(to_host_f64(lse), rl)
    print(f"unit variance d={d}: max-abs/RMS", " ".join(f"{k}={v:.2e}" for k, v in rms.items()),
          "| fraction of the rounding bound", " ".join(f"{k}={v:.2f}" for k, v in frac.items()),
          f"| lse={lse_err:.2e}", flush=True)
    assert lse_err <= TOL_BF16_LSE
    assert rms["out"] <= TOL_BF16_REL_RMS
    for k, v in frac.items():
        assert v <= 1.0, (k, v)
