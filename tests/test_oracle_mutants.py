"""Planted mistakes in copies of the oracle must fail its pins.

Each mutant is the oracle function with one plausible slip (a dropped term, a wrong sign, a wrong
index or axis, a transposed operand, a missing scale).  If a pin let one through, the pins would
not be protecting the oracle.  Everything here runs on the CPU.
"""

import numpy as np
import pytest

from oracle import attention_fp64 as oa

from oracle_pins import (
    check_backward_autograd,
    check_backward_fd,
    check_backward_invariants,
    check_forward,
    check_forward_closed_forms,
    check_merge,
)

SMALL = [(3, 5, 2), (17, 31, 8), (2, 2, 1), (4, 7, 3)]


def _fwd(mutation):
    def head_attention(q, k, v, scale, row_block=1024):
        q, k, v = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
        s = scale * (q @ k.T)
        if mutation == "no_scale":
            s = q @ k.T
        m = s.max(axis=1)
        if mutation == "max_wrong_axis":
            m = np.broadcast_to(s.max(axis=0).mean(), m.shape)
        z = np.exp(s - m[:, None]).sum(axis=1)
        lse = m + np.log(z)
        if mutation == "lse_drops_log_z":
            lse = m
        p = np.exp(s - lse[:, None])
        if mutation == "unnormalised":
            p = np.exp(s - m[:, None])
        out = p @ v
        if mutation == "value_rows_reversed":
            out = p @ v[::-1]
        return out, lse
    return head_attention


@pytest.mark.parametrize("mutation", ["no_scale", "lse_drops_log_z", "unnormalised",
                                      "value_rows_reversed", "max_wrong_axis"])
def test_forward_mutants_fail(mutation):
    mutant = _fwd(mutation)
    failed = 0
    for check in (lambda: check_forward(mutant, shapes=SMALL),
                  lambda: check_forward_closed_forms(mutant)):
        try:
            check()
        except AssertionError:
            failed += 1
    if mutation == "max_wrong_axis":
        # a wrong shift is exact in exact arithmetic; the pins must not mistake it for an error
        assert failed == 0
    else:
        assert failed >= 1, f"mutant {mutation} passed every forward pin"


def _merge(mutation):
    def lse_merge(part_out, part_lse):
        part_out = np.asarray(part_out, dtype=np.float64)
        part_lse = np.asarray(part_lse, dtype=np.float64)
        M = part_lse.max(axis=0)
        w = np.exp(part_lse - M)
        if mutation == "weight_sign":
            w = np.exp(M - part_lse)
        den = w.sum(axis=0)
        if mutation == "den_counts_partials":
            den = np.full_like(den, part_lse.shape[0])
        num = (part_out * w[..., None]).sum(axis=0)
        lse = M + np.log(den)
        if mutation == "lse_drops_log_den":
            lse = M
        return num / den[..., None], lse
    return lse_merge


@pytest.mark.parametrize("mutation", ["weight_sign", "den_counts_partials", "lse_drops_log_den"])
def test_merge_mutants_fail(mutation):
    with pytest.raises(AssertionError):
        check_merge(oa.head_partials, _merge(mutation), oa.head_attention)


def _bwd(mutation):
    def head_attention_bwd(q, k, v, do, lse, D, scale, row_block=1024):
        q, k, v, do = (np.asarray(x, dtype=np.float64) for x in (q, k, v, do))
        s = scale * (q @ k.T)
        p = np.exp(s - np.asarray(lse)[:, None])
        dv = p.T @ do
        if mutation == "dv_transposed":
            dv = (p @ np.eye(p.shape[1])).T @ do[::-1]
        dp = do @ v.T
        ds = p * (dp - np.asarray(D)[:, None])
        if mutation == "ds_sign":
            ds = p * (np.asarray(D)[:, None] - dp)
        if mutation == "ds_drops_D":
            ds = p * dp
        dk = scale * (ds.T @ q)
        if mutation == "dk_no_scale":
            dk = ds.T @ q
        dq = scale * (ds @ k)
        if mutation == "dq_uses_v":
            dq = scale * (ds @ v)
        return dq, dk, dv
    return head_attention_bwd


@pytest.mark.parametrize("mutation", ["dv_transposed", "ds_sign", "ds_drops_D", "dk_no_scale",
                                      "dq_uses_v"])
def test_backward_mutants_fail(mutation):
    mutant = _bwd(mutation)
    failed = 0
    for check in (check_backward_fd, check_backward_autograd, check_backward_invariants):
        try:
            check(mutant, oa.head_attention, oa.head_bwd_preprocess)
        except AssertionError:
            failed += 1
    assert failed >= 2, f"mutant {mutation} was caught by only {failed} backward pin(s)"
