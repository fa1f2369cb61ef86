"""The fp64 oracle against its pins (brute force, library routines, closed forms, invariants)."""

import numpy as np
import pytest

import oracle
from oracle import attention_fp64 as oa

from oracle_pins import (
    check_backward_autograd,
    check_backward_chunks,
    check_backward_fd,
    check_backward_invariants,
    check_chunk_bounds,
    check_forward,
    check_forward_closed_forms,
    check_forward_permutation,
    check_merge,
)


def test_forward_brute_force_and_sdpa():
    check_forward(oa.head_attention)


def test_forward_closed_forms():
    check_forward_closed_forms(oa.head_attention)


def test_forward_permutation():
    check_forward_permutation(oa.head_attention)


def test_merge_eq5():
    check_merge(oa.head_partials, oa.lse_merge, oa.head_attention)


def test_backward_finite_differences():
    check_backward_fd(oa.head_attention_bwd, oa.head_attention, oa.head_bwd_preprocess)


def test_backward_autograd():
    check_backward_autograd(oa.head_attention_bwd, oa.head_attention, oa.head_bwd_preprocess)


def test_backward_invariants_and_closed_forms():
    check_backward_invariants(oa.head_attention_bwd, oa.head_attention, oa.head_bwd_preprocess)


def test_backward_chunk_additivity():
    check_backward_chunks(oa.head_attention_bwd, oa.head_attention, oa.head_bwd_preprocess,
                          oa.chunk_bounds)


def test_chunk_bounds_partition():
    check_chunk_bounds(oa.chunk_bounds)


@pytest.mark.parametrize("nk,R,r", [(0, 1, 0), (5, 0, 0), (5, 6, 0), (5, 2, 2), (5, 2, -1)])
def test_chunk_bounds_rejects(nk, R, r):
    with pytest.raises(ValueError):
        oa.chunk_bounds(nk, R, r)


def test_merge_rejects_all_empty_rows():
    with pytest.raises(ValueError):
        oa.lse_merge(np.zeros((2, 3, 4)), np.full((2, 3), -np.inf))


def test_row_blocking_does_not_change_results():
    """Rows are independent: the memory blocking of the oracle gives the same rows."""
    rng = np.random.default_rng(11)
    q, k, v = rng.standard_normal((70, 8)), rng.standard_normal((33, 8)), rng.standard_normal((33, 8))
    do = rng.standard_normal((70, 8))
    O1, L1 = oa.head_attention(q, k, v, 0.3, row_block=7)
    O2, L2 = oa.head_attention(q, k, v, 0.3, row_block=1000)
    np.testing.assert_allclose(O1, O2, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(L1, L2, rtol=1e-14, atol=1e-15)
    D = oa.head_bwd_preprocess(O2, do)
    g1 = oa.head_attention_bwd(q, k, v, do, L2, D, 0.3, row_block=7)
    g2 = oa.head_attention_bwd(q, k, v, do, L2, D, 0.3, row_block=1000)
    for a, b in zip(g1, g2):
        np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-14)


def test_batched_helpers_match_heads():
    rng = np.random.default_rng(12)
    B, H, nq, nk, d, R = 2, 3, 11, 19, 4, 3
    q, k, v = (rng.standard_normal((B, H, n, d)) for n in (nq, nk, nk))
    do = rng.standard_normal((B, H, nq, d))
    O, L = oracle.attention(q, k, v, 0.5)
    Oc, Lc = oracle.attention_chunked(q, k, v, 0.5, R)
    np.testing.assert_allclose(Oc, O, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(Lc, L, rtol=1e-13, atol=1e-14)
    dq, dk, dv = oracle.attention_bwd(q, k, v, O, do, L, 0.5)
    for b in range(B):
        for h in range(H):
            Oh, Lh = oa.head_attention(q[b, h], k[b, h], v[b, h], 0.5)
            np.testing.assert_array_equal(O[b, h], Oh)
            g = oa.head_attention_bwd(q[b, h], k[b, h], v[b, h], do[b, h], Lh,
                                      oa.head_bwd_preprocess(Oh, do[b, h]), 0.5)
            np.testing.assert_array_equal(dq[b, h], g[0])
            np.testing.assert_array_equal(dk[b, h], g[1])
            np.testing.assert_array_equal(dv[b, h], g[2])
