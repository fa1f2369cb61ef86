"""The multi-fidelity tokenizer (ringx_tt_tokenize) against the fp64 tokenizer oracle."""

import numpy as np
import pytest
import torch

import oracle
from paper_2507_16697_amd import inputs, ringx

from parity_util import TOL_BF16_REL_RMS, TOL_F32, max_abs_err, rel_rms_err

pytestmark = pytest.mark.gpu


def _field(seed, shape):
    return np.random.default_rng(seed).standard_normal(shape).astype(np.float32)


CASES = [  # (k, ratio, p, centre)
    (1, 1, 1, (0, 0, 0)), (1, 8, 1, (63, 5, 40)), (4, 2, 1, (3, 60, 31)), (8, 1, 1, (20, 20, 20)),
    (2, 2, 2, (0, 63, 1)), (4, 1, 2, (33, 2, 61)), (2, 4, 1, (62, 62, 62)), (16, 1, 2, (7, 9, 11)),
]


@pytest.mark.parametrize("k,ratio,p,centre", CASES)
def test_tokenizer_fp32(k, ratio, p, centre):
    f = _field(61, (4, 64, 64, 64))
    g = torch.from_numpy(f).cuda()
    sigma = k / 2.0
    tok = ringx.ringx_tt_tokenize(g, k, ratio, centre, p, sigma=sigma)
    torch.cuda.synchronize()
    ref = oracle.tt_tokenize(f.astype(np.float64), k, ratio, centre, p, float(np.float32(sigma)))
    assert tok.shape == ref.shape
    assert max_abs_err(tok.cpu().numpy(), ref) <= TOL_F32


def test_tokenizer_edge_shapes():
    """k = 32 (the largest window), one channel, a non-cubic field."""
    f = _field(62, (1, 64, 32, 128))
    g = torch.from_numpy(f).cuda()
    tok = ringx.ringx_tt_tokenize(g, 32, 1, (31, 0, 100), 1, sigma=9.0)
    tok2 = ringx.ringx_tt_tokenize(g, 2, 2, (1, 31, 127), 4, sigma=0.7)
    torch.cuda.synchronize()
    assert max_abs_err(tok.cpu().numpy(),
                       oracle.tt_tokenize(f.astype(np.float64), 32, 1, (31, 0, 100), 1,
                                          9.0)) <= TOL_F32
    assert max_abs_err(tok2.cpu().numpy(),
                       oracle.tt_tokenize(f.astype(np.float64), 2, 2, (1, 31, 127), 4,
                                          float(np.float32(0.7)))) <= TOL_F32


def test_tokenizer_turbulence_modes_bf16():
    """The synthetic 256^3 divergence-free field, three modes with Table III's (filter, ratio)
    pairs and patch 2: every mode has (256/16)^3 tokens; bf16 tokens to the parity bar."""
    u = inputs.turbulence_field(256, seed=4).astype(np.float32)
    g = torch.from_numpy(u).cuda()
    for k, ratio, centre in ((1, 8, (17, 200, 3)), (4, 2, (128, 0, 255)), (8, 1, (0, 0, 0))):
        tok = ringx.ringx_tt_tokenize(g, k, ratio, centre, 2, out_dtype=torch.bfloat16)
        torch.cuda.synchronize()
        ref = oracle.tt_tokenize(u.astype(np.float64), k, ratio, centre, 2, k / 2.0)
        assert tok.shape == (16 ** 3, 3 * 8) == ref.shape
        assert rel_rms_err(tok.float().cpu().numpy(), ref) <= TOL_BF16_REL_RMS


@pytest.mark.parametrize("shape,k,ratio,p,centre", [((2, 24, 18, 30), 3, 1, 2, (5, 17, 29)),
                                                    ((2, 24, 18, 30), 2, 1, 1, (0, 9, 3)),
                                                    ((1, 48, 48, 48), 3, 2, 4, (47, 0, 13))])
def test_tokenizer_generic_kernel(shape, k, ratio, p, centre):
    """Filters that are not powers of two, and subdomain rows not a multiple of 4 cells, take the
    one-thread-per-cell kernel."""
    f = _field(63, shape)
    g = torch.from_numpy(f).cuda()
    tok = ringx.ringx_tt_tokenize(g, k, ratio, centre, p, sigma=1.1)
    torch.cuda.synchronize()
    ref = oracle.tt_tokenize(f.astype(np.float64), k, ratio, centre, p, float(np.float32(1.1)))
    assert max_abs_err(tok.cpu().numpy(), ref) <= TOL_F32
