"""Pins of the tokenizer oracle (oracle/tokenizer_fp64.py) against what the definition and the
paper fix: brute force on tiny fields, closed forms, invariants and Table III's sequence lengths;
and planted mistakes in copies of the oracle that the pins must catch."""

import itertools
import math

import numpy as np
import pytest

from oracle import tokenizer_fp64 as tk


def _brute(field, k, ratio, centre, p, sigma):
    """Triple loops written from the definition, pure Python."""
    C, D, H, W = field.shape
    size = (D // ratio, H // ratio, W // ratio)
    w = [math.exp(-((i - (k - 1) / 2) ** 2) / (2 * sigma * sigma)) for i in range(k)]
    s = sum(w)
    w = [x / s for x in w]
    g = [n // k for n in size]
    P = [n // p for n in g]
    out = np.zeros((P[0] * P[1] * P[2], C * p ** 3))
    for c, a, b, e in itertools.product(range(C), range(g[0]), range(g[1]), range(g[2])):
        acc = 0.0
        for i, j, l in itertools.product(range(k), range(k), range(k)):
            z = (centre[0] - size[0] // 2 + k * a + i) % D
            y = (centre[1] - size[1] // 2 + k * b + j) % H
            x = (centre[2] - size[2] // 2 + k * e + l) % W
            acc += w[i] * w[j] * w[l] * field[c, z, y, x]
        t = (a // p * P[1] + b // p) * P[2] + e // p
        f = ((c * p + a % p) * p + b % p) * p + e % p
        out[t, f] = acc
    return out


BRUTE_CASES = [(1, 1, (0, 0, 0), 1), (2, 1, (3, 1, 5), 2), (2, 2, (7, 0, 2), 1),
               (4, 1, (5, 6, 7), 1), (1, 2, (1, 7, 3), 2)]


def check_brute(tok):
    rng = np.random.default_rng(7)
    field = rng.standard_normal((2, 8, 8, 8))
    for k, ratio, centre, p in BRUTE_CASES:
        sigma = max(k / 2, 0.5)
        got = tok(field, k, ratio, centre, p, sigma)
        ref = _brute(field, k, ratio, centre, p, sigma)
        assert got.shape == ref.shape
        assert np.max(np.abs(got - ref)) <= 1e-13


def check_identity(tok):
    """k = 1, ratio = 1, p = 1 with the centre at size//2: the tokens are the field, cell by
    cell in x-fastest order, one feature per channel."""
    field = np.random.default_rng(8).standard_normal((4, 4, 6, 8))
    got = tok(field, 1, 1, (2, 3, 4), 1, 0.5)
    assert np.array_equal(got, field.reshape(4, -1).T)


def check_constant(tok):
    field = np.full((3, 16, 16, 16), 2.5)
    got = tok(field, 4, 2, (9, 1, 15), 2, 1.7)
    assert np.max(np.abs(got - 2.5)) <= 1e-14


def check_periodic_shift(tok):
    """Moving the centre by k cells shifts the filtered grid by one cell (periodic field)."""
    field = np.random.default_rng(10).standard_normal((1, 16, 16, 16))
    a = tok(field, 4, 1, (8, 8, 8), 1, 2.0).reshape(4, 4, 4)
    b = tok(field, 4, 1, (8, 8, 12), 1, 2.0).reshape(4, 4, 4)
    assert np.max(np.abs(np.roll(a, -1, axis=2) - b)) <= 1e-14


CHECKS = (check_brute, check_identity, check_constant, check_periodic_shift)


@pytest.mark.parametrize("check", CHECKS)
def test_oracle_pins(check):
    check(tk.tt_tokenize)


def test_separable_field():
    """Y = f(z) g(y) h(x): the filter acts per axis, F(Y) = (w*f)(w*g)(w*h) block-wise."""
    rng = np.random.default_rng(9)
    f, g, h = (rng.standard_normal(16) for _ in range(3))
    field = np.einsum("z,y,x->zyx", f, g, h)[None]
    k, sigma = 4, 1.3
    w = tk.gaussian_weights(k, sigma)
    got = tk.gaussian_filter(field, k, sigma)[0]
    ref = np.einsum("z,y,x->zyx", *(v.reshape(-1, k) @ w for v in (f, g, h)))
    assert np.max(np.abs(got - ref)) <= 1e-13


def test_weights_are_a_normalised_gaussian():
    w = tk.gaussian_weights(8, 4.0)
    assert abs(w.sum() - 1.0) <= 1e-15
    assert np.allclose(w, w[::-1], rtol=0, atol=1e-16)            # symmetric about (k-1)/2
    assert np.isclose(w[4] / w[5], math.exp((1.5 ** 2 - 0.5 ** 2) / 32.0))
    assert np.array_equal(tk.gaussian_weights(1, 0.3), np.ones(1))


def test_table_iii_sequence_lengths():
    """Table III: every fidelity mode of a 1024^3 box has the same token count, and times the
    time steps it gives the listed sequence lengths (Small 1M, Medium 4M, Large 2M, XL 1M)."""
    D = 1024
    configs = {  # name: (patch, (filters), (ratios), steps, sequence length)
        "Small": (2, (1, 4, 8), (8, 2, 1), 4, 1 << 20),
        "Medium": (1, (1, 4, 8), (8, 2, 1), 2, 1 << 22),
        "Large": (1, (1, 4, 8), (8, 2, 1), 1, 1 << 21),
        "XL": (1, (2, 8, 16), (8, 2, 1), 4, 1 << 20),
    }
    for name, (p, ks, ratios, steps, seq) in configs.items():
        counts = {tk.mode_tokens(D, D, D, k, r, p) for k, r in zip(ks, ratios)}
        assert len(counts) == 1, name
        assert counts.pop() * steps == seq, name


# ----------------------------------------------------------------------------------------------
# planted mistakes


def _mutant(mutation):
    def weights(k, sigma):
        i = np.arange(k, dtype=np.float64)
        centre = k / 2.0 if mutation == "weights_off_centre" else (k - 1) / 2.0
        w = np.exp(-((i - centre) ** 2) / (2.0 * sigma * sigma))
        return w if mutation == "weights_unnormalised" else w / w.sum()

    def tok(field, k, ratio, centre, p, sigma):
        field = np.asarray(field, dtype=np.float64)
        C, D, H, W = field.shape
        sub = field
        for axis, (n, c) in enumerate(zip((D // ratio, H // ratio, W // ratio), centre)):
            start = c - n // 2 + (1 if mutation == "crop_start_off_by_one" else 0)
            idx = start + np.arange(n)
            idx = np.clip(idx, 0, field.shape[axis + 1] - 1) if mutation == "crop_clamped" \
                else idx % field.shape[axis + 1]
            sub = np.take(sub, idx, axis=axis + 1)
        w = weights(k, sigma)
        _, Z, Y, X = sub.shape
        blocks = sub.reshape(C, Z // k, k, Y // k, k, X // k, k)
        grid = np.einsum("cairjsl,i,j,l->cars", blocks, w, w, w)
        g = grid.reshape(C, Z // k // p, p, Y // k // p, p, X // k // p, p)
        order = (1, 3, 5, 0, 2, 4, 6)
        if mutation == "features_x_slowest":
            order = (1, 3, 5, 0, 6, 4, 2)
        if mutation == "tokens_z_fastest":
            order = (5, 3, 1, 0, 2, 4, 6)
        g = g.transpose(order)
        return g.reshape(-1, C * p * p * p)
    return tok


@pytest.mark.parametrize("mutation", ["weights_unnormalised", "weights_off_centre",
                                      "crop_start_off_by_one", "crop_clamped",
                                      "features_x_slowest", "tokens_z_fastest"])
def test_tokenizer_mutants_fail(mutation):
    mutant = _mutant(mutation)
    failed = 0
    for check in CHECKS:
        try:
            check(mutant)
        except AssertionError:
            failed += 1
    assert failed >= 1, mutation


def test_unmutated_copy_passes():
    for check in CHECKS:
        check(_mutant("none"))
