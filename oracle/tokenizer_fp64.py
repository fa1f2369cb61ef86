"""Plain fp64 CPU oracle for the Turbulence Transformer's multi-fidelity tokenizer.

TEST INFRASTRUCTURE ONLY (same rules as attention_fp64: imported only by tests, the smoke check
and the benchmark's CPU-baseline leg; shares no code with the HIP path).

What it computes (arXiv 2507.16697 Sec. III-B "Turbulence Transformer": the three fidelity modes, and
Table III's filter / mode-size-ratio pairs): one fidelity mode of a field Y[c, z, y, x]
(x fastest) is

  1. the subdomain selection C(Y): a block of D/ratio x H/ratio x W/ratio cells centred at
     (cz, cy, cx), i.e. cells start + i with start = centre - size // 2, taken periodically;
  2. the Gaussian filter F(.) of size k^3 applied with stride k, which gives the (D/(ratio k)) x
     (H/(ratio k)) x (W/(ratio k)) grid the paper states for F(Y):
        F(Y)[c, a, b, e] = sum_{i,j,l < k} w_i w_j w_l Y[c, k a + i, k b + j, k e + l],
        w_i = exp(-(i - (k-1)/2)^2 / (2 sigma^2)) / sum_m exp(-(m - (k-1)/2)^2 / (2 sigma^2));
  3. patchify with patch p (the model's patch size): token t = px + Px (py + Py pz), feature
     f = ((c p + iz) p + iy) p + ix, giving tokens [L, C p^3].

Readings (the paper does not fix them):
T1  The Gaussian's width sigma is not given; it is an explicit argument (k/2 by default in the
    binding).  The weights are normalised so that a constant field passes unchanged; k = 1 is the
    identity.
T2  The filter is a k^3 convolution with stride k (non-overlapping windows), the reading under
    which F(Y) has the stated D/k x H/k x W/k shape.
T3  Subdomains wrap periodically (the turbulence boxes are periodic); size // 2 cells lie before
    the centre.
T4  Table III lists (filter; mode-size ratio) as (1, 4, 8); (8x, 2x, 1x): the pairs are
    (k, ratio) = (1, 8), (4, 2), (8, 1), so every mode has (D / (8 p))^3 tokens per step, which
    reproduces Table III's sequence lengths (1M = 64^3 x 4 steps for Small, and so on).
"""

from __future__ import annotations

import numpy as np

__all__ = ["gaussian_weights", "crop", "gaussian_filter", "patchify", "tt_tokenize",
           "mode_tokens"]


def gaussian_weights(k: int, sigma: float) -> np.ndarray:
    """Normalised 1D Gaussian weights over a window of k cells (reading T1)."""
    i = np.arange(k, dtype=np.float64)
    w = np.exp(-((i - (k - 1) / 2.0) ** 2) / (2.0 * sigma * sigma))
    return w / w.sum()


def crop(field: np.ndarray, size: tuple, centre: tuple) -> np.ndarray:
    """Periodic subdomain of `size` (z, y, x) cells centred at `centre` (reading T3)."""
    out = field
    for axis, (n, c) in enumerate(zip(size, centre)):
        idx = (c - n // 2 + np.arange(n)) % field.shape[axis + 1]
        out = np.take(out, idx, axis=axis + 1)
    return out


def gaussian_filter(field: np.ndarray, k: int, sigma: float) -> np.ndarray:
    """k^3 Gaussian window with stride k over field[c, z, y, x] (reading T2)."""
    C, Z, Y, X = field.shape
    w = gaussian_weights(k, sigma)
    blocks = field.reshape(C, Z // k, k, Y // k, k, X // k, k)
    return np.einsum("cairjsl,i,j,l->cars", blocks, w, w, w, optimize=True)


def patchify(grid: np.ndarray, p: int) -> np.ndarray:
    """Tokens [L, C p^3] of p^3 patches, token index x-fastest, feature ((c p + iz) p + iy) p + ix."""
    C, Z, Y, X = grid.shape
    g = grid.reshape(C, Z // p, p, Y // p, p, X // p, p)    # c, pz, iz, py, iy, px, ix
    g = g.transpose(1, 3, 5, 0, 2, 4, 6)                     # pz, py, px, c, iz, iy, ix
    return g.reshape((Z // p) * (Y // p) * (X // p), C * p * p * p)


def tt_tokenize(field: np.ndarray, k: int, ratio: int, centre: tuple, p: int,
                sigma: float) -> np.ndarray:
    """One fidelity mode: patchify(F_k(C_ratio(Y))) as tokens [L, C p^3] (steps 1-3 above)."""
    _, D, H, W = field.shape
    sub = crop(np.asarray(field, dtype=np.float64), (D // ratio, H // ratio, W // ratio), centre)
    return patchify(gaussian_filter(sub, k, sigma), p)


def mode_tokens(D: int, H: int, W: int, k: int, ratio: int, p: int) -> int:
    """Tokens of one fidelity mode per time step."""
    return (D // (ratio * k * p)) * (H // (ratio * k * p)) * (W // (ratio * k * p))
