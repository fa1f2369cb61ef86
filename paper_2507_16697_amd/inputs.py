"""Seeded synthetic inputs shaped like the paper's attention workloads.

This module generates inputs only: it holds none of the attention arithmetic, and it is the one
piece of code shared by the HIP path's tests/benchmark and by the fp64 oracle.

Rules common to every workload:
  * every (tensor, b, h) slab is its own PCG64 stream,
    numpy.random.default_rng([seed, tensor, b, h]).standard_normal((N, d)), with tensor = 0, 1, 2, 3
    for Q, K, V, dO (independent streams, so a huge tensor is generated slab by slab, in parallel);
  * values are scaled in fp64, then stored as fp32 (round to nearest even) or as bf16 bits
    (fp64 -> fp32 -> bf16, each step round to nearest even).

Workloads (layout [B, H, N, d]):
  exact_fp32_n1k         B=1 H=2  Nq=Nk=1024     d=64  R=4 fp32  seed 0 ~N(0,1)          fwd
  shard_n16k_d64         B=1 H=16 Nq=Nk=16384    d=64  R=4 bf16  seed 1 ~0.5 N(0,1); dO seed 2 ~N(0,1)
                         (tokens of a 32x32x16 patch grid, x fastest; the values are i.i.d.)
  ring8_nk262k_d128      B=1 H=16 Nq=32768 Nk=262144 d=128 R=8 bf16 seed 3 ~N(0,1)/sqrt2, dO seed 3
                         too (one GPU's query shard of an 8-way ring over a 64^3 token grid)
  turbulence_nk262k_d64  B=1 H=16 Nq=65536 Nk=262144 d=64 R=4 bf16, tokens of a synthetic
                         divergence-free k^-5/3 velocity field (see turbulence_qkv); fwd only
  long_nk524k_d128       B=1 H=16 Nq=65536 Nk=524288 d=128 R=8 bf16 seed 5, Q,K,V,dO ~N(0,1)/sqrt2

Turbulence tokens stand in for the JHTDB forced-isotropic-turbulence snapshots the paper trains on
(Sec. V-B), which are not available here.
"""

from __future__ import annotations

import concurrent.futures
import dataclasses
import hashlib
import math
import os

import numpy as np

# ----------------------------------------------------------------------------------------------
# storage conversions


def f64_to_f32(x) -> np.ndarray:
    """fp64 -> fp32, round to nearest even (numpy's cast)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def f32_to_bf16_bits(x32) -> np.ndarray:
    """fp32 -> bf16 bit pattern (uint16), round to nearest even on the 16 dropped bits.

    Inputs here are finite (for finite values the 32-bit sum below cannot overflow); NaN payloads
    are not handled.
    """
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def f64_to_bf16_bits(x) -> np.ndarray:
    return f32_to_bf16_bits(f64_to_f32(x))


def bf16_bits_to_f32(bits) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_bits_to_f64(bits) -> np.ndarray:
    return bf16_bits_to_f32(bits).astype(np.float64)


def sha256_of(arr: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(arr).tobytes()).hexdigest()


# ----------------------------------------------------------------------------------------------
# workload descriptions


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    Nq: int
    Nk: int
    d: int
    R: int
    dtype: str          # "fp32" or "bf16": storage of q, k, v, out, dout
    passes: str         # "fwd" or "fwd+bwd"
    seed: int
    std: float          # Q, K, V ~ std * N(0, 1)
    do_seed: int | None  # None: dO uses the Q/K/V seed
    do_std: float
    kind: str = "iid"   # "iid" or "turbulence"

    @property
    def scale(self) -> float:
        """Softmax scale 1/sqrt(d), as the fp32 value handed to the kernels."""
        return float(np.float32(1.0 / math.sqrt(self.d)))

    def gemm_unit(self) -> float:
        """U = 2 B H Nq Nk d: the flops of one of the two attention contractions."""
        return 2.0 * self.B * self.H * self.Nq * self.Nk * self.d


WORKLOADS = {
    w.name: w
    for w in [
        Workload("exact_fp32_n1k", 1, 2, 1024, 1024, 64, 4, "fp32", "fwd", 0, 1.0, None, 1.0),
        Workload("shard_n16k_d64", 1, 16, 16384, 16384, 64, 4, "bf16", "fwd+bwd", 1, 0.5, 2, 1.0),
        Workload("ring8_nk262k_d128", 1, 16, 32768, 262144, 128, 8, "bf16", "fwd+bwd", 3,
                 1.0 / math.sqrt(2.0), None, 1.0 / math.sqrt(2.0)),
        Workload("turbulence_nk262k_d64", 1, 16, 65536, 262144, 64, 4, "bf16", "fwd", 4, 1.0, None,
                 1.0, kind="turbulence"),
        Workload("long_nk524k_d128", 1, 16, 65536, 524288, 128, 8, "bf16", "fwd+bwd", 5,
                 1.0 / math.sqrt(2.0), None, 1.0 / math.sqrt(2.0)),
    ]
}


_TENSOR_ID = {"q": 0, "k": 1, "v": 2, "do": 3}


def slab(seed: int, tensor: str, b: int, h: int, N: int, d: int, std: float, store: str):
    """One (b, h) slab of `tensor`: std * N(0,1) from default_rng([seed, tensor id, b, h])."""
    x = np.random.default_rng([seed, _TENSOR_ID[tensor], b, h]).standard_normal((N, d)) * std
    return f64_to_f32(x) if store == "fp32" else f64_to_bf16_bits(x)


def _draw(seed, tensor, B, H, N, d, std, store, threads) -> np.ndarray:
    out = np.empty((B, H, N, d), dtype=np.float32 if store == "fp32" else np.uint16)

    def fill(bh):
        b, h = divmod(bh, H)
        out[b, h] = slab(seed, tensor, b, h, N, d, std, store)

    if threads <= 1 or B * H == 1:
        for bh in range(B * H):
            fill(bh)
    else:
        with concurrent.futures.ThreadPoolExecutor(threads) as ex:
            list(ex.map(fill, range(B * H)))
    return out


def make_iid(B, H, Nq, Nk, d, *, seed, std=1.0, store="bf16", with_do=True, do_seed=None,
             do_std=1.0, threads=None) -> dict:
    """i.i.d. Gaussian Q, K, V (and dO) with the common drawing rules.

    Returns {"q","k","v"[,"do"]}: float32 arrays for store="fp32", uint16 bf16 bits for "bf16".
    """
    threads = threads or min(16, os.cpu_count() or 1)
    t = {name: _draw(seed, name, B, H, n, d, std, store, threads)
         for name, n in (("q", Nq), ("k", Nk), ("v", Nk))}
    if with_do:
        t["do"] = _draw(seed if do_seed is None else do_seed, "do", B, H, Nq, d, do_std, store,
                        threads)
    return t


def to_f64(arr: np.ndarray, store: str) -> np.ndarray:
    """Exact fp64 value of a stored tensor (the oracle's input)."""
    return arr.astype(np.float64) if store == "fp32" else bf16_bits_to_f64(arr)


# ----------------------------------------------------------------------------------------------
# turbulence-shaped tokens


def turbulence_field(n: int = 256, seed: int = 4, kmax_damp: float = 100.0) -> np.ndarray:
    """Synthetic divergence-free velocity field u[c, z, y, x] (x fastest) on a periodic n^3 grid.

      wavenumbers k = fftfreq(n, 1/n) (integers); E(k) = k^(-5/3) exp(-k/kmax_damp), k = |k| > 0;
      amplitude a(k) = sqrt(E(|k|) / (4 pi |k|^2)), a(0) = 0, and 0 on every mode with a Nyquist
      component |k_i| = n/2;
      phases theta = default_rng(seed).uniform(0, 2pi, (3, n, n, n)); u_hat_c = a exp(i theta_c);
      Leray projection u_hat <- u_hat - k (k . u_hat) / |k|^2;
      u = Re(ifftn(u_hat)) per component, normalised to unit RMS over all components.
    """
    k1 = np.fft.fftfreq(n, 1.0 / n)
    kz, ky, kx = np.meshgrid(k1, k1, k1, indexing="ij")
    kk = np.sqrt(kx * kx + ky * ky + kz * kz)
    with np.errstate(divide="ignore", invalid="ignore"):
        E = np.where(kk > 0, kk ** (-5.0 / 3.0) * np.exp(-kk / kmax_damp), 0.0)
        amp = np.where(kk > 0, np.sqrt(E / (4.0 * np.pi * kk * kk)), 0.0)
    nyq = n // 2
    amp[(np.abs(kx) == nyq) | (np.abs(ky) == nyq) | (np.abs(kz) == nyq)] = 0.0
    theta = np.random.default_rng(seed).uniform(0.0, 2.0 * np.pi, (3, n, n, n))
    uh = amp[None] * np.exp(1j * theta)
    del theta
    kvec = (kx, ky, kz)  # component c = 0, 1, 2 is (x, y, z)
    with np.errstate(divide="ignore", invalid="ignore"):
        kdotu = kvec[0] * uh[0] + kvec[1] * uh[1] + kvec[2] * uh[2]
        fac = np.where(kk > 0, kdotu / (kk * kk), 0.0)
    for c in range(3):
        uh[c] = uh[c] - kvec[c] * fac
    del kdotu, fac
    u = np.empty((3, n, n, n), dtype=np.float64)
    for c in range(3):
        u[c] = np.real(np.fft.ifftn(uh[c]))
    u /= math.sqrt(float(np.mean(u * u)))
    return u


def patchify(u: np.ndarray, p: int) -> np.ndarray:
    """Tokens of p^3 patches: T[t, f], t = px + P (py + P pz), f = ((c p + iz) p + iy) p + ix."""
    C, n = u.shape[0], u.shape[1]
    P = n // p
    x = u.reshape(C, P, p, P, p, P, p)             # c, pz, iz, py, iy, px, ix
    x = x.transpose(1, 3, 5, 0, 2, 4, 6)           # pz, py, px, c, iz, iy, ix
    return np.ascontiguousarray(x.reshape(P * P * P, C * p * p * p))


def layer_norm(x: np.ndarray, eps: float = 1e-5) -> np.ndarray:
    """LayerNorm over the last axis, biased variance, no affine parameters."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def turbulence_qkv(n=256, p=4, width=1024, heads=16, nq=65536, field_seed=4,
                   embed_seed=40, proj_seeds=(41, 42, 43), block=16384) -> dict:
    """Q, K, V (bf16 bits, [1, heads, N, width/heads]) from turbulence tokens.

    Tokens T = patchify(turbulence_field(n), p); X = LayerNorm(T W_e), W_e ~ N(0, 1/F) of shape
    [F, width] from default_rng(embed_seed); W_q, W_k, W_v ~ N(0, 1/width) from proj_seeds;
    Q = X[:nq] W_q, K = X W_k, V = X W_v; feature f goes to head f // (width/heads).
    """
    T = patchify(turbulence_field(n, field_seed), p)
    ntok, F = T.shape
    We = np.random.default_rng(embed_seed).standard_normal((F, width)) / math.sqrt(F)
    Ws = [np.random.default_rng(s).standard_normal((width, width)) / math.sqrt(width)
          for s in proj_seeds]
    dh = width // heads
    out = {"q": np.empty((1, heads, nq, dh), np.uint16),
           "k": np.empty((1, heads, ntok, dh), np.uint16),
           "v": np.empty((1, heads, ntok, dh), np.uint16)}
    for t0 in range(0, ntok, block):
        t1 = min(ntok, t0 + block)
        X = layer_norm(T[t0:t1] @ We)
        for name, W in zip(("q", "k", "v"), Ws):
            if name == "q" and t0 >= nq:
                continue
            r1 = min(t1, nq) if name == "q" else t1
            Y = X[: r1 - t0] @ W                        # [rows, width]
            bits = f64_to_bf16_bits(Y).reshape(r1 - t0, heads, dh).transpose(1, 0, 2)
            out[name][0, :, t0:r1] = bits
    return out


# ----------------------------------------------------------------------------------------------


def cache_dir() -> str:
    return os.environ.get("RINGX_INPUT_CACHE", "/tmp/ringx_inputs")


def make_workload(name: str, use_cache: bool = True) -> dict:
    """Inputs of a named workload: {"q","k","v"[,"do"]} in their storage type (see make_iid)."""
    w = WORKLOADS[name]
    path = os.path.join(cache_dir(), name + ".npz")
    if use_cache and os.path.exists(path):
        with np.load(path, allow_pickle=False) as z:
            return {key: z[key] for key in z.files}
    if w.kind == "turbulence":
        t = turbulence_qkv(nq=w.Nq)
    else:
        t = make_iid(w.B, w.H, w.Nq, w.Nk, w.d, seed=w.seed, std=w.std, store=w.dtype,
                     with_do=(w.passes != "fwd"), do_seed=w.do_seed, do_std=w.do_std)
    if use_cache:
        os.makedirs(cache_dir(), exist_ok=True)
        tmp = path + f".tmp{os.getpid()}.npz"
        np.savez(tmp, **t)
        os.replace(tmp, path)
    return t
