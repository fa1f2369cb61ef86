"""Seeded input generators: storage conversions, determinism, turbulence field, patchify."""

import math

import numpy as np
import pytest
import torch

from paper_2507_16697_amd import inputs


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100_000) * 10.0 ** rng.integers(-30, 30, 100_000),
                        [0.0, -0.0, 1.0, -1.0, 1.00390625, 1.0078125, 1.01171875, 3.0e38, 1e-40]])
    x32 = x.astype(np.float32)
    ours = inputs.f32_to_bf16_bits(x32)
    ref = torch.from_numpy(x32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = inputs.bf16_bits_to_f32(ours)
    np.testing.assert_array_equal(back, torch.from_numpy(x32).to(torch.bfloat16).float().numpy())


def test_ties_round_to_even():
    # 1 + 2^-8 lies halfway between bf16 neighbours 1 and 1 + 2^-7: ties go to the even mantissa.
    assert inputs.bf16_bits_to_f32(inputs.f64_to_bf16_bits(1.0 + 2.0 ** -8))[()] == 1.0
    assert inputs.bf16_bits_to_f32(inputs.f64_to_bf16_bits(1.0 + 3 * 2.0 ** -8))[()] == 1.0 + 2.0 ** -6


def test_seeded_draws_are_deterministic():
    a = inputs.make_iid(1, 2, 33, 45, 8, seed=9, std=0.5, store="bf16")
    b = inputs.make_iid(1, 2, 33, 45, 8, seed=9, std=0.5, store="bf16")
    for key in a:
        assert inputs.sha256_of(a[key]) == inputs.sha256_of(b[key])
    c = inputs.make_iid(1, 2, 33, 45, 8, seed=10, std=0.5, store="bf16")
    assert inputs.sha256_of(a["q"]) != inputs.sha256_of(c["q"])


def test_each_slab_is_its_own_stream():
    B, H, nq, nk, d = 2, 3, 5, 7, 4
    t = inputs.make_iid(B, H, nq, nk, d, seed=3, std=0.5, do_std=0.5, store="fp32", threads=4)
    for name, n, tid in (("q", nq, 0), ("k", nk, 1), ("v", nk, 2), ("do", nq, 3)):
        for b in range(B):
            for h in range(H):
                ref = np.random.default_rng([3, tid, b, h]).standard_normal((n, d)) * 0.5
                np.testing.assert_array_equal(t[name][b, h], ref.astype(np.float32))
    assert not np.array_equal(t["q"][0, 0], t["q"][0, 1])
    serial = inputs.make_iid(B, H, nq, nk, d, seed=3, std=0.5, store="bf16", threads=1)
    parallel = inputs.make_iid(B, H, nq, nk, d, seed=3, std=0.5, store="bf16", threads=5)
    for name in serial:
        np.testing.assert_array_equal(serial[name], parallel[name])


def test_separate_do_seed():
    t = inputs.make_iid(1, 1, 4, 6, 2, seed=1, std=0.5, store="fp32", do_seed=2, do_std=1.0)
    ref = np.random.default_rng([2, 3, 0, 0]).standard_normal((4, 2)).astype(np.float32)
    np.testing.assert_array_equal(t["do"][0, 0], ref)


def test_workload_table():
    w = inputs.WORKLOADS["ring8_nk262k_d128"]
    assert (w.B, w.H, w.Nq, w.Nk, w.d, w.R) == (1, 16, 32768, 262144, 128, 8)
    assert w.gemm_unit() == pytest.approx(3.518437e13, rel=1e-6)
    assert w.scale == np.float32(1 / math.sqrt(128))
    for w in inputs.WORKLOADS.values():
        assert w.Nk % w.R == 0 and w.Nq >= 1


def test_turbulence_field_properties():
    n = 32
    u = inputs.turbulence_field(n=n, seed=4)
    assert u.shape == (3, n, n, n) and np.isrealobj(u)
    assert math.isclose(float(np.mean(u * u)), 1.0, rel_tol=1e-12)
    uh = np.stack([np.fft.fftn(u[c]) for c in range(3)])
    k1 = np.fft.fftfreq(n, 1.0 / n)
    kz, ky, kx = np.meshgrid(k1, k1, k1, indexing="ij")
    div = kx * uh[0] + ky * uh[1] + kz * uh[2]
    assert np.max(np.abs(div)) <= 1e-10 * np.max(np.abs(uh))
    # shell-summed energy follows k^(-5/3) (damping exp(-k/100) is ~1 here)
    kk = np.sqrt(kx ** 2 + ky ** 2 + kz ** 2)
    e = 0.5 * np.sum(np.abs(uh) ** 2, axis=0)
    shells = np.arange(2, 12)
    Ek = np.array([e[(kk >= s - 0.5) & (kk < s + 0.5)].sum() for s in shells])
    slope = np.polyfit(np.log(shells), np.log(Ek), 1)[0]
    assert -1.95 < slope < -1.40, slope


def test_patchify_index_map():
    n, p, C = 8, 2, 3
    c, z, y, x = np.meshgrid(np.arange(C), np.arange(n), np.arange(n), np.arange(n), indexing="ij")
    u = (c * 1000000 + z * 10000 + y * 100 + x).astype(np.float64)
    T = inputs.patchify(u, p)
    P = n // p
    assert T.shape == (P ** 3, C * p ** 3)
    for t in [0, 1, P, P * P, P ** 3 - 1, 37]:
        px, py, pz = t % P, (t // P) % P, t // (P * P)
        for f in [0, 1, p, p * p, p ** 3, C * p ** 3 - 1, 13]:
            ix, iy, iz, cc = f % p, (f // p) % p, (f // (p * p)) % p, f // (p ** 3)
            assert T[t, f] == u[cc, pz * p + iz, py * p + iy, px * p + ix]


def test_layer_norm():
    x = np.random.default_rng(1).standard_normal((5, 64)) * 3 + 2
    y = inputs.layer_norm(x)
    np.testing.assert_allclose(y.mean(axis=1), 0, atol=1e-12)
    np.testing.assert_allclose((y ** 2).mean(axis=1), 1, rtol=1e-4)


def test_turbulence_qkv_small():
    t = inputs.turbulence_qkv(n=16, p=2, width=64, heads=4, nq=100, block=128)
    assert t["q"].shape == (1, 4, 100, 16) and t["k"].shape == (1, 4, 512, 16)
    # Q and K come from the same tokens through different projections: recompute one row
    T = inputs.patchify(inputs.turbulence_field(16, 4), 2)
    We = np.random.default_rng(40).standard_normal((24, 64)) / math.sqrt(24)
    Wq = np.random.default_rng(41).standard_normal((64, 64)) / math.sqrt(64)
    X = inputs.layer_norm(T[:3] @ We)
    ref = inputs.f64_to_bf16_bits(X @ Wq)            # [3, 64]
    np.testing.assert_array_equal(t["q"][0, 1, :3], ref[:, 16:32])
