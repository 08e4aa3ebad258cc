"""Pins of the oracle's projection generator (CPU only).

The paper fixes no generator (App. A.2 only requires per-layer, per-side seeds
held fixed); the oracle's generator is pinned to the published definitions of
Philox4x32-10 and SplitMix64 through their known-answer values, to the N(0, 1)
law through moments, and to RNE bf16 rounding through torch's conversion and
hand-picked halfway cases.
"""
import numpy as np
import pytest
import torch

from golden_io import load
from oracle import rng


def test_philox_known_answers():
    kat = load("philox4x32_10_kat.json")
    for v in kat["vectors"]:
        c = [int(x, 16) for x in v["ctr"]]
        k = [int(x, 16) for x in v["key"]]
        out = rng.philox4x32_10(*c, *k)
        assert [int(o) for o in out] == [int(x, 16) for x in v["out"]]


def test_philox_vectorised_matches_scalar():
    ctr = np.arange(5, dtype=np.uint64) * np.uint64(0x01000193)
    vec = rng.philox4x32_10(ctr, ctr + np.uint64(7), ctr ^ np.uint64(3), ctr, 0x1234, 0xABCD)
    for i in range(5):
        one = rng.philox4x32_10(int(ctr[i]), int(ctr[i]) + 7, int(ctr[i]) ^ 3, int(ctr[i]), 0x1234, 0xABCD)
        assert [int(o) for o in one] == [int(v[i]) for v in vec]


def test_splitmix64_reference_stream():
    g = load("splitmix64_seed0.json")
    s = int(g["state0"], 16)
    for want in g["outputs"]:
        s, out = rng.splitmix64_next(s)
        assert out == int(want, 16)


def test_side_seeds_distinct_and_stable():
    seeds = {rng.side_seed(0, layer, side) for layer in range(64) for side in (0, 1)}
    assert len(seeds) == 128
    assert rng.side_seed(5, 3, 1) == rng.side_seed(5, 3, 1)
    assert rng.side_seed(5, 3, 1) != rng.side_seed(6, 3, 1)
    with pytest.raises(ValueError):
        rng.side_seed(0, 0, 2)


def test_gaussian_moments():
    z = rng.gaussian_map_f64(rng.side_seed(11, 0, 0), 400_000, 1).ravel()
    n = z.size
    assert abs(z.mean()) < 5 / np.sqrt(n)
    assert abs(z.var() - 1.0) < 5 * np.sqrt(2.0 / n)
    kurt = np.mean(z ** 4) / z.var() ** 2
    assert abs(kurt - 3.0) < 5 * np.sqrt(24.0 / n)
    # symmetric tails: P(|z| > 1.96) ~ 0.05
    tail = np.mean(np.abs(z) > 1.959963984540054)
    assert abs(tail - 0.05) < 5 * np.sqrt(0.05 * 0.95 / n)


def test_map_scale_is_one_over_sqrt_k():
    k = 16
    P = rng.gaussian_map_f64(rng.side_seed(2, 1, 1), 20_000, k)
    assert abs(P.var() * k - 1.0) < 0.02
    # columns are independent: E[P^T P] = I
    PtP = P.T @ P / P.shape[0] * k
    assert np.max(np.abs(PtP - np.eye(k))) < 0.06


def test_uniforms_in_open_closed_ranges():
    # extreme words: u1 never 0 (log finite), u2 < 1
    zero = np.zeros(1, dtype=np.uint32)
    ones = np.full(1, 0xFFFFFFFF, dtype=np.uint32)
    z_min = rng.box_muller(zero, zero, zero, zero)  # u1 = 2^-53, u2 = 0
    assert np.isfinite(z_min).all() and z_min[0] > 8.0
    z_max = rng.box_muller(ones, ones, zero, zero)  # u1 = 1 -> z = 0
    assert z_max[0] == 0.0


def test_bf16_rounding_matches_torch_rne():
    x = np.random.default_rng(0).standard_normal(100_000).astype(np.float32) * 37.0
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(rng.round_bf16_from_f32(x), want)


def test_bf16_rounding_halfway_cases():
    # 1 + 2^-8 lies halfway between bf16 neighbours 1 and 1 + 2^-7: ties to even (1)
    # 1 + 3*2^-8 lies halfway between 1 + 2^-7 and 1 + 2^-6: ties to even (1 + 2^-6)
    x = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 1 + 2 ** -8 + 2 ** -20], dtype=np.float32)
    got = rng.round_bf16_from_f32(x)
    np.testing.assert_array_equal(got, np.array([1.0, 1 + 2 ** -6, -1.0, 1 + 2 ** -7], dtype=np.float32))


def test_projection_pair_dtypes():
    p32_in, p32_out = rng.projection_pair(0, 0, 64, 48, 8, 4, "f32")
    pb_in, pb_out = rng.projection_pair(0, 0, 64, 48, 8, 4, "bf16")
    assert p32_in.shape == (64, 8) and p32_out.shape == (48, 4)
    # bf16 values are exactly representable: their low 16 float32 bits are zero
    bits = pb_in.astype(np.float32).view(np.uint32)
    assert np.all(bits & 0xFFFF == 0)
    assert np.max(np.abs(pb_in - p32_in) / np.abs(p32_in).max()) < 2 ** -7
    # the two sides of a layer, and two layers, draw different maps
    q_in, _ = rng.projection_pair(0, 1, 64, 48, 8, 4, "f32")
    assert not np.allclose(p32_in, q_in)


def test_rademacher_entries_and_signs():
    # every entry is exactly +-1/sqrt(k); its sign is bit 31 of the first Philox
    # word of its counter, checked against the scalar known-answer path
    seed = rng.side_seed(3, 2, 1)
    d, k = 37, 8
    P = rng.rademacher_map_f64(seed, d, k)
    assert np.all(np.abs(P) == 1.0 / np.sqrt(8.0))
    for v, c in ((0, 0), (5, 3), (36, 7)):
        e = v * k + c
        x0 = rng.philox4x32_10(e & 0xFFFFFFFF, e >> 32, 0, 0, seed & 0xFFFFFFFF, seed >> 32)[0]
        assert (P[v, c] < 0) == bool(int(x0) >> 31)
    big = rng.rademacher_map_f64(rng.side_seed(7, 0, 0), 4096, 64)
    frac = np.mean(big > 0)
    assert abs(frac - 0.5) < 5 * 0.5 / np.sqrt(big.size)  # balanced signs (5 sigma)


def test_rademacher_projection_unbiased():
    # E[<P^T x, P^T y>] = <x, y> over maps (independent entries of variance 1/k)
    gen = np.random.default_rng(0)
    d, k = 40, 16
    x, y = gen.standard_normal(d), gen.standard_normal(d)
    vals = [float((rng.rademacher_map_f64(rng.side_seed(s, 0, 0), d, k).T @ x)
                  @ (rng.rademacher_map_f64(rng.side_seed(s, 0, 0), d, k).T @ y)) for s in range(400)]
    mean, sd = np.mean(vals), np.std(vals) / np.sqrt(len(vals))
    assert abs(mean - float(x @ y)) < 5 * sd
    # column norms are exactly d/k
    P = rng.rademacher_map_f64(rng.side_seed(1, 0, 1), d, k)
    assert np.allclose(np.sum(P * P, axis=0), d / k, rtol=0, atol=1e-12)


def test_projection_pair_kinds():
    g = rng.projection_pair(5, 1, 20, 12, 4, 8, "bf16")
    r = rng.projection_pair(5, 1, 20, 12, 4, 8, "bf16", kind="rademacher")
    assert np.all(np.abs(r[0]) == rng.round_to_dtype(np.array([0.5]), "bf16")[0])
    assert np.all(np.sign(r[1]) != 0) and not np.allclose(g[1], r[1])
    with pytest.raises(KeyError):
        rng.projection_pair(5, 1, 20, 12, 4, 8, "bf16", kind="sparse")
