"""Pins of the random-mask oracle (oracle/mask.py): gathered entries equal the
dense weight gradient of Eq. 1 at the mask's coordinates; masks are disjoint,
sorted, of the requested size and stable; the draw is uniform over the
entries (frequency test over many seeds); masked inner products are the
Frobenius product restricted to the mask."""
import numpy as np
import pytest

from oracle import gradients as og
from oracle import mask as om


def test_gather_equals_dense_gradient_entries():
    rng = np.random.default_rng(0)
    T, d_in, d_out = 9, 13, 7
    A, B = rng.standard_normal((T, d_in)), rng.standard_normal((T, d_out))
    rows, cols = om.mask_indices(3, 2, d_in, d_out, 20, 1)
    G = og.weight_gradient(A, B)
    np.testing.assert_allclose(om.masked_gradient(A, B, rows, cols), G[rows, cols], rtol=1e-13)
    np.testing.assert_allclose(om.masked_gradient_loop(A, B, rows, cols), G[rows, cols], rtol=1e-13)
    Gl = og.weight_gradient(A, B, 4)
    np.testing.assert_allclose(om.masked_gradient(A, B, rows, cols, 4), Gl[rows, cols], rtol=1e-13)


def test_masks_disjoint_sorted_stable():
    d_in, d_out, m = 64, 48, 100
    masks = [om.mask_indices(11, 5, d_in, d_out, m, j) for j in range(10)]
    flat = [c * d_out + r for r, c in masks]
    for f in flat:
        assert len(f) == m and np.all(np.diff(f) > 0)
        assert np.all((f >= 0) & (f < d_in * d_out))
    allf = np.concatenate(flat)
    assert len(np.unique(allf)) == 10 * m  # pairwise disjoint
    r, c = om.mask_indices(11, 5, d_in, d_out, m, 3)
    np.testing.assert_array_equal(r, masks[3][0])  # deterministic
    r2, _ = om.mask_indices(11, 6, d_in, d_out, m, 3)
    assert not np.array_equal(r2, r)  # per-layer seeds differ
    with pytest.raises(ValueError):
        om.mask_indices(11, 5, 4, 4, 9, 0)  # more than half the entries


def test_draw_is_uniform():
    # every entry of a 6 x 5 gradient is kept with probability m / 30
    d_in, d_out, m, seeds = 6, 5, 3, 3000
    counts = np.zeros(d_in * d_out)
    for s in range(seeds):
        r, c = om.mask_indices(s, 0, d_in, d_out, m, 0)
        counts[c * d_out + r] += 1
    p = m / (d_in * d_out)
    sd = np.sqrt(seeds * p * (1 - p))
    assert np.max(np.abs(counts - seeds * p)) < 5 * sd


def test_masked_inner_product_is_restricted_frobenius():
    rng = np.random.default_rng(1)
    Ai, Bi = rng.standard_normal((6, 10)), rng.standard_normal((6, 8))
    Aj, Bj = rng.standard_normal((4, 10)), rng.standard_normal((4, 8))
    rows, cols = om.mask_indices(2, 0, 10, 8, 30, 0)
    vi, vj = om.masked_gradient(Ai, Bi, rows, cols), om.masked_gradient(Aj, Bj, rows, cols)
    Gi, Gj = og.weight_gradient(Ai, Bi), og.weight_gradient(Aj, Bj)
    M = np.zeros_like(Gi)
    M[rows, cols] = 1.0
    assert np.isclose(vi @ vj, np.sum(Gi * Gj * M), rtol=1e-12)
