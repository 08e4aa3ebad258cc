"""Pins of the oracle's scoring and top-k (CPU only)."""
import numpy as np
import pytest

from oracle import scoring as osc


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def test_score_matches_loops_with_and_without_diag():
    Q, X = _rand((3, 7), 1), _rand((5, 7), 2)
    d = np.exp(_rand(7, 3))
    np.testing.assert_allclose(osc.score(Q, X), osc.score_loop(Q, X), rtol=0, atol=1e-12)
    np.testing.assert_allclose(osc.score(Q, X, d), osc.score_loop(Q, X, d), rtol=0, atol=1e-12)


def test_score_is_graddot_and_linear_in_d():
    Q, X = _rand((4, 6), 4), _rand((9, 6), 5)
    for q in range(4):
        for j in range(9):
            assert abs(osc.score(Q, X)[q, j] - float(Q[q] @ X[j])) < 1e-12
    d1, d2 = np.exp(_rand(6, 6)), np.exp(_rand(6, 7))
    np.testing.assert_allclose(osc.score(Q, X, 2 * d1 + d2), 2 * osc.score(Q, X, d1) + osc.score(Q, X, d2),
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(osc.score(Q, X, np.ones(6)), osc.score(Q, X), rtol=0, atol=0)


def _brute_topk(row, k):
    order = sorted(range(len(row)), key=lambda j: (-row[j], j))[:k]
    return order, [row[j] for j in order]


def test_topk_matches_brute_force_with_ties():
    rng_ = np.random.default_rng(8)
    S = rng_.integers(-3, 4, size=(6, 40)).astype(np.float64)  # heavy ties
    idx, val = osc.topk(S, 11)
    for q in range(6):
        bi, bv = _brute_topk(list(S[q]), 11)
        assert list(idx[q]) == bi
        assert list(val[q]) == bv


def test_topk_edges():
    S = np.zeros((2, 5))
    idx, _ = osc.topk(S, 5)
    assert idx.tolist() == [[0, 1, 2, 3, 4]] * 2  # all equal -> index order
    idx, val = osc.topk(S, 0)
    assert idx.shape == (2, 0) and val.shape == (2, 0)
    with pytest.raises(ValueError):
        osc.topk(S, 6)
    S = np.array([[1.0, -0.0, 0.0, -1.0]])
    idx, _ = osc.topk(S, 3)
    assert idx.tolist() == [[0, 1, 2]]  # -0.0 and 0.0 compare equal


def test_cosine_against_loops_and_invariants():
    rng = np.random.default_rng(3)
    Q = rng.standard_normal((3, 7))
    X = rng.standard_normal((5, 7))
    X[2] = 0.0  # a zero row scores 0
    d = np.exp(rng.standard_normal(7))
    for dd in (None, d):
        S = osc.cosine_scores(Q, X, dd)
        np.testing.assert_allclose(S, osc.cosine_loop(Q, X, dd), rtol=1e-12, atol=1e-15)
        assert np.all(np.abs(S) <= 1 + 1e-12)  # Cauchy-Schwarz
        assert np.all(S[:, 2] == 0)
        # invariant to positive row scalings of either side
        S2 = osc.cosine_scores(Q * np.array([[2.0], [0.5], [7.0]]), X * 3.0, dd)
        np.testing.assert_allclose(S2, S, rtol=1e-12, atol=1e-15)
    # identical rows have cosine 1; opposite rows -1; with d, the preconditioned query matters
    np.testing.assert_allclose(osc.cosine_scores(X[:2], X[:2]).diagonal(), 1.0, rtol=1e-14)
    np.testing.assert_allclose(osc.cosine_scores(X[:2], -X[:2]).diagonal(), -1.0, rtol=1e-14)
    np.testing.assert_allclose(osc.cosine_scores(Q / d, Q * 1.0, d).diagonal(), 1.0, rtol=1e-13)
    # the dot-product scores divided by the two norms
    S = osc.cosine_scores(Q, X[:2], d)
    ref = osc.score(Q, X[:2], d) / np.linalg.norm(Q * d, axis=1)[:, None] / np.linalg.norm(X[:2], axis=1)[None, :]
    np.testing.assert_allclose(S, ref, rtol=1e-12)
