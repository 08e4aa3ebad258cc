"""Pins of the cross-Gram oracle (oracle/crossgram.py) against what the paper and
the mathematics fix: Eq. 4's hand-worked value, brute force over Eq. 1, route
equality, symmetry / positive semi-definiteness with the squared norms on the
diagonal, identity projection (Eq. 2 with P = I), the T = 1 rank-one case,
lengths = truncation, bilinearity, and the route FLOP counts against the
leading terms of the App. A.4 table."""
import numpy as np
import pytest

from golden_io import load as load_golden
from oracle import cost as oc
from oracle import crossgram as ocg
from oracle import gradients as og


def _batch(rng, n, T, dims, lengths=False):
    out = []
    for d_in, d_out in dims:
        A = rng.standard_normal((n, T, d_in))
        B = rng.standard_normal((n, T, d_out))
        L = rng.integers(0, T + 1, n) if lengths else None
        out.append((A, B, L))
    return out


DIMS = [(5, 3), (2, 7), (4, 4)]


def test_eq4_worked_example():
    g = load_golden("eq4_worked_example.json")
    b1 = [(np.array([g["A_i"]]), np.array([g["B_i"]]), None)]
    b2 = [(np.array([g["A_j"]]), np.array([g["B_j"]]), None)]
    for route in ("factorized", "materialized"):
        assert ocg.cross_gram(b1, b2, route)[0, 0] == g["value"]


def test_brute_force_tiny():
    rng = np.random.default_rng(1)
    b1 = _batch(rng, 3, 4, DIMS[:2], lengths=True)
    b2 = _batch(rng, 2, 3, DIMS[:2], lengths=True)
    ref = ocg.cross_gram_brute_force(b1, b2)
    for route in ("factorized", "materialized"):
        np.testing.assert_allclose(ocg.cross_gram(b1, b2, route), ref, rtol=1e-12, atol=1e-12)


def test_routes_agree_unequal_batches_and_lengths():
    rng = np.random.default_rng(2)
    b1 = _batch(rng, 5, 9, DIMS, lengths=True)
    b2 = _batch(rng, 3, 6, DIMS, lengths=True)
    Kf = ocg.cross_gram(b1, b2, "factorized")
    Km = ocg.cross_gram(b1, b2, "materialized")
    assert Kf.shape == (5, 3)
    np.testing.assert_allclose(Kf, Km, rtol=1e-12, atol=1e-10)


def test_gram_symmetric_psd_diagonal_is_sq_norm():
    rng = np.random.default_rng(3)
    b = _batch(rng, 6, 5, DIMS, lengths=True)
    K = ocg.cross_gram(b, b)
    np.testing.assert_allclose(K, K.T, rtol=1e-12, atol=1e-10)
    assert np.linalg.eigvalsh(K).min() >= -1e-9 * np.abs(K).max()
    for route in ("factorized", "materialized"):
        np.testing.assert_allclose(np.diag(K), ocg.sq_norms(b, route), rtol=1e-12)


def test_identity_projection_reproduces_cross_gram():
    # Eq. 2 with P_a = I, P_g = I: projected features are vec(DW) in Kronecker
    # order, so their inner products are the cross-Gram of Eq. 4
    rng = np.random.default_rng(4)
    b1 = _batch(rng, 3, 4, DIMS)
    b2 = _batch(rng, 2, 6, DIMS)
    def phi(batch, i):
        return og.feature_vector([og.project_factored(A[i], B[i], np.eye(A.shape[2]), np.eye(B.shape[2]))
                                  for A, B, _ in batch])
    F1 = np.stack([phi(b1, i) for i in range(3)])
    F2 = np.stack([phi(b2, j) for j in range(2)])
    np.testing.assert_allclose(F1 @ F2.T, ocg.cross_gram(b1, b2), rtol=1e-12, atol=1e-10)


def test_single_token_is_rank_one_product():
    rng = np.random.default_rng(5)
    b1 = _batch(rng, 2, 1, DIMS[:1])
    b2 = _batch(rng, 3, 1, DIMS[:1])
    (A1, B1, _), (A2, B2, _) = b1[0], b2[0]
    want = (A1[:, 0] @ A2[:, 0].T) * (B1[:, 0] @ B2[:, 0].T)
    np.testing.assert_allclose(ocg.cross_gram(b1, b2), want, rtol=1e-12)


def test_lengths_equal_truncation_and_zero_length():
    rng = np.random.default_rng(6)
    A1, B1 = rng.standard_normal((2, 7, 4)), rng.standard_normal((2, 7, 3))
    A2, B2 = rng.standard_normal((1, 5, 4)), rng.standard_normal((1, 5, 3))
    K = ocg.cross_gram([(A1, B1, [3, 0])], [(A2, B2, [4])])
    K_trunc = ocg.cross_gram([(A1[:1, :3], B1[:1, :3], None)], [(A2[:, :4], B2[:, :4], None)])
    assert K[0, 0] == pytest.approx(K_trunc[0, 0], rel=1e-12)
    assert K[1, 0] == 0.0


def test_bilinear_and_zero():
    rng = np.random.default_rng(7)
    b1 = _batch(rng, 2, 4, DIMS[:2])
    b2 = _batch(rng, 2, 4, DIMS[:2])
    K = ocg.cross_gram(b1, b2)
    scaled = [(A * 2.0, B * 3.0, L) for A, B, L in b1]
    np.testing.assert_allclose(ocg.cross_gram(scaled, b2), 6.0 * K, rtol=1e-12)
    zero = [(A, B * 0.0, L) for A, B, L in b2]
    assert not ocg.cross_gram(b1, zero).any()


def test_route_flop_counts():
    # hand-derived: one pair, T = 2, d_in = 3, d_out = 5: two 2x2 Grams over 3 and 5
    # features (2*4*3 + 2*4*5) and the 4-entry product sum (2*4) -> 72
    assert oc.crossgram_flops_factorized(1, 1, 2, 2, 3, 5) == 72
    # G for 2 examples (2 * 2 * 2*3*5 = 120) and one Frobenius product (2*15) -> 150
    assert oc.crossgram_flops_materialized(1, 1, 2, 2, 3, 5) == 150
    # leading terms of the App. A.4 table (times 2 for multiply-add)
    n1, n2, T, Ni, No = 8, 1, 2048, 1024, 4096
    f = oc.crossgram_flops_factorized(n1, n2, T, T, Ni, No)
    m = oc.crossgram_flops_materialized(n1, n2, T, T, Ni, No)
    assert f / (2 * oc.crossgram_factorized(n1, n2, T, Ni, No)) == pytest.approx(1.0, rel=1e-3)
    assert m / (2 * oc.crossgram_materialized(n1, n2, T, Ni, No)) == pytest.approx(1.0, rel=1e-12)
    # the regimes of App. A.4: short sequences favour the factorized route,
    # long ones the materialized route, for this layer and batch
    assert oc.crossgram_flops_factorized(8, 1, 32, 32, Ni, No) < oc.crossgram_flops_materialized(8, 1, 32, 32, Ni, No)
    assert f > m
