"""Pins of the oracle's gradient and projection functions (CPU only).

Each test checks the oracle against something other than itself: hand-worked
values (tests/golden), pure-Python brute force, the Kronecker form of Eq. 1,
the closed form of Eq. 4, invariants that hold exactly, and the Monte-Carlo
unbiasedness of Gaussian projections.
"""
import numpy as np
import pytest

from golden_io import load
from oracle import gradients as og
from oracle import rng


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def test_eq1_worked_example():
    g = load("eq1_eq2_worked_example.json")
    A, B = np.array(g["A"], float), np.array(g["B"], float)
    np.testing.assert_array_equal(og.weight_gradient_loop(A, B), g["G"])
    np.testing.assert_array_equal(og.weight_gradient(A, B), g["G"])
    np.testing.assert_array_equal(og.vec_columns(og.weight_gradient(A, B)), g["vec_DW"])
    np.testing.assert_array_equal(og.kron_sum(A, B), g["vec_DW"])


def test_eq2_worked_example_both_routes():
    g = load("eq1_eq2_worked_example.json")
    A, B = np.array(g["A"], float), np.array(g["B"], float)
    P_in, P_out = np.array(g["P_in"], float), np.array(g["P_out"], float)
    phi_f = og.project_example([dict(A=A, B=B, P_in=P_in, P_out=P_out)], "factored")
    phi_m = og.project_example([dict(A=A, B=B, P_in=P_in, P_out=P_out)], "materialized")
    np.testing.assert_array_equal(phi_f, g["phi"])
    np.testing.assert_array_equal(phi_m, g["phi"])
    np.testing.assert_array_equal(og.project_brute_force(A, B, P_in, P_out).reshape(-1), g["phi"])


def test_eq1_loop_equals_matrix_form_and_kron():
    A, B = _rand((7, 5), 1), _rand((7, 3), 2)
    G = og.weight_gradient(A, B)
    np.testing.assert_allclose(og.weight_gradient_loop(A, B), G, rtol=0, atol=1e-13)
    np.testing.assert_allclose(og.kron_sum(A, B), og.vec_columns(G), rtol=0, atol=1e-13)
    # element formula by hand: DW[r, c] = sum_t B[t, r] A[t, c]
    for r in range(3):
        for c in range(5):
            assert abs(G[r, c] - sum(B[t, r] * A[t, c] for t in range(7))) < 1e-13


@pytest.mark.parametrize("shape", [(5, 6, 4, 3, 2), (1, 3, 2, 2, 3), (4, 8, 8, 4, 4)])
def test_brute_force_matches_factored_and_materialized(shape):
    T, d_in, d_out, k_in, k_out = shape
    A, B = _rand((T, d_in), 3), _rand((T, d_out), 4)
    P_in, P_out = _rand((d_in, k_in), 5), _rand((d_out, k_out), 6)
    bf = og.project_brute_force(A, B, P_in, P_out)
    np.testing.assert_allclose(og.project_factored(A, B, P_in, P_out), bf, rtol=0, atol=1e-12)
    G = og.weight_gradient_loop(A, B)
    np.testing.assert_allclose(og.project_materialized(G, P_in, P_out), bf, rtol=0, atol=1e-12)


def test_factored_equals_materialized_eq2():
    A, B = _rand((33, 40), 7), _rand((33, 24), 8)
    P_in, P_out = _rand((40, 12), 9), _rand((24, 5), 10)
    f = og.project_factored(A, B, P_in, P_out)
    m = og.project_materialized(og.weight_gradient(A, B), P_in, P_out)
    assert np.linalg.norm(f - m) / np.linalg.norm(m) < 1e-12
    # Eq. 2 in Kronecker form: (P_a (x) P_g) vec(DW), P_a = P_in^T, P_g = P_out^T
    kron = np.kron(P_in.T, P_out.T) @ og.vec_columns(og.weight_gradient(A, B))
    np.testing.assert_allclose(f.reshape(-1), kron, rtol=0, atol=1e-10)


def test_eq4_worked_example_and_loop():
    g = load("eq4_worked_example.json")
    args = [np.array(g[k], float) for k in ("A_i", "B_i", "A_j", "B_j")]
    assert og.ghost_dot(*args) == g["value"]
    assert og.ghost_dot_loop(*args) == g["value"]


def test_eq4_equals_frobenius_of_materialized():
    A_i, B_i = _rand((9, 6), 11), _rand((9, 4), 12)
    A_j, B_j = _rand((5, 6), 13), _rand((5, 4), 14)
    want = float(np.sum(og.weight_gradient(A_i, B_i) * og.weight_gradient(A_j, B_j)))
    assert abs(og.ghost_dot(A_i, B_i, A_j, B_j) - want) < 1e-11
    assert abs(og.ghost_dot_loop(A_i, B_i, A_j, B_j) - want) < 1e-11


def test_identity_projection_gives_ghost_dot():
    # k = d and P = I: phi_i = vec of (A^T B), so <phi_i, phi_j> must equal Eq. 4.
    d_in, d_out = 6, 5
    I_in, I_out = np.eye(d_in), np.eye(d_out)
    ex = [(_rand((8, d_in), 20 + s), _rand((8, d_out), 30 + s)) for s in range(3)]
    phis = [og.project_example([dict(A=A, B=B, P_in=I_in, P_out=I_out)]) for A, B in ex]
    for i in range(3):
        for j in range(3):
            want = og.ghost_dot(ex[i][0], ex[i][1], ex[j][0], ex[j][1])
            assert abs(float(phis[i] @ phis[j]) - want) < 1e-10 * max(1.0, abs(want))
    # and ||G_i||_F^2 is the diagonal
    G0 = og.weight_gradient(*ex[0])
    assert abs(float(phis[0] @ phis[0]) - float(np.sum(G0 * G0))) < 1e-10 * float(np.sum(G0 * G0))


def test_jl_unbiasedness_of_generated_maps():
    # E_P[<phi_i, phi_j>] = <G_i, G_j>_F when E[P P^T] = I on both sides.
    d_in, d_out, k_in, k_out, T = 5, 4, 3, 2, 6
    A_i, B_i = _rand((T, d_in), 40), _rand((T, d_out), 41)
    A_j, B_j = _rand((T, d_in), 42), _rand((T, d_out), 43)
    exact = float(np.sum(og.weight_gradient(A_i, B_i) * og.weight_gradient(A_j, B_j)))
    est = []
    for s in range(2000):
        P_in = rng.gaussian_map_f64(rng.side_seed(s, 0, 0), d_in, k_in)
        P_out = rng.gaussian_map_f64(rng.side_seed(s, 0, 1), d_out, k_out)
        fi = og.project_factored(A_i, B_i, P_in, P_out).reshape(-1)
        fj = og.project_factored(A_j, B_j, P_in, P_out).reshape(-1)
        est.append(float(fi @ fj))
    est = np.array(est)
    se = est.std(ddof=1) / np.sqrt(est.size)
    assert abs(est.mean() - exact) < 4 * se
    # a wrong scale (1/k instead of 1/sqrt(k) per side) would shrink the mean by k_in*k_out
    assert abs(est.mean() / (k_in * k_out) - exact) > 4 * se


def test_single_token_is_rank_one():
    A, B = _rand((1, 7), 50), _rand((1, 6), 51)
    P_in, P_out = _rand((7, 4), 52), _rand((6, 3), 53)
    psi = og.project_factored(A, B, P_in, P_out)
    np.testing.assert_allclose(psi, np.outer(P_in.T @ A[0], P_out.T @ B[0]), rtol=0, atol=1e-12)
    assert np.linalg.matrix_rank(psi) == 1


def test_token_split_additivity_and_permutation():
    A, B = _rand((19, 9), 60), _rand((19, 7), 61)
    P_in, P_out = _rand((9, 4), 62), _rand((7, 5), 63)
    full = og.project_factored(A, B, P_in, P_out)
    for s in (0, 1, 8, 16, 19):
        parts = og.project_factored(A[:s], B[:s], P_in, P_out) + og.project_factored(A[s:], B[s:], P_in, P_out)
        np.testing.assert_allclose(parts, full, rtol=0, atol=1e-12)
    perm = np.random.default_rng(0).permutation(19)
    np.testing.assert_allclose(og.project_factored(A[perm], B[perm], P_in, P_out), full, rtol=0, atol=1e-12)


def test_bilinearity_and_zero():
    A, B = _rand((6, 5), 70), _rand((6, 4), 71)
    A2 = _rand((6, 5), 72)
    P_in, P_out = _rand((5, 3), 73), _rand((4, 2), 74)
    f = lambda a, b: og.project_factored(a, b, P_in, P_out)  # noqa: E731
    np.testing.assert_allclose(f(2.5 * A - A2, B), 2.5 * f(A, B) - f(A2, B), rtol=0, atol=1e-12)
    np.testing.assert_allclose(f(A, -3.0 * B), -3.0 * f(A, B), rtol=0, atol=1e-12)
    assert not np.any(f(np.zeros_like(A), B))
    assert not np.any(f(A, np.zeros_like(B)))


def test_lengths_equal_truncation():
    A, B = _rand((12, 5), 80), _rand((12, 3), 81)
    P_in, P_out = _rand((5, 2), 82), _rand((3, 2), 83)
    for L in (0, 1, 7, 12):
        np.testing.assert_array_equal(og.project_factored(A, B, P_in, P_out, L),
                                      og.project_factored(A[:L], B[:L], P_in, P_out))
        np.testing.assert_array_equal(og.weight_gradient(A, B, L), og.weight_gradient(A[:L], B[:L]))
    assert not np.any(og.project_factored(A, B, P_in, P_out, 0))
    with pytest.raises(ValueError):
        og.project_factored(A, B, P_in, P_out, 13)


def test_feature_vector_layer_order_and_aggregation():
    blocks = [_rand((2, 3), 90), _rand((4, 1), 91)]
    phi = og.feature_vector(blocks)
    np.testing.assert_array_equal(phi[:6], blocks[0].reshape(-1))
    np.testing.assert_array_equal(phi[6:], blocks[1].reshape(-1))
    other = [_rand((2, 3), 92), _rand((4, 1), 93)]
    # inner product of concatenations = sum of per-layer inner products
    want = sum(float(np.sum(a * b)) for a, b in zip(blocks, other))
    assert abs(float(phi @ og.feature_vector(other)) - want) < 1e-12
