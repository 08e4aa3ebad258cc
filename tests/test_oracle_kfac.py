"""Pins of the K-FAC / EK-FAC oracle (oracle/kfac.py) against the definitions of
the cited methods and what the mathematics fixes: token-loop factor sums, the
explicit Kronecker solve, EK-FAC eigenvalues as the diagonal of the second
moment in the Kronecker eigenbasis, EK-FAC = K-FAC for a product design, the
closed-form mean eigenvalues behind App. B's damping rule, the scalar case,
identity factors, the large-damping limit, self-adjointness and definiteness."""
import numpy as np
import pytest

from oracle import gradients as og
from oracle import kfac as ok


def _layer(rng, n, T, d_in, d_out, k_in, k_out, lengths=False):
    A = rng.standard_normal((n, T, d_in)) * rng.uniform(0.2, 3.0, d_in)
    B = rng.standard_normal((n, T, d_out)) * rng.uniform(0.2, 3.0, d_out)
    P_in = rng.standard_normal((d_in, k_in)) / np.sqrt(k_in)
    P_out = rng.standard_normal((d_out, k_out)) / np.sqrt(k_out)
    L = rng.integers(0, T + 1, n) if lengths else None
    return dict(A=A, B=B, P_in=P_in, P_out=P_out, lengths=L)


def _psis(L):
    lens = L["lengths"]
    return [og.project_factored(L["A"][i], L["B"][i], L["P_in"], L["P_out"],
                                None if lens is None else int(lens[i]))
            for i in range(L["A"].shape[0])]


def test_factor_sums_token_loop_and_lengths():
    rng = np.random.default_rng(0)
    L = _layer(rng, 3, 5, 6, 4, 3, 2, lengths=True)
    SA, SG, nt, ne = ok.factor_sums(L["A"], L["B"], L["P_in"], L["P_out"], L["lengths"])
    SA2, SG2, nt2, ne2 = ok.factor_sums_loop(L["A"], L["B"], L["P_in"], L["P_out"], L["lengths"])
    assert np.allclose(SA, SA2, rtol=1e-13, atol=1e-13) and np.allclose(SG, SG2, rtol=1e-13, atol=1e-13)
    assert nt == nt2 == int(np.sum(L["lengths"])) and ne == ne2 == 3
    # linearity: projecting the unprojected second moment gives the same sums
    M = sum(L["A"][i][: L["lengths"][i]].T @ L["A"][i][: L["lengths"][i]] for i in range(3))
    assert np.allclose(SA, L["P_in"].T @ M @ L["P_in"], rtol=1e-12, atol=1e-12)
    assert np.allclose(SA, SA.T) and np.allclose(SG, SG.T)


def test_scalar_case_closed_form():
    # k_in = k_out = 1: A = mean a~^2, S = sum g~^2 / N, E = A S, delta = 0.1 A S
    rng = np.random.default_rng(1)
    L = _layer(rng, 4, 3, 5, 2, 1, 1)
    a = np.einsum("ntd,dk->ntk", L["A"], L["P_in"])[..., 0]
    g = np.einsum("ntd,dk->ntk", L["B"], L["P_out"])[..., 0]
    C = ok.fit_layers([L])[0]
    A_ = np.mean(a ** 2)
    S_ = np.sum(g ** 2) / 4
    assert np.isclose(C.E_kfac[0, 0], A_ * S_, rtol=1e-12)
    psi = np.array([[2.5]])
    assert np.isclose(C.precondition(psi, "kfac")[0, 0], 2.5 / (1.1 * A_ * S_), rtol=1e-12)


@pytest.mark.parametrize("k_in,k_out", [(3, 2), (2, 4), (4, 4)])
def test_kfac_matches_kronecker_solve(k_in, k_out):
    rng = np.random.default_rng(2 + k_in)
    L = _layer(rng, 5, 6, 7, 5, k_in, k_out, lengths=True)
    C = ok.fit_layers([L])[0]
    # the factors' eigendecompositions reproduce them
    assert np.allclose(C.Q_a @ np.diag(C.lam_a) @ C.Q_a.T, C.A, rtol=1e-12, atol=1e-12)
    assert np.allclose(C.Q_g.T @ C.Q_g, np.eye(k_out), atol=1e-12)
    assert np.all(np.diff(C.lam_a) >= 0) and np.all(np.diff(C.lam_g) >= 0)
    X = rng.standard_normal((k_in, k_out))
    for rel, abs_ in ((0.1, 0.0), (0.0, 0.3), (0.5, 1e-3)):
        delta = ok.damping(C.E_kfac, rel, abs_)
        want = ok.kfac_dense_precondition(X, C.A, C.S, delta)
        got = C.precondition(X, "kfac", rel, abs_)
        assert np.allclose(got, want, rtol=1e-10, atol=1e-12)


def test_ekfac_eigenvalues_are_fisher_diagonal_and_solve():
    rng = np.random.default_rng(3)
    L = _layer(rng, 6, 4, 5, 6, 3, 4, lengths=True)
    psis = _psis(L)
    C = ok.fit_layers([L])[0].correct(psis)
    assert np.allclose(C.E_ekfac, ok.ekfac_fisher_diagonal(psis, C.Q_a, C.Q_g), rtol=1e-12, atol=1e-14)
    X = rng.standard_normal((3, 4))
    delta = ok.damping(C.E_ekfac)
    want = ok.ekfac_dense_precondition(X, C.Q_a, C.Q_g, C.E_ekfac, delta)
    assert np.allclose(C.precondition(X, "ekfac"), want, rtol=1e-10, atol=1e-12)


def test_mean_eigenvalues_closed_forms():
    # K-FAC: mean(lam_A lam_G^T) = tr(A) tr(S) / (k_in k_out);
    # EK-FAC: the rotation keeps Frobenius norms, so mean(E) = mean ||Psi_i||^2 / (k_in k_out)
    rng = np.random.default_rng(4)
    L = _layer(rng, 5, 7, 8, 6, 4, 3)
    psis = _psis(L)
    C = ok.fit_layers([L])[0].correct(psis)
    assert np.isclose(np.mean(C.E_kfac), np.trace(C.A) * np.trace(C.S) / 12, rtol=1e-12)
    want = np.mean([np.sum(P ** 2) for P in psis]) / 12
    assert np.isclose(np.mean(C.E_ekfac), want, rtol=1e-12)
    assert np.isclose(ok.damping(C.E_ekfac), 0.1 * want, rtol=1e-12)


def test_ekfac_equals_kfac_on_product_design():
    # One token per example, and the examples are every pairing of a set of
    # inputs with a set of output gradients: the second moment then factorizes
    # exactly, and EK-FAC's correction returns K-FAC's eigenvalues.
    rng = np.random.default_rng(5)
    d_in, d_out, k_in, k_out = 5, 4, 3, 2
    a = rng.standard_normal((4, d_in))
    g = rng.standard_normal((3, d_out))
    A = np.array([[a[j]] for j in range(4) for _ in range(3)])
    B = np.array([[g[k]] for _ in range(4) for k in range(3)])
    L = dict(A=A, B=B, P_in=rng.standard_normal((d_in, k_in)), P_out=rng.standard_normal((d_out, k_out)),
             lengths=None)
    C = ok.fit_layers([L])[0].correct(_psis(L))
    assert np.allclose(C.E_ekfac, C.E_kfac, rtol=1e-10, atol=1e-12)


def test_identity_factors_and_damping_limit():
    k_in, k_out = 3, 4
    rng = np.random.default_rng(6)
    X = rng.standard_normal((k_in, k_out))
    Q_a, Q_g = np.eye(k_in), np.eye(k_out)
    E = np.ones((k_in, k_out))
    assert np.allclose(ok.precondition(X, Q_a, Q_g, E, ok.damping(E)), X / 1.1)
    # delta -> infinity: delta * P(X) -> X (the GradDot block)
    L = _layer(rng, 4, 5, 6, 6, k_in, k_out)
    C = ok.fit_layers([L])[0]
    d = 1e9
    assert np.allclose(d * ok.precondition(X, C.Q_a, C.Q_g, C.E_kfac, d), X, rtol=1e-6, atol=1e-8)


@pytest.mark.parametrize("kind", ["kfac", "ekfac"])
def test_self_adjoint_and_positive(kind):
    rng = np.random.default_rng(7)
    L = _layer(rng, 6, 5, 7, 5, 4, 3)
    C = ok.fit_layers([L])[0].correct(_psis(L))
    X, Y = rng.standard_normal((4, 3)), rng.standard_normal((4, 3))
    PX, PY = C.precondition(X, kind), C.precondition(Y, kind)
    assert np.isclose(np.sum(PX * Y), np.sum(X * PY), rtol=1e-11)
    assert np.sum(PX * X) > 0


@pytest.mark.parametrize("kind", ["kfac", "ekfac"])
def test_scores_sum_layers_of_kronecker_solves(kind):
    rng = np.random.default_rng(8)
    layers = [_layer(rng, 5, 4, 6, 5, 2, 3, lengths=True), _layer(rng, 5, 4, 4, 7, 3, 2)]
    phi_t = np.stack([og.feature_vector([_psis(L)[i] for L in layers]) for i in range(5)])
    offsets = [0, 6]
    curv = ok.fit_layers(layers, phi_t, offsets)
    phi_q = rng.standard_normal((2, 12))
    S = ok.curvature_scores(phi_q, phi_t, curv, offsets, kind)
    for q in range(2):
        for j in range(5):
            s = 0.0
            for C, o, (ki, ko) in zip(curv, offsets, [(2, 3), (3, 2)]):
                Xq = phi_q[q, o:o + ki * ko].reshape(ki, ko)
                E = C.eigenvalues(kind)
                delta = ok.damping(E)
                if kind == "kfac":
                    Pq = ok.kfac_dense_precondition(Xq, C.A, C.S, delta)
                else:
                    Pq = ok.ekfac_dense_precondition(Xq, C.Q_a, C.Q_g, E, delta)
                s += float(np.sum(Pq * phi_t[j, o:o + ki * ko].reshape(ki, ko)))
            assert np.isclose(S[q, j], s, rtol=1e-10, atol=1e-12)


def test_errors():
    with pytest.raises(ValueError):
        ok.kfac_factors(np.eye(2), np.eye(2), 0, 1)
    with pytest.raises(ValueError):
        ok.ekfac_eigenvalues([], np.eye(2), np.eye(2))
    C = ok.LayerCurvature(np.eye(2), np.eye(2), 1, 1)
    with pytest.raises(ValueError):
        C.eigenvalues("ekfac")
    with pytest.raises(ValueError):
        C.eigenvalues("other")
