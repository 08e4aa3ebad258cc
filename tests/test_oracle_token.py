"""Pins of the token-level attribution oracle (oracle/token.py): token sums
equal the sequence-level scores (App. D), loops, the unprojected formula
against the factorized inner product of Eq. 4, identity maps reducing the
projected form to the unprojected one, and preconditioned blocks summing to
the curvature scores."""
import numpy as np

from oracle import gradients as og
from oracle import kfac as ok
from oracle import token as otk


def _layers(rng, n, T, dims, lengths=None):
    out = []
    for d_in, d_out, k_in, k_out in dims:
        out.append(dict(A=rng.standard_normal((n, T, d_in)), B=rng.standard_normal((n, T, d_out)),
                        P_in=rng.standard_normal((d_in, k_in)) / np.sqrt(k_in),
                        P_out=rng.standard_normal((d_out, k_out)) / np.sqrt(k_out), lengths=lengths))
    return out


DIMS = [(6, 5, 3, 2), (4, 7, 2, 4)]


def test_token_sums_recover_sequence_scores_and_loops():
    rng = np.random.default_rng(0)
    lens = np.array([5, 0, 3])
    train = _layers(rng, 3, 5, DIMS, lens)
    q = [rng.standard_normal((k_in, k_out)) for _, _, k_in, k_out in DIMS]
    S = otk.token_scores(train, q)
    np.testing.assert_allclose(S, otk.token_scores_loop(train, q), rtol=1e-12, atol=1e-12)
    assert np.all(S[1] == 0) and np.all(S[2, 3:] == 0)
    phi = np.stack([og.feature_vector([og.project_factored(L["A"][i], L["B"][i], L["P_in"], L["P_out"],
                                                           int(lens[i])) for L in train]) for i in range(3)])
    qrow = og.feature_vector(q)
    np.testing.assert_allclose(S.sum(axis=1), phi @ qrow, rtol=1e-12, atol=1e-12)


def test_unprojected_formula_and_identity_maps():
    rng = np.random.default_rng(1)
    train = _layers(rng, 2, 4, [(5, 3, 5, 3), (2, 6, 2, 6)])
    query = _layers(rng, 1, 3, [(5, 3, 5, 3), (2, 6, 2, 6)])
    S = otk.unprojected_token_scores(train, query)
    # token sums = the factorized inner product of Eq. 4, summed over layers
    for i in range(2):
        want = sum(og.ghost_dot(L["A"][i], L["B"][i], Q["A"][0], Q["B"][0]) for L, Q in zip(train, query))
        assert np.isclose(S[i].sum(), want, rtol=1e-12)
    # with P = I the projected form is the unprojected one (R~ = DW^T in the (c, r) layout)
    ident = [dict(L, P_in=np.eye(L["A"].shape[2]), P_out=np.eye(L["B"].shape[2])) for L in train]
    q = [og.weight_gradient(Q["A"][0], Q["B"][0]).T for Q in query]
    np.testing.assert_allclose(otk.token_scores(ident, q), S, rtol=1e-12, atol=1e-12)


def test_preconditioned_blocks_sum_to_curvature_scores():
    rng = np.random.default_rng(2)
    train = _layers(rng, 4, 6, DIMS)
    offsets = [0, 6]
    phi = np.stack([og.feature_vector([og.project_factored(L["A"][i], L["B"][i], L["P_in"], L["P_out"])
                                       for L in train]) for i in range(4)])
    curv = ok.fit_layers(train, phi, offsets)
    qrow = rng.standard_normal((1, 14))
    for kind in ("kfac", "ekfac"):
        pq = ok.precondition_features(qrow, curv, offsets, kind)[0]
        blocks = [pq[0:6].reshape(3, 2), pq[6:14].reshape(2, 4)]
        S = otk.token_scores(train, blocks)
        np.testing.assert_allclose(S.sum(axis=1), ok.curvature_scores(qrow, phi, curv, offsets, kind)[0],
                                   rtol=1e-10, atol=1e-12)
