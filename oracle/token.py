"""Token-level attribution (oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

App. D ("Token-Level Attribution Examples"): for one layer and a query-side
matrix R^(j) (N_o x N_i), the contribution of token position t of training
example i is

    s_t^(i,j) = (g_t^(i))^T R^(j) a_t^(i),   sum_t s_t^(i,j) = <DW^(i), R^(j)>_F,

summed over the attributed layers; R^(j) = DW^(j) for GradDot and the
preconditioned query gradient for K-FAC / EK-FAC.

On projected factors (App. A.2: every factorized operation applies to the
projected pair unchanged) the layer's query-side matrix is its k_in x k_out
block R~ of the query's feature row (phi, or its preconditioned row), element
(c, r) the coefficient of a~_t[c] g~_t[r] (the layout of Eq. 2), so

    s_t = a~_t^T R~ g~_t,   a~_t = P_in^T a_t,  g~_t = P_out^T g_t,

and the token sum equals the inner product of the query row with the training
example's phi (reading T1).  Unprojected (P = I) this is the paper's formula
with R = DW^(j) transposed into the (c, r) layout.  Arithmetic is float64.
"""

import numpy as np

from . import gradients as og


def token_scores(layers, q_blocks):
    """[n, T] token scores of every training example for one query.

    layers: list of dicts with A [n, T, d_in], B [n, T, d_out], P_in, P_out and
    optional lengths; q_blocks: per layer the query's k_in x k_out block.
    Positions past an example's length score 0."""
    n, T = np.shape(layers[0]["A"])[:2]
    S = np.zeros((n, T))
    for L, R in zip(layers, q_blocks):
        R = np.asarray(R, dtype=np.float64)
        lens = L.get("lengths")
        for i in range(n):
            Ti = T if lens is None else int(lens[i])
            At = np.asarray(L["A"][i][:Ti], dtype=np.float64) @ np.asarray(L["P_in"], dtype=np.float64)
            Bt = np.asarray(L["B"][i][:Ti], dtype=np.float64) @ np.asarray(L["P_out"], dtype=np.float64)
            S[i, :Ti] += np.einsum("tc,cr,tr->t", At, R, Bt)
    return S


def token_scores_loop(layers, q_blocks):
    """The same scores with explicit loops over tokens and block entries (tiny only)."""
    n, T = np.shape(layers[0]["A"])[:2]
    S = np.zeros((n, T))
    for L, R in zip(layers, q_blocks):
        P_in, P_out = np.asarray(L["P_in"], dtype=np.float64), np.asarray(L["P_out"], dtype=np.float64)
        lens = L.get("lengths")
        for i in range(n):
            Ti = T if lens is None else int(lens[i])
            for t in range(Ti):
                a = P_in.T @ np.asarray(L["A"][i][t], dtype=np.float64)
                g = P_out.T @ np.asarray(L["B"][i][t], dtype=np.float64)
                s = 0.0
                for c in range(R.shape[0]):
                    for r in range(R.shape[1]):
                        s += a[c] * R[c][r] * g[r]
                S[i, t] += s
    return S


def unprojected_token_scores(train_layers, query_layers, qi=0):
    """The paper's formula with R = DW^(q) of query example qi (GradDot):
    s_t = g_t^T DW^(q) a_t = sum_s (a_t . a_s^q)(g_t . g_s^q)."""
    n, T = np.shape(train_layers[0]["A"])[:2]
    S = np.zeros((n, T))
    for L, Q in zip(train_layers, query_layers):
        qlen = None if Q.get("lengths") is None else int(Q["lengths"][qi])
        R = og.weight_gradient(Q["A"][qi], Q["B"][qi], qlen)  # d_out x d_in
        lens = L.get("lengths")
        for i in range(n):
            Ti = T if lens is None else int(lens[i])
            A = np.asarray(L["A"][i][:Ti], dtype=np.float64)
            B = np.asarray(L["B"][i][:Ti], dtype=np.float64)
            S[i, :Ti] += np.einsum("tr,rc,tc->t", B, R, A)
    return S
