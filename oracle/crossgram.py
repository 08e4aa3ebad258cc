"""Cross-Gram matrices of unprojected per-example weight gradients (oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 3.2 "Factorized inner product" (Eq. 4) and "FLOP-aware routing", and
App. A.4 (routing-complexity table, "Routing"): for two batches of examples,
the cross-Gram matrix holds the inner products of their per-example weight
gradients, summed over the attributed layers,

    K[i, j] = sum_l < DW_l^(i), DW_l^(j) >_F ,   i in batch 1, j in batch 2.

Two exact routes compute each layer's contribution:

  factorized    Eq. 4: sum_{t < T_i} sum_{s < T_j} <a_t^(i), a_s^(j)> <g_t^(i), g_s^(j)>,
                i.e. the sum of the entries of (A_i A_j^T) * (B_i B_j^T);
  materialized  build DW = B^T A for every example (Eq. 1) and take the
                Frobenius inner product of the dense matrices.

Per-example squared norms are the diagonal of a batch's Gram with itself,
||DW^(i)||_F^2, and are routed the same way (App. A.4 "Routing").

A batch is given as a list over layers of (A, B, lengths): A [n, T, d_in],
B [n, T, d_out] (rows = token positions, as in ``gradients``), lengths None or
an int sequence [n] keeping the first lengths[i] tokens of example i.  All
arithmetic is float64.
"""

import numpy as np

from . import gradients as og


def _length(lengths, i):
    return None if lengths is None else int(lengths[i])


def _check(batch1, batch2):
    if len(batch1) != len(batch2):
        raise ValueError("both batches must list the same layers")
    for (A1, B1, _), (A2, B2, _) in zip(batch1, batch2):
        if np.shape(A1)[2] != np.shape(A2)[2] or np.shape(B1)[2] != np.shape(B2)[2]:
            raise ValueError("a layer's d_in / d_out must agree across batches")


def layer_cross_gram(A1, B1, len1, A2, B2, len2, route):
    """One layer's contribution to K, by the chosen exact route."""
    n1, n2 = np.shape(A1)[0], np.shape(A2)[0]
    K = np.zeros((n1, n2), dtype=np.float64)
    if route == "factorized":
        for i in range(n1):
            for j in range(n2):
                K[i, j] = og.ghost_dot(A1[i], B1[i], A2[j], B2[j], _length(len1, i), _length(len2, j))
    elif route == "materialized":
        G1 = [og.weight_gradient(A1[i], B1[i], _length(len1, i)) for i in range(n1)]
        G2 = [og.weight_gradient(A2[j], B2[j], _length(len2, j)) for j in range(n2)]
        for i in range(n1):
            for j in range(n2):
                K[i, j] = float(np.sum(G1[i] * G2[j]))
    else:
        raise ValueError("route must be 'factorized' or 'materialized'")
    return K


def cross_gram(batch1, batch2, route="factorized"):
    """K [n1, n2]: sum over layers of <DW^(i), DW^(j)>_F (Eq. 4 summed over
    layers); both routes give the same K in exact arithmetic."""
    _check(batch1, batch2)
    K = None
    for (A1, B1, len1), (A2, B2, len2) in zip(batch1, batch2):
        part = layer_cross_gram(A1, B1, len1, A2, B2, len2, route)
        K = part if K is None else K + part
    return K


def sq_norms(batch, route="factorized"):
    """||DW^(i)||_F^2 summed over layers, for every example of one batch."""
    n = np.shape(batch[0][0])[0]
    out = np.zeros(n, dtype=np.float64)
    for A, B, lengths in batch:
        for i in range(n):
            L = _length(lengths, i)
            if route == "factorized":
                out[i] += og.ghost_dot(A[i], B[i], A[i], B[i], L, L)
            elif route == "materialized":
                G = og.weight_gradient(A[i], B[i], L)
                out[i] += float(np.sum(G * G))
            else:
                raise ValueError("route must be 'factorized' or 'materialized'")
    return out


def cross_gram_brute_force(batch1, batch2):
    """Eq. 1 and the Frobenius inner product written out with pure Python
    loops over tokens and matrix entries.  Tiny inputs only."""
    _check(batch1, batch2)
    n1, n2 = np.shape(batch1[0][0])[0], np.shape(batch2[0][0])[0]
    K = np.zeros((n1, n2), dtype=np.float64)
    for (A1, B1, len1), (A2, B2, len2) in zip(batch1, batch2):
        for i in range(n1):
            G1 = og.weight_gradient_loop(A1[i], B1[i], _length(len1, i))
            for j in range(n2):
                G2 = og.weight_gradient_loop(A2[j], B2[j], _length(len2, j))
                s = 0.0
                for r in range(G1.shape[0]):
                    for c in range(G1.shape[1]):
                        s += G1[r, c] * G2[r, c]
                K[i, j] += s
    return K
