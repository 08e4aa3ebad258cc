"""Per-example gradients of a linear layer and their projections (oracle side).

Notation (Sec. 3.2, "Two representations of gradients"): a linear layer
z = W a with W in R^{N_o x N_i}; for one example, the inputs at its T token
positions are a_t in R^{N_i} and the loss gradients w.r.t. the outputs are
g_t in R^{N_o}.  The arrays used here hold those vectors as rows:

    A[t, :] = a_t      A has shape [T, d_in]   (d_in  = N_i)
    B[t, :] = g_t      B has shape [T, d_out]  (d_out = N_o)

so that A and B are the "factors" of the factorized representation.

The projection maps are stored as P_in = P_a^T in R^{d_in x k_in} and
P_out = P_g^T in R^{d_out x k_out} (Eq. 2 applies P_a, P_g to columns).

Flatten order.  Eq. 1 writes vec(DW) = sum_t a_t (x) g_t with vec stacking
columns, so element (r, c) of DW (row r of the output side, column c of the
input side) sits at flat index c*N_o + r.  Eq. 2 keeps that structure in the
projected space: element (c, r) of the k_in x k_out block Psi sits at
c*k_out + r, i.e. Psi stored row-major.

All arithmetic is float64.  ``length`` (optional) keeps only the first
``length`` token positions of an example (variable T_i, Eq. 4).
"""

import numpy as np


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def _take_tokens(A, B, length):
    A, B = _f64(A), _f64(B)
    if A.ndim != 2 or B.ndim != 2 or A.shape[0] != B.shape[0]:
        raise ValueError("A [T, d_in] and B [T, d_out] must share T")
    T = A.shape[0]
    if length is not None:
        if not 0 <= length <= T:
            raise ValueError("length must lie in [0, T]")
        T = int(length)
    return A[:T], B[:T]


def weight_gradient_loop(A, B, length=None):
    """DW = sum_t g_t a_t^T as an explicit loop over token positions (Eq. 1).

    Returns the d_out x d_in matrix G.  For tiny inputs only (the definition
    written out term by term).
    """
    A, B = _take_tokens(A, B, length)
    G = np.zeros((B.shape[1], A.shape[1]), dtype=np.float64)
    for t in range(A.shape[0]):
        G += np.outer(B[t], A[t])
    return G


def weight_gradient(A, B, length=None):
    """DW = B^T A, the same sum over tokens as ``weight_gradient_loop`` (Eq. 1)."""
    A, B = _take_tokens(A, B, length)
    return B.T @ A


def vec_columns(G):
    """vec(DW): stack the columns of the d_out x d_in gradient (Eq. 1)."""
    return _f64(G).T.reshape(-1)


def kron_sum(A, B, length=None):
    """sum_t a_t (x) g_t written with Kronecker products (right side of Eq. 1)."""
    A, B = _take_tokens(A, B, length)
    out = np.zeros(A.shape[1] * B.shape[1], dtype=np.float64)
    for t in range(A.shape[0]):
        out += np.kron(A[t], B[t])
    return out


def project_factored(A, B, P_in, P_out, length=None):
    """Factor projection, left side of Eq. 2: Psi = (A P_in)^T (B P_out).

    Rows of A P_in are the projected inputs a~_t = P_a a_t, rows of B P_out the
    projected output gradients g~_t = P_g g_t; Psi[c, r] = sum_t a~_t[c] g~_t[r].
    Returns Psi with shape [k_in, k_out].
    """
    A, B = _take_tokens(A, B, length)
    return (A @ _f64(P_in)).T @ (B @ _f64(P_out))


def project_materialized(G, P_in, P_out):
    """Kronecker projection of the materialized gradient, right side of Eq. 2.

    (P_a (x) P_g) vec(DW) = vec(P_g DW P_a^T); as a k_in x k_out block in the
    flatten order above this is Psi = (P_out^T G P_in)^T.
    """
    return (_f64(P_out).T @ _f64(G) @ _f64(P_in)).T


def project_brute_force(A, B, P_in, P_out, length=None):
    """Psi[c, r] = sum_t sum_u sum_v A[t, v] P_in[v, c] B[t, u] P_out[u, r],
    with pure Python loops.  Tiny inputs only."""
    A, B = _take_tokens(A, B, length)
    P_in, P_out = _f64(P_in), _f64(P_out)
    T, d_in = A.shape
    d_out = B.shape[1]
    k_in, k_out = P_in.shape[1], P_out.shape[1]
    Psi = np.zeros((k_in, k_out), dtype=np.float64)
    for c in range(k_in):
        for r in range(k_out):
            s = 0.0
            for t in range(T):
                for v in range(d_in):
                    for u in range(d_out):
                        s += A[t, v] * P_in[v, c] * B[t, u] * P_out[u, r]
            Psi[c, r] = s
    return Psi


def feature_vector(blocks):
    """phi = concatenation of the row-major flattened per-layer blocks, in layer
    order (cross-layer aggregation sums per-layer inner products, so phi's inner
    product is the sum over layers)."""
    return np.concatenate([_f64(b).reshape(-1) for b in blocks])


def project_example(layers, route="factored"):
    """phi_i for one example.

    ``layers`` is a sequence of dicts with keys A, B, P_in, P_out and optional
    length.  ``route`` selects which exact form computes each block
    ("factored" or "materialized"); in exact arithmetic both give the same phi.
    """
    blocks = []
    for L in layers:
        length = L.get("length")
        if route == "factored":
            blocks.append(project_factored(L["A"], L["B"], L["P_in"], L["P_out"], length))
        elif route == "materialized":
            G = weight_gradient(L["A"], L["B"], length)
            blocks.append(project_materialized(G, L["P_in"], L["P_out"]))
        else:
            raise ValueError("route must be 'factored' or 'materialized'")
    return feature_vector(blocks)


def ghost_dot(A_i, B_i, A_j, B_j, len_i=None, len_j=None):
    """Factorized inner product, Eq. 4:

        <vec DW_i, vec DW_j> = sum_{t<T_i} sum_{s<T_j} <a_t, a_s> <g_t, g_s>
                             = sum((A_i A_j^T) * (B_i B_j^T)).
    """
    A_i, B_i = _take_tokens(A_i, B_i, len_i)
    A_j, B_j = _take_tokens(A_j, B_j, len_j)
    return float(np.sum((A_i @ A_j.T) * (B_i @ B_j.T)))


def ghost_dot_loop(A_i, B_i, A_j, B_j):
    """Eq. 4 as its double sum over token pairs, pure Python loops (tiny only)."""
    A_i, B_i, A_j, B_j = _f64(A_i), _f64(B_i), _f64(A_j), _f64(B_j)
    s = 0.0
    for t in range(A_i.shape[0]):
        for u in range(A_j.shape[0]):
            s += float(A_i[t] @ A_j[u]) * float(B_i[t] @ B_j[u])
    return s
