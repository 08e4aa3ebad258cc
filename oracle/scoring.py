"""Attribution scores from projected features, and per-query top-k (oracle side).

Also the cosine variant (Grad-Cos; LESS's cosine metric) of the same scores.

GradDot (Sec. 4.1; gradient similarity at one checkpoint, Sec. 2) scores a query
against a training example by the inner product of their gradients.  With the
per-layer blocks concatenated into phi, the score over all layers is
<phi_q, phi_j> = sum_l <phi_{q,l}, phi_{j,l}> (cross-layer aggregation).

The optional diagonal preconditioner d > 0 is applied once, in "multiply" form:
S[q, j] = sum_f phi_q[f] d[f] phi_j[f].  The paper defines no diagonal
preconditioner at scoring time; this is the reading used by the library
(a coordinate-wise linear map, in the spirit of Adam's coordinate-wise
preconditioning in Eq. 3 but without its nonlinearity).
"""

import numpy as np


def score(phi_q, phi_train, d=None):
    """S = (Phi_q diag(d)) Phi_train^T in float64; d = None means d = 1."""
    Q = np.asarray(phi_q, dtype=np.float64)
    X = np.asarray(phi_train, dtype=np.float64)
    if d is not None:
        Q = Q * np.asarray(d, dtype=np.float64)[None, :]
    return Q @ X.T


def score_loop(phi_q, phi_train, d=None):
    """The same scores as triple Python loops (tiny inputs only)."""
    Q = np.asarray(phi_q, dtype=np.float64)
    X = np.asarray(phi_train, dtype=np.float64)
    nq, F = Q.shape
    nt = X.shape[0]
    S = np.zeros((nq, nt), dtype=np.float64)
    for q in range(nq):
        for j in range(nt):
            s = 0.0
            for f in range(F):
                s += Q[q, f] * (1.0 if d is None else float(d[f])) * X[j, f]
            S[q, j] = s
    return S


def cosine_scores(phi_q, phi_train, d=None):
    """Grad-Cos / LESS-style scores (Sec. 2 "Grad-Cos"; App. A.3, LESS as TracIn
    with a cosine metric): the cosine between the (preconditioned) query row
    q' = q * d and the training row x, <q', x> / (|q'| |x|), taken as 0 when
    either norm is 0."""
    Q = np.asarray(phi_q, dtype=np.float64)
    X = np.asarray(phi_train, dtype=np.float64)
    if d is not None:
        Q = Q * np.asarray(d, dtype=np.float64)[None, :]
    nq = np.linalg.norm(Q, axis=1)
    nx = np.linalg.norm(X, axis=1)
    iq = np.where(nq > 0, 1.0 / np.where(nq > 0, nq, 1.0), 0.0)
    ix = np.where(nx > 0, 1.0 / np.where(nx > 0, nx, 1.0), 0.0)
    return (Q @ X.T) * iq[:, None] * ix[None, :]


def cosine_loop(phi_q, phi_train, d=None):
    """The same cosines with explicit loops over rows and features (tiny only)."""
    Q = np.asarray(phi_q, dtype=np.float64)
    X = np.asarray(phi_train, dtype=np.float64)
    S = np.zeros((Q.shape[0], X.shape[0]))
    for q in range(Q.shape[0]):
        qd = [Q[q, f] * (1.0 if d is None else float(d[f])) for f in range(Q.shape[1])]
        nq = sum(v * v for v in qd) ** 0.5
        for j in range(X.shape[0]):
            nx = sum(v * v for v in X[j]) ** 0.5
            dot = sum(a * b for a, b in zip(qd, X[j]))
            S[q, j] = dot / (nq * nx) if nq > 0 and nx > 0 else 0.0
    return S


def topk(S, k):
    """Per row: indices and values of the k largest scores, largest first; equal
    scores are ordered by lower training index.  Returns (idx int64, val)."""
    S = np.asarray(S)
    if not 0 <= k <= S.shape[1]:
        raise ValueError("k must lie in [0, n_train]")
    idx = np.empty((S.shape[0], k), dtype=np.int64)
    for q in range(S.shape[0]):
        # stable sort of -S keeps lower indices first among equal scores
        idx[q] = np.argsort(-S[q], kind="stable")[:k]
    val = np.take_along_axis(S, idx, axis=1)
    return idx, val
