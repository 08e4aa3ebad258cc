"""Kronecker-factored curvature on projected factors: K-FAC and EK-FAC (oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 3.2 states that factorized gradients support the preconditioned comparisons
of K-FAC (Martens & Grosse, 2015) and EK-FAC (George et al., 2018), and App. A.2
("Factor projection") that these statistics apply unchanged to the projected
pair (a~_t, g~_t).  The paper prints no formula for either method, so this
module follows the cited methods' definitions, with the readings below.

Per layer, with projected token rows a~_t (k_in) and g~_t (k_out) of example i
and its block Psi_i = sum_t a~_t g~_t^T (k_in x k_out, the layout of Eq. 2):

  input factor      A = (1 / N_tok) sum_i sum_t a~_t a~_t^T        (k_in x k_in)
  gradient factor   S = (1 / N)     sum_i sum_t g~_t g~_t^T        (k_out x k_out)

N_tok is the number of token positions summed, N the number of examples.  This
scaling makes A (x) S the token-independence approximation of the
per-example second moment E_i[vec(Psi_i) vec(Psi_i)^T], the quantity EK-FAC
re-estimates, so both methods live on one scale (reading K1).

Eigendecompositions A = Q_A diag(lam_A) Q_A^T, S = Q_G diag(lam_G) Q_G^T
(ascending eigenvalues).  Eigenvalues of the curvature, laid out like Psi:

  K-FAC    E[c, r] = lam_A[c] lam_G[r]
  EK-FAC   E[c, r] = (1 / N) sum_i ((Q_A^T Psi_i Q_G)[c, r])^2
           (the second moment of the gradients in the Kronecker eigenbasis,
            George et al.'s eigenvalue correction)

Damping (App. B, fidelity settings: 0.1 times the mean eigenvalue of each
layer), written delta = rel * mean(E) + abs; the token-level examples of
App. D use a fixed damping, which ``abs`` expresses (reading K2).

Preconditioned query block (inverse of the damped curvature applied to Psi_q):

  P(Psi_q) = Q_A [ (Q_A^T Psi_q Q_G) / (E + delta) ] Q_G^T

and the curvature-aware score of query q against training example j is the sum
over layers of <P(Psi_q), Psi_j>_F (cross-layer aggregation as in GradDot).

Arithmetic is float64; eigendecompositions use numpy.linalg.eigh (LAPACK).
Parity: pinned.  The Kronecker-solve form, the Fisher-diagonal form of the
EK-FAC eigenvalues and the token loops in ``kfac_dense_precondition``,
``ekfac_fisher_diagonal`` and ``factor_sums_loop`` restate the definitions
independently of the eigenbasis formulas (tests/test_oracle_kfac.py).
"""

import numpy as np


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def _rows(A, length):
    A = _f64(A)
    if length is None:
        return A
    if not 0 <= length <= A.shape[0]:
        raise ValueError("length must lie in [0, T]")
    return A[: int(length)]


# ------------------------------------------------------------ factor statistics
def factor_sums(A, B, P_in, P_out, lengths=None):
    """Sums over examples and their token positions of a~ a~^T and g~ g~^T.

    A [n, T, d_in], B [n, T, d_out] hold the factor rows of n examples;
    lengths (None or [n]) keeps each example's first lengths[i] positions.
    Returns (SA [k_in, k_in], SG [k_out, k_out], n_tokens, n_examples).
    """
    P_in, P_out = _f64(P_in), _f64(P_out)
    n = np.shape(A)[0]
    SA = np.zeros((P_in.shape[1], P_in.shape[1]))
    SG = np.zeros((P_out.shape[1], P_out.shape[1]))
    tokens = 0
    for i in range(n):
        L = None if lengths is None else int(lengths[i])
        At = _rows(A[i], L) @ P_in      # rows a~_t
        Bt = _rows(B[i], L) @ P_out     # rows g~_t
        SA += At.T @ At
        SG += Bt.T @ Bt
        tokens += At.shape[0]
    return SA, SG, tokens, n


def factor_sums_loop(A, B, P_in, P_out, lengths=None):
    """``factor_sums`` with one outer product per token position (tiny only)."""
    P_in, P_out = _f64(P_in), _f64(P_out)
    SA = np.zeros((P_in.shape[1], P_in.shape[1]))
    SG = np.zeros((P_out.shape[1], P_out.shape[1]))
    tokens = 0
    for i in range(np.shape(A)[0]):
        L = None if lengths is None else int(lengths[i])
        Ai, Bi = _rows(A[i], L), _rows(B[i], L)
        for t in range(Ai.shape[0]):
            a = P_in.T @ Ai[t]
            g = P_out.T @ Bi[t]
            SA += np.outer(a, a)
            SG += np.outer(g, g)
            tokens += 1
    return SA, SG, tokens, np.shape(A)[0]


def kfac_factors(SA, SG, n_tokens, n_examples):
    """The normalized factors A = SA / N_tok and S = SG / N (reading K1)."""
    if n_tokens <= 0 or n_examples <= 0:
        raise ValueError("factors need at least one token and one example")
    return _f64(SA) / n_tokens, _f64(SG) / n_examples


def eigenbasis(M):
    """Symmetric eigendecomposition M = Q diag(lam) Q^T, eigenvalues ascending."""
    lam, Q = np.linalg.eigh(_f64(M))
    return lam, Q


# ------------------------------------------------------------------ eigenvalues
def kfac_eigenvalues(lam_a, lam_g):
    """K-FAC's curvature eigenvalues lam_A[c] lam_G[r], laid out like Psi."""
    return np.outer(_f64(lam_a), _f64(lam_g))


def rotate(Psi, Q_a, Q_g):
    """Psi in the Kronecker eigenbasis: Q_A^T Psi Q_G."""
    return _f64(Q_a).T @ _f64(Psi) @ _f64(Q_g)


def ekfac_sums(psis, Q_a, Q_g):
    """Sum over examples of the squared rotated blocks (Q_A^T Psi_i Q_G)^2."""
    out = None
    for P in psis:
        R = rotate(P, Q_a, Q_g) ** 2
        out = R if out is None else out + R
    return out


def ekfac_eigenvalues(psis, Q_a, Q_g):
    """EK-FAC's corrected eigenvalues: the mean over examples of the squared
    rotated blocks (George et al.'s eigenvalue correction)."""
    psis = list(psis)
    if not psis:
        raise ValueError("the correction needs at least one example")
    return ekfac_sums(psis, Q_a, Q_g) / len(psis)


def ekfac_fisher_diagonal(psis, Q_a, Q_g):
    """The same eigenvalues from their definition as the diagonal of the
    second-moment matrix F = mean_i vec(Psi_i) vec(Psi_i)^T in the Kronecker
    eigenbasis U = Q_A (x) Q_G, with vec the row-major flattening of Psi
    (tiny only: F has (k_in k_out)^2 entries)."""
    V = np.stack([_f64(P).reshape(-1) for P in psis])
    F = V.T @ V / V.shape[0]
    U = np.kron(_f64(Q_a), _f64(Q_g))
    k_in, k_out = np.shape(Q_a)[0], np.shape(Q_g)[0]
    return np.diag(U.T @ F @ U).reshape(k_in, k_out)


def damping(E, rel=0.1, abs_=0.0):
    """delta = rel * mean eigenvalue of the layer + abs (App. B; reading K2)."""
    return rel * float(np.mean(_f64(E))) + abs_


# --------------------------------------------------------------- preconditioning
def precondition(Psi_q, Q_a, Q_g, E, delta):
    """Q_A [ (Q_A^T Psi_q Q_G) / (E + delta) ] Q_G^T."""
    R = rotate(Psi_q, Q_a, Q_g) / (_f64(E) + delta)
    return _f64(Q_a) @ R @ _f64(Q_g).T


def kfac_dense_precondition(Psi_q, A, S, delta):
    """K-FAC's preconditioned block from its definition: solve
    (A (x) S + delta I) vec(X) = vec(Psi_q) with the explicit Kronecker matrix
    and row-major vec (tiny only)."""
    A, S = _f64(A), _f64(S)
    H = np.kron(A, S) + delta * np.eye(A.shape[0] * S.shape[0])
    x = np.linalg.solve(H, _f64(Psi_q).reshape(-1))
    return x.reshape(A.shape[0], S.shape[0])


def ekfac_dense_precondition(Psi_q, Q_a, Q_g, E, delta):
    """EK-FAC's preconditioned block from its definition: solve
    (U diag(vec E) U^T + delta I) vec(X) = vec(Psi_q), U = Q_A (x) Q_G (tiny only)."""
    U = np.kron(_f64(Q_a), _f64(Q_g))
    H = U @ np.diag(_f64(E).reshape(-1)) @ U.T + delta * np.eye(U.shape[0])
    x = np.linalg.solve(H, _f64(Psi_q).reshape(-1))
    return x.reshape(np.shape(Q_a)[0], np.shape(Q_g)[0])


# ----------------------------------------------------------------- whole layers
class LayerCurvature:
    """One layer's fitted curvature: factors, eigenbases, both eigenvalue sets."""

    def __init__(self, SA, SG, n_tokens, n_examples):
        self.A, self.S = kfac_factors(SA, SG, n_tokens, n_examples)
        self.lam_a, self.Q_a = eigenbasis(self.A)
        self.lam_g, self.Q_g = eigenbasis(self.S)
        self.E_kfac = kfac_eigenvalues(self.lam_a, self.lam_g)
        self.E_ekfac = None

    def correct(self, psis):
        """Fit EK-FAC's eigenvalues from the training blocks Psi_i."""
        self.E_ekfac = ekfac_eigenvalues(psis, self.Q_a, self.Q_g)
        return self

    def eigenvalues(self, kind):
        if kind == "kfac":
            return self.E_kfac
        if kind == "ekfac":
            if self.E_ekfac is None:
                raise ValueError("EK-FAC eigenvalues not fitted")
            return self.E_ekfac
        raise ValueError("kind must be 'kfac' or 'ekfac'")

    def precondition(self, Psi_q, kind, rel=0.1, abs_=0.0):
        E = self.eigenvalues(kind)
        return precondition(Psi_q, self.Q_a, self.Q_g, E, damping(E, rel, abs_))


def fit_layers(layers, phi_train=None, offsets=None):
    """Fit every layer from its captured factors.

    layers: list of dicts with A [n, T, d_in], B [n, T, d_out], P_in, P_out and
    optional lengths.  With phi_train [n, F] and the layer offsets (column of
    each layer's block), also fits EK-FAC's eigenvalues from the blocks.
    """
    out = []
    for li, L in enumerate(layers):
        SA, SG, nt, ne = factor_sums(L["A"], L["B"], L["P_in"], L["P_out"], L.get("lengths"))
        C = LayerCurvature(SA, SG, nt, ne)
        if phi_train is not None:
            k_in, k_out = np.shape(L["P_in"])[1], np.shape(L["P_out"])[1]
            o = offsets[li]
            psis = [_f64(row[o:o + k_in * k_out]).reshape(k_in, k_out) for row in phi_train]
            C.correct(psis)
        out.append(C)
    return out


def precondition_features(phi_q, curv, offsets, kind, rel=0.1, abs_=0.0):
    """Preconditioned query features: every layer block of every row replaced
    by its preconditioned block (columns outside the layers are zero)."""
    phi_q = _f64(phi_q)
    out = np.zeros_like(phi_q)
    for C, o in zip(curv, offsets):
        k_in, k_out = C.Q_a.shape[0], C.Q_g.shape[0]
        for q in range(phi_q.shape[0]):
            Psi = phi_q[q, o:o + k_in * k_out].reshape(k_in, k_out)
            out[q, o:o + k_in * k_out] = C.precondition(Psi, kind, rel, abs_).reshape(-1)
    return out


def curvature_scores(phi_q, phi_train, curv, offsets, kind, rel=0.1, abs_=0.0):
    """S[q, j] = sum over layers of <P(Psi_q), Psi_j>_F."""
    Pq = precondition_features(phi_q, curv, offsets, kind, rel, abs_)
    return Pq @ _f64(phi_train).T
