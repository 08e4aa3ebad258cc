"""Closed-form operation and storage counts of the two exact routes (oracle side).

Sec. 3.2 ("Two representations of gradients", "FLOP-aware routing") and App. A.4
(routing-complexity table, "Regimes") give the counts for storage and for
cross-Gram matrices.  For the operation the library routes -- producing the
projected per-example gradient of one linear layer -- the two forms of Eq. 2
cost, per example with T token positions (multiply-add = 2 FLOP):

  factored:      A P_in  (2 T d_in k_in)  +  B P_out (2 T d_out k_out)
                 + token contraction (A P_in)^T (B P_out)  (2 T k_in k_out)
  materialized:  G = B^T A (2 T d_in d_out), then P_out^T G P_in by the cheaper
                 association:
                   (G P_in) first:   2 d_out d_in k_in + 2 d_out k_in k_out
                   (P_out^T G) first: 2 d_out d_in k_out + 2 k_out d_in k_in
"""


def factored_flops(d_in, d_out, k_in, k_out, T):
    return 2 * T * (d_in * k_in + d_out * k_out + k_in * k_out)


def materialized_flops(d_in, d_out, k_in, k_out, T):
    build = 2 * T * d_in * d_out
    right_first = 2 * d_out * d_in * k_in + 2 * d_out * k_in * k_out
    left_first = 2 * d_out * d_in * k_out + 2 * k_out * d_in * k_in
    return build + min(right_first, left_first)


def factor_bytes(d_in, d_out, T, elt_bytes):
    """Bytes of one example's two factor blocks A [T, d_in] and B [T, d_out]."""
    return T * (d_in + d_out) * elt_bytes


def storage_factorized(N_i, N_o, T):
    """Values stored by the factorized form: T (N_i + N_o)."""
    return T * (N_i + N_o)


def storage_materialized(N_i, N_o):
    """Values stored by the materialized form: N_i N_o."""
    return N_i * N_o


def storage_threshold(N_i, N_o):
    """The factorized form is smaller exactly when T < N_i N_o / (N_i + N_o)."""
    return N_i * N_o / (N_i + N_o)


def crossgram_factorized(B1, B2, T, N_i, N_o):
    """Leading-order cross-Gram cost of the factorized route (App. A.4 table)."""
    return B1 * B2 * T * T * (N_i + N_o)


def crossgram_materialized(B1, B2, T, N_i, N_o):
    """Leading-order cross-Gram cost of the materialized route (App. A.4 table)."""
    return (B1 + B2) * T * N_i * N_o + B1 * B2 * N_i * N_o


def crossgram_flops_factorized(n1, n2, T1, T2, d_in, d_out):
    """Exact FLOPs of one layer's cross-Gram by Eq. 4 (multiply-add = 2):
    per pair the input Gram A_i A_j^T (2 T1 T2 d_in), the output-gradient Gram
    B_i B_j^T (2 T1 T2 d_out) and the sum of their elementwise product
    (2 T1 T2).  Leading term: the factorized row of the App. A.4 table."""
    return 2 * n1 * n2 * T1 * T2 * (d_in + d_out + 1)


def crossgram_flops_materialized(n1, n2, T1, T2, d_in, d_out):
    """Exact FLOPs of one layer's cross-Gram through dense gradients: DW = B^T A
    for every example (2 T d_in d_out each) and one Frobenius inner product
    per pair (2 d_in d_out).  Leading terms: the materialized row of App. A.4."""
    return 2 * (n1 * T1 + n2 * T2) * d_in * d_out + 2 * n1 * n2 * d_in * d_out
