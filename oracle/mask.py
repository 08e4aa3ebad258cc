"""Random coordinate masks of the weight gradient, gathered from the factors
(oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

App. A.2 ("Random maps"): a random mask keeps a fixed random subset M of the
entries of DW; since entry (r, c) of DW is sum_t g_{t,r} a_{t,c} (Eq. 1), the
kept entries are gathered from the factors with |M| products per token
position, without forming DW.  AdamW-influence uses ten disjoint masks of 512
or 8192 coordinates per layer (App. B, fidelity settings).  The paper does not
say how a mask is drawn; the reading here (M1):

    base     = SM(seed)                      (SplitMix64, as for the maps)
    s(layer) = SM(base XOR (2^63 + layer))   (the maps use base XOR (2 layer + side))
    draw i   = ((x0 * 2^32 + x1) mod (d_out * d_in)) with
               (x0, x1, x2, x3) = Philox4x32-10(counter (i lo, i hi, 0, 0), key s)
    the stream of draws with repeats removed (first occurrence kept) is cut
    into runs of m; mask j is run j (so masks 0, 1, ... are disjoint), its
    entries sorted by their flat index in the column-stacked order of Eq. 1,
    u = c * d_out + r (entry (r, c) = DW[r, c], r < d_out, c < d_in).

The masked block of an example is the vector DW[r_e, c_e] over the mask's
entries in that order.  Arithmetic is float64.

Parity: the index layout is this library's reading ("parity unpinned" with
respect to the paper); the gathered values are pinned to Eq. 1's dense DW.
"""

import numpy as np

from . import gradients as og
from . import rng as orng

MASK_KEY_BIT = 1 << 63


def mask_seed(global_seed, layer):
    return orng.sm(orng.sm(global_seed) ^ (MASK_KEY_BIT + layer))


def mask_indices(global_seed, layer, d_in, d_out, m, mask_id=0):
    """(rows, cols) int64 arrays of mask `mask_id` (m entries) of a layer,
    sorted by u = c * d_out + r."""
    N = d_in * d_out
    need = (mask_id + 1) * m
    if m < 1 or mask_id < 0 or 2 * need > N:
        raise ValueError("masks need m >= 1 and (mask_id + 1) * m <= d_in * d_out / 2")
    s = mask_seed(global_seed, layer)
    seen, order = set(), []
    i = 0
    while len(order) < need:
        batch = np.arange(i, i + 4 * need, dtype=np.uint64)
        x0, x1, _, _ = orng.philox4x32_10(batch & np.uint64(orng.MASK32), batch >> np.uint64(32),
                                          np.zeros_like(batch), np.zeros_like(batch),
                                          s & orng.MASK32, s >> 32)
        u = ((x0.astype(np.uint64) << np.uint64(32)) | x1.astype(np.uint64)) % np.uint64(N)
        for v in u.tolist():
            if v not in seen:
                seen.add(v)
                order.append(v)
                if len(order) == need:
                    break
        i += 4 * need
    run = np.sort(np.array(order[mask_id * m:(mask_id + 1) * m], dtype=np.int64))
    return run % d_out, run // d_out


def masked_gradient(A, B, rows, cols, length=None):
    """DW[rows[e], cols[e]] = sum_t B[t, rows[e]] A[t, cols[e]], gathered from
    the factors (one product per entry and token)."""
    A, B = og._take_tokens(A, B, length)
    return np.einsum("te,te->e", B[:, np.asarray(rows)], A[:, np.asarray(cols)])


def masked_gradient_loop(A, B, rows, cols, length=None):
    """The same sums with explicit loops (tiny only)."""
    A, B = og._take_tokens(A, B, length)
    out = np.zeros(len(rows))
    for e, (r, c) in enumerate(zip(rows, cols)):
        s = 0.0
        for t in range(A.shape[0]):
            s += B[t, r] * A[t, c]
        out[e] = s
    return out
