"""Helpers shared by the GPU parity tests: oracle evaluation on the inputs the
library consumed, and error metrics.  Inputs come from the seeded generators
in workloads.py; expected values come only from oracle/."""
import numpy as np
import torch

from oracle import gradients as og
from oracle import rng as orng


def rel_fro(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(x - ref)
    return num / den if den > 0 else num


def host64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def oracle_maps(seed, layers, dtype):
    return [orng.projection_pair(seed, i, L["d_in"], L["d_out"], L["k_in"], L["k_out"], dtype)
            for i, L in enumerate(layers)]


def oracle_phi_rows(layers, maps, inputs, examples, lengths=None):
    """phi rows (float64) of the given examples: inputs[l] = (A, B) host float64
    arrays [n, T, d]; blocks by the factored definition (Eq. 2, left side)."""
    rows = []
    for i in examples:
        blocks = []
        for l, L in enumerate(layers):
            A, B = inputs[l]
            P_in, P_out = maps[l]
            length = None if lengths is None else int(lengths[i])
            blocks.append(og.project_factored(A[i], B[i], P_in, P_out, length))
        rows.append(og.feature_vector(blocks))
    return np.stack(rows)


def per_layer_errors(phi, ref, layers):
    """Relative Frobenius error of each layer block over the checked examples."""
    out, off = [], 0
    for L in layers:
        w = L["k_in"] * L["k_out"]
        out.append(rel_fro(phi[:, off:off + w], ref[:, off:off + w]))
        off += w
    return out
