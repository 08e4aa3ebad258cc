"""Synthetic workloads: layer shapes and seeded input generators.

This module holds NO arithmetic of the attribution method.  It only describes
workload shapes and draws seeded synthetic factor blocks / features with torch's
counter-free generators, so that the HIP library and the oracle can be fed the
very same values.  Both the tests and ``bench.py`` import it; nothing in the
library does.

Workloads (synthetic stand-ins; no dataset or checkpoint is used):

* ``tiny``      one 64->64 linear layer, T=16, 8 train + 4 query examples, fp32
                N(0,1) factors, k_in=k_out=8, seed 0.
* ``gpt2``      12 GPT-2-small blocks, each with linear layers 768->2304,
                768->768, 768->3072, 3072->768 (48 layers); T=512, batch 32,
                bf16, A ~ N(0,1), B ~ 1e-3 N(0,1); k_in=k_out=16 (F = 12,288);
                4096 train vs 256 query examples for scoring.
* ``llama8b``   32 Llama-3-8B blocks, each with q 4096->4096, k 4096->1024,
                v 4096->1024, o 4096->4096, gate 4096->14336, up 4096->14336,
                down 14336->4096 (224 layers); T=2048, batch 8, bf16, A and B
                drawn from a Student-t with 4 degrees of freedom; k_in=k_out=32
                (F = 229,376).  q/k/v read the same input block and so do
                gate/up, as in the real network.
* ``routing``   one 8192->28672 layer, T=32, batch 64, bf16 N(0,1), k=64.
* ``lora_b``    one 8->4096 layer (a rank-8 adapter's B matrix), T=32,
                batch 64, bf16 N(0,1), k_in=8, k_out=64.
* ``narrow``    one 128->128 layer, T=2048, batch 8, bf16 N(0,1), k=64.
* ``score``     Phi_train 200000 x 8192 and Phi_query 2048 x 8192, bf16 N(0,1);
                positive diagonal preconditioner log-uniform on [1e-3, 1e3];
                fp32 scores plus per-query top-100.
* ``curvature`` K-FAC / EK-FAC attribution: 28 Qwen2.5-7B-shaped blocks, each
                with q 3584->3584, k 3584->512, v 3584->512, o 3584->3584,
                gate 3584->18944, up 3584->18944, down 18944->3584 (196
                layers); T=512, 512 training sequences in batches of 32 and 1
                query, bf16 Student-t(4) factors, k_in=k_out=64 (F = 802,816).
                Stands in for the paper's throughput runs (Table
                "throughput-full": Qwen models, WikiText-103, T=512, 512
                training sequences, factor projection k_a=k_g=64).
* ``crossgram`` unprojected cross-Gram routing sweep: 24 Pythia-410M-shaped
                blocks, each with linear layers 1024->3072 (query/key/value),
                1024->1024 (attention output), 1024->4096 and 4096->1024 (MLP)
                (96 layers); 8 training examples against 1 query, T in
                {32, 128, 512, 2048}, bf16 N(0,1) factors.  Stands in for the
                routing ablation over sequence length on Pythia-410M /
                WikiText-103 (App. B, "Routing Across Sequence Lengths").
"""

import hashlib

import torch


def _layer(name, d_in, d_out, k_in, k_out, a_group):
    return {"name": name, "d_in": d_in, "d_out": d_out, "k_in": k_in,
            "k_out": k_out, "a_group": a_group}


def _gpt2_layers(k=16):
    out = []
    for b in range(12):
        out += [_layer(f"h{b}.attn.c_attn", 768, 2304, k, k, f"h{b}.ln1"),
                _layer(f"h{b}.attn.c_proj", 768, 768, k, k, f"h{b}.attn_out"),
                _layer(f"h{b}.mlp.c_fc", 768, 3072, k, k, f"h{b}.ln2"),
                _layer(f"h{b}.mlp.c_proj", 3072, 768, k, k, f"h{b}.gelu")]
    return out


def _llama_layers(k=32, blocks=32):
    out = []
    for b in range(blocks):
        attn_in, mlp_in = f"L{b}.attn_in", f"L{b}.mlp_in"
        out += [_layer(f"L{b}.q_proj", 4096, 4096, k, k, attn_in),
                _layer(f"L{b}.k_proj", 4096, 1024, k, k, attn_in),
                _layer(f"L{b}.v_proj", 4096, 1024, k, k, attn_in),
                _layer(f"L{b}.o_proj", 4096, 4096, k, k, f"L{b}.attn_core"),
                _layer(f"L{b}.gate_proj", 4096, 14336, k, k, mlp_in),
                _layer(f"L{b}.up_proj", 4096, 14336, k, k, mlp_in),
                _layer(f"L{b}.down_proj", 14336, 4096, k, k, f"L{b}.act")]
    return out


def _qwen7b_layers(k=64, blocks=28):
    out = []
    for b in range(blocks):
        attn_in, mlp_in = f"Q{b}.attn_in", f"Q{b}.mlp_in"
        out += [_layer(f"Q{b}.q_proj", 3584, 3584, k, k, attn_in),
                _layer(f"Q{b}.k_proj", 3584, 512, k, k, attn_in),
                _layer(f"Q{b}.v_proj", 3584, 512, k, k, attn_in),
                _layer(f"Q{b}.o_proj", 3584, 3584, k, k, f"Q{b}.attn_core"),
                _layer(f"Q{b}.gate_proj", 3584, 18944, k, k, mlp_in),
                _layer(f"Q{b}.up_proj", 3584, 18944, k, k, mlp_in),
                _layer(f"Q{b}.down_proj", 18944, 3584, k, k, f"Q{b}.act")]
    return out


def _pythia_layers(blocks=24):
    out = []
    for b in range(blocks):
        out += [_layer(f"l{b}.attention.query_key_value", 1024, 3072, 1, 1, f"l{b}.ln_attn"),
                _layer(f"l{b}.attention.dense", 1024, 1024, 1, 1, f"l{b}.attn_core"),
                _layer(f"l{b}.mlp.dense_h_to_4h", 1024, 4096, 1, 1, f"l{b}.ln_mlp"),
                _layer(f"l{b}.mlp.dense_4h_to_h", 4096, 1024, 1, 1, f"l{b}.act")]
    return out


WORKLOADS = {
    "tiny": {"layers": [_layer("fc", 64, 64, 8, 8, "fc.in")], "T": 16,
             "batch": 12, "n_train": 8, "n_query": 4, "dtype": "f32",
             "dist_a": "normal", "dist_b": "normal", "b_scale": 1.0, "seed": 0},
    "gpt2": {"layers": _gpt2_layers(), "T": 512, "batch": 32, "n_train": 4096,
             "n_query": 256, "dtype": "bf16", "dist_a": "normal",
             "dist_b": "normal", "b_scale": 1e-3, "seed": 2},
    "llama8b": {"layers": _llama_layers(), "T": 2048, "batch": 8,
                "dtype": "bf16", "dist_a": "student_t4", "dist_b": "student_t4",
                "b_scale": 1.0, "seed": 3},
    "routing": {"layers": [_layer("wide", 8192, 28672, 64, 64, "wide.in")],
                "T": 32, "batch": 64, "dtype": "bf16", "dist_a": "normal",
                "dist_b": "normal", "b_scale": 1.0, "seed": 4},
    "lora_b": {"layers": [_layer("lora_B", 8, 4096, 8, 64, "lora.mid")],
               "T": 32, "batch": 64, "dtype": "bf16", "dist_a": "normal",
               "dist_b": "normal", "b_scale": 1.0, "seed": 5},
    "narrow": {"layers": [_layer("narrow", 128, 128, 64, 64, "narrow.in")],
               "T": 2048, "batch": 8, "dtype": "bf16", "dist_a": "normal",
               "dist_b": "normal", "b_scale": 1.0, "seed": 6},
    "score": {"n_train": 200000, "n_query": 2048, "F": 8192, "dtype": "bf16",
              "topk": 100, "d_log10_range": (-3.0, 3.0), "seed": 7},
    "curvature": {"layers": _qwen7b_layers(), "T": 512, "batch": 32, "n_train": 512, "n_query": 1,
                  "dtype": "bf16", "dist_a": "student_t4", "dist_b": "student_t4", "b_scale": 1.0,
                  "seed": 9},
    "crossgram": {"layers": _pythia_layers(), "T_sweep": (32, 128, 512, 2048), "n_train": 8,
                  "n_query": 1, "dtype": "bf16", "dist_a": "normal", "dist_b": "normal",
                  "b_scale": 1.0, "seed": 8},
}

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


def stream_seed(*parts):
    """Stable 63-bit seed from any tuple of labels (independent of PYTHONHASHSEED)."""
    h = hashlib.sha256(repr(parts).encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def _gen(device, *parts):
    g = torch.Generator(device=device)
    g.manual_seed(stream_seed(*parts))
    return g


def draw(shape, dist, dtype, device, *parts, scale=1.0):
    """Seeded sample of ``shape`` in ``dtype`` on ``device``.

    dist "normal": N(0, 1).  dist "student_t4": Student-t with 4 degrees of
    freedom, drawn as Z / sqrt(V / 4) with V = -2 ln(U1 U2) ~ chi-squared(4).
    Values are drawn in float32 and rounded once to ``dtype``.
    """
    g = _gen(device, *parts)
    z = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if dist == "student_t4":
        u = torch.rand((2,) + tuple(shape), generator=g, device=device,
                       dtype=torch.float32).clamp_min_(1e-30)
        v = -2.0 * torch.log(u[0] * u[1])
        z = z / torch.sqrt(v / 4.0)
    elif dist != "normal":
        raise ValueError(dist)
    if scale != 1.0:
        z = z * scale
    return z.to(TORCH_DTYPE[dtype] if isinstance(dtype, str) else dtype)


def factor_blocks(wl, layer_idx, batch_idx, n, T, device, dtype=None, a_cache=None):
    """(A [n, T, d_in], B [n, T, d_out]) for one layer of a workload and batch.

    Layers that share an input group get the identical A tensor (the same object
    when ``a_cache`` is given), as q/k/v and gate/up do in a real block.
    """
    L = wl["layers"][layer_idx]
    dtype = dtype or wl["dtype"]
    key = (L["a_group"], batch_idx, n, T)
    if a_cache is not None and key in a_cache:
        A = a_cache[key]
    else:
        A = draw((n, T, L["d_in"]), wl["dist_a"], dtype, device,
                 wl["seed"], "A", L["a_group"], batch_idx)
        if a_cache is not None:
            a_cache[key] = A
    B = draw((n, T, L["d_out"]), wl["dist_b"], dtype, device,
             wl["seed"], "B", L["name"], batch_idx, scale=wl["b_scale"])
    return A, B


def strided_copy(t, ld):
    """The rows of t in a buffer whose rows are ld >= t.shape[1] elements apart
    (returned as a [rows, F] view; the padding is zero)."""
    if ld is None or ld == t.shape[1]:
        return t
    buf = torch.zeros((t.shape[0], ld), dtype=t.dtype, device=t.device)
    buf[:, :t.shape[1]].copy_(t)
    return buf[:, :t.shape[1]]


def score_inputs(wl, device, n_query=None, n_train=None, F=None, ld=None):
    """(Phi_query, Phi_train, d) for the scoring workload (optionally resized).
    With `ld`, both feature matrices are stored with rows ld elements apart
    (same values as the dense draw)."""
    nq = n_query or wl["n_query"]
    nt = n_train or wl["n_train"]
    F = F or wl["F"]
    q = strided_copy(draw((nq, F), "normal", wl["dtype"], device, wl["seed"], "phi_q"), ld)
    x = strided_copy(draw((nt, F), "normal", wl["dtype"], device, wl["seed"], "phi_train"), ld)
    lo, hi = wl["d_log10_range"]
    g = _gen(device, wl["seed"], "d")
    u = torch.rand(F, generator=g, device=device, dtype=torch.float32)
    d = torch.pow(10.0, lo + (hi - lo) * u)
    return q, x, d


def feature_dim(wl):
    return sum(L["k_in"] * L["k_out"] for L in wl["layers"])
