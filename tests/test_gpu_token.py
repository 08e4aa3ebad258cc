"""GPU parity of token-level attribution (through the C ABI) against the
float64 oracle (oracle/token.py).

* token scores of seeded query rows: relative Frobenius error <= 1e-5 (float32
  sums of exact products, bf16 captures included);
* property at any size: per training example, the token scores sum to the
  sequence score <phi_q, phi_i> computed by the score kernel from the phi the
  same call wrote (1e-4 relative to the largest |score|, float32 sums in two
  orders), for GradDot rows and for K-FAC / EK-FAC preconditioned rows;
* positions past an example's length are exactly zero."""
import numpy as np
import pytest
import torch

import paper_2609_38767_amd as dt
import workloads as W
from gpu_util import host64, oracle_maps, rel_fro
from oracle import rng as orng
from oracle import token as otk
from paper_2609_38767_amd.session import Curvature, ProjectionSession, score

pytestmark = pytest.mark.gpu
DEV = "cuda"

LAYERS = [dict(name="t0", d_in=100, d_out=72, k_in=24, k_out=40, a_group="g0"),
          dict(name="t1", d_in=100, d_out=18, k_in=8, k_out=8, a_group="g0"),
          dict(name="t2", d_in=40, d_out=256, k_in=16, k_out=64, a_group="g2"),
          dict(name="t3", d_in=320, d_out=64, k_in=64, k_out=64, a_group="g4")]
FORMS = {"fused": dt.DATTRI_FORM_FUSED, "split": dt.DATTRI_FORM_SPLIT}


def _inputs(layers, n, T, dtype, seed):
    wl = dict(layers=layers, dtype=dtype, dist_a="normal", dist_b="normal", b_scale=1.0, seed=seed)
    cache = {}
    return [W.factor_blocks(wl, li, 0, n, T, DEV, dtype, a_cache=cache) for li in range(len(layers))]


def _sums_match(scores, phi_q, phi):
    S, _, _ = score(phi_q.float().contiguous(), phi.float().contiguous())
    tok = scores.sum(dim=2)
    torch.cuda.synchronize()
    err = (tok - S).abs().max().item() / max(S.abs().max().item(), 1e-30)
    return err


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("form", ["fused", "split"])
@pytest.mark.parametrize("n_q", [6, 3, 1])  # query groups of 4 + 2 slots; 2 + 1 (two-slot instance); one row
def test_token_scores_against_oracle(dtype, form, n_q):
    print(f"[token] dtype={dtype} form={form} n_q={n_q}", flush=True)
    lens = [150, 0, 64, 149, 1]
    n, T = len(lens), 150
    inputs = _inputs(LAYERS, n, T, dtype, seed=71)
    lengths = torch.tensor(lens, dtype=torch.int32, device=DEV)
    s = ProjectionSession(LAYERS, dtype=dtype, seed=73, form=FORMS[form])
    for li, (A, B) in enumerate(inputs):
        s.capture(li, A, B, lengths)
    g = torch.Generator(device=DEV).manual_seed(75)
    phi_q = torch.randn((n_q, s.F), generator=g, device=DEV)
    scores, phi = s.token_scores(phi_q, n)
    torch.cuda.synchronize()
    maps = oracle_maps(73, LAYERS, dtype)
    oracle_layers = [dict(A=host64(A), B=host64(B), P_in=P[0], P_out=P[1], lengths=lens)
                     for (A, B), P in zip(inputs, maps)]
    qh = host64(phi_q)
    got = host64(scores)
    for q in range(n_q):
        blocks = []
        for li, L in enumerate(LAYERS):
            o, w = s.offsets[li], L["k_in"] * L["k_out"]
            blocks.append(qh[q, o:o + w].reshape(L["k_in"], L["k_out"]))
        ref = otk.token_scores(oracle_layers, blocks)
        e = rel_fro(got[q], ref)
        assert e <= 1e-5, (q, e)
        for i, Ti in enumerate(lens):
            assert np.all(got[q, i, Ti:] == 0.0)
    assert _sums_match(scores, phi_q, phi) <= 1e-4
    # phi written by the same call equals the plain projection
    ref_phi = s.project(n, route=dt.DATTRI_ROUTE_FACTORED)
    torch.cuda.synchronize()
    assert torch.equal(phi, ref_phi)


@pytest.mark.parametrize("kind", ["kfac", "ekfac"])
def test_token_sums_are_curvature_scores(kind):
    n, T = 8, 96
    inputs = _inputs(LAYERS, n, T, "bf16", seed=81)
    s = ProjectionSession(LAYERS, dtype="bf16", seed=83)
    for li, (A, B) in enumerate(inputs):
        s.capture(li, A, B)
    c = Curvature(s)
    phi = c.project_and_fit(n)
    c.eigen()
    c.accumulate_ekfac(phi)
    g = torch.Generator(device=DEV).manual_seed(85)
    q = torch.randn((3, s.F), generator=g, device=DEV)
    pq = c.precondition(q, kind, out_dtype="f32")
    scores, phi2 = s.token_scores(pq, n)
    torch.cuda.synchronize()
    assert _sums_match(scores, pq, phi2) <= 1e-4


@pytest.mark.timeout(600)
def test_token_scores_full_size_sampled():
    """The curvature workload's batch (196 Qwen2.5-7B-shaped layers, 32 x 512
    tokens, k = 64) with one query row: token scores at sampled (example,
    position) pairs against the oracle (each needs only that token row of
    every layer), and the property at every position: token sums equal the
    sequence scores."""
    wl = W.WORKLOADS["curvature"]
    layers, n, T = wl["layers"], wl["batch"], wl["T"]
    print("[token] full size: building inputs", flush=True)
    cache = {}
    s = ProjectionSession(layers, dtype="bf16", seed=wl["seed"])
    inputs = []
    for li in range(len(layers)):
        A, B = W.factor_blocks(wl, li, 0, n, T, DEV, "bf16", a_cache=cache)
        s.capture(li, A, B)
        inputs.append((A, B))
    g = torch.Generator(device=DEV).manual_seed(87)
    q = torch.randn((1, s.F), generator=g, device=DEV)
    scores, phi = s.token_scores(q, n)
    torch.cuda.synchronize()
    assert torch.isfinite(scores).all()
    assert _sums_match(scores, q, phi) <= 1e-4
    pairs = [(0, 0), (0, 511), (5, 17), (13, 256), (17, 333), (21, 100), (31, 0), (31, 511)]
    ei = torch.tensor([p[0] for p in pairs], device=DEV)
    ti = torch.tensor([p[1] for p in pairs], device=DEV)
    print("[token] full size: oracle at 8 sampled positions over 196 layers", flush=True)
    qh = host64(q)[0]
    oracle_layers, blocks = [], []
    for li, L in enumerate(layers):
        A, B = inputs[li]
        P_in, P_out = orng.projection_pair(wl["seed"], li, L["d_in"], L["d_out"], L["k_in"], L["k_out"], "bf16")
        # each sampled token row as a one-token example: [8, 1, d]
        oracle_layers.append(dict(A=host64(A[ei, ti])[:, None, :], B=host64(B[ei, ti])[:, None, :],
                                  P_in=P_in, P_out=P_out))
        o, w = s.offsets[li], L["k_in"] * L["k_out"]
        blocks.append(qh[o:o + w].reshape(L["k_in"], L["k_out"]))
    ref = otk.token_scores(oracle_layers, blocks)[:, 0]
    got = host64(scores[0, ei, ti])
    err = rel_fro(got, ref)
    print(f"[token] full size sampled rel err {err:.3e}", flush=True)
    assert err <= 1e-5, (got, ref)
