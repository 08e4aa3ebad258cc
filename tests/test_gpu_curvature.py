"""GPU parity of the K-FAC / EK-FAC curvature path (through the C ABI) against
the float64 oracle (oracle/kfac.py), stage by stage on the same inputs and end
to end.

Each stage is fed the oracle's own values for its inputs (factor blocks and
maps; factor sums; eigenbases; fitted states), so that it is compared element
by element with no dependence on another stage's rounding.

Tolerances (relative Frobenius error):
* factor sums, EK-FAC sums, preconditioned blocks: 1e-5 (float32 accumulation
  of exactly representable products; bf16 inputs are exact in float32 and the
  bf16 MFMA products are exact, so the same bound holds for bf16 captures);
  bf16 outputs: 1e-2 (one rounding to 8 significant bits, 2^-9 relative).
* eigenvalues: 1e-5 of the largest; eigenvectors: reconstruction and
  orthogonality 1e-5, and columns equal up to sign (1e-4) where the oracle's
  spectrum has relative gaps of at least 1e-2 (the eigenvector perturbation
  bound |dA| / gap with |dA| ~ 1e-7 |A| from float32 storage of the sums).
* end to end (fit -> eigen -> correction -> precondition -> score): 1e-3 for
  float32 captures with well-separated spectra (the same gap bound applied
  through the rotation of every example), 2e-2 for bf16; K-FAC alone with the
  seeded maps, whose result does not depend on the eigenbasis: 1e-4.
"""
import numpy as np
import pytest
import torch

import paper_2609_38767_amd as dt
import workloads as W
from gpu_util import host64, oracle_maps, rel_fro
from oracle import gradients as og
from oracle import kfac as ok
from oracle import rng as orng
from paper_2609_38767_amd.session import Curvature, ProjectionSession, feature_rows, score

pytestmark = pytest.mark.gpu
DEV = "cuda"

LAYERS = [dict(name="c0", d_in=100, d_out=72, k_in=24, k_out=40, a_group="g0"),
          dict(name="c1", d_in=100, d_out=18, k_in=8, k_out=8, a_group="g0"),
          dict(name="c2", d_in=40, d_out=256, k_in=16, k_out=64, a_group="g2"),
          dict(name="c3", d_in=9, d_out=13, k_in=5, k_out=3, a_group="g3"),
          dict(name="c4", d_in=320, d_out=64, k_in=64, k_out=64, a_group="g4")]


def _inputs(layers, n, T, dtype, seed, batch=0):
    wl = dict(layers=layers, dtype=dtype, dist_a="student_t4", dist_b="normal", b_scale=1.0, seed=seed)
    cache, out = {}, []
    for li in range(len(layers)):
        out.append(W.factor_blocks(wl, li, batch, n, T, DEV, dtype, a_cache=cache))
    return out


def _session(layers, inputs, dtype, seed, lengths=None):
    s = ProjectionSession(layers, dtype=dtype, seed=seed)
    for li, (A, B) in enumerate(inputs):
        s.capture(li, A, B, lengths)
    return s


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T,lens", [(37, [37, 0, 1, 20, 33]), (1100, [1100, 700, 513, 0, 1099])])
def test_factor_sums(dtype, T, lens):
    n = len(lens)
    print(f"[curvature] factor sums dtype={dtype} T={T}", flush=True)
    inputs = _inputs(LAYERS, n, T, dtype, seed=21)
    lengths = torch.tensor(lens, dtype=torch.int32, device=DEV)
    s = _session(LAYERS, inputs, dtype, 5, lengths)
    c = Curvature(s)
    c.accumulate_factors()
    torch.cuda.synchronize()
    maps = oracle_maps(5, LAYERS, dtype)
    for li, L in enumerate(LAYERS):
        A, B = host64(inputs[li][0]), host64(inputs[li][1])
        SA, SG, nt, ne = ok.factor_sums(A, B, maps[li][0], maps[li][1], lens)
        ga, gg = host64(c.field(li, "sum_a")), host64(c.field(li, "sum_g"))
        ea, eg = rel_fro(ga, SA), rel_fro(gg, SG)
        print(f"  layer {li}: sum_a {ea:.2e} sum_g {eg:.2e}")
        assert ea <= 1e-5 and eg <= 1e-5, (li, ea, eg)
        assert np.array_equal(ga, ga.T) and np.array_equal(gg, gg.T)
        assert c.field(li, "counts").tolist() == [nt, ne, 0]


DMA_LAYERS = [dict(name="d0", d_in=128, d_out=96, k_in=32, k_out=24, a_group="h0"),
              dict(name="d1", d_in=64, d_out=256, k_in=64, k_out=20, a_group="h1")]


def test_factor_sums_direct_load_instances():
    # bf16 sides with 16-byte rows and 2 or 4 map tiles stream their rows by
    # direct loads (k of 20, 24, 32 -> 2 tiles; 64 -> 4), ragged lengths over
    # several row chunks, against the oracle's token loop
    lens = [300, 171, 0]
    n, T = len(lens), 300
    inputs = _inputs(DMA_LAYERS, n, T, "bf16", seed=23)
    lengths = torch.tensor(lens, dtype=torch.int32, device=DEV)
    s = _session(DMA_LAYERS, inputs, "bf16", 9, lengths)
    c = Curvature(s)
    c.accumulate_factors()
    torch.cuda.synchronize()
    maps = oracle_maps(9, DMA_LAYERS, "bf16")
    for li, L in enumerate(DMA_LAYERS):
        A, B = host64(inputs[li][0]), host64(inputs[li][1])
        SA, SG, nt, ne = ok.factor_sums(A, B, maps[li][0], maps[li][1], lens)
        ga, gg = host64(c.field(li, "sum_a")), host64(c.field(li, "sum_g"))
        ea, eg = rel_fro(ga, SA), rel_fro(gg, SG)
        assert ea <= 1e-5 and eg <= 1e-5, (li, ea, eg)
        assert np.array_equal(ga, ga.T) and np.array_equal(gg, gg.T)
        assert c.field(li, "counts").tolist() == [nt, ne, 0]


FIT_CASES = [("auto", None), ("factored", dt.DATTRI_FORM_FUSED), ("factored", dt.DATTRI_FORM_SPLIT),
             ("materialized", None)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("route,form", FIT_CASES)
def test_project_and_fit(dtype, route, form):
    """Projection with the factor sums taken in the same pass: phi equal to the
    plain projection's, sums and counts equal to the oracle's."""
    routes = {"auto": dt.DATTRI_ROUTE_AUTO, "factored": dt.DATTRI_ROUTE_FACTORED,
              "materialized": dt.DATTRI_ROUTE_MATERIALIZED}
    lens = [300, 0, 129, 64]
    n, T = len(lens), 300
    print(f"[curvature] project_and_fit dtype={dtype} route={route} form={form}", flush=True)
    inputs = _inputs(LAYERS, n, T, dtype, seed=61)
    lengths = torch.tensor(lens, dtype=torch.int32, device=DEV)
    s = ProjectionSession(LAYERS, dtype=dtype, seed=7, form=form)
    for li, (A, B) in enumerate(inputs):
        s.capture(li, A, B, lengths)
    c = Curvature(s)
    phi = c.project_and_fit(n, route=routes[route])
    ref_phi = s.project(n, route=routes[route])
    torch.cuda.synchronize()
    assert torch.equal(phi, ref_phi)
    maps = oracle_maps(7, LAYERS, dtype)
    for li in range(len(LAYERS)):
        A, B = host64(inputs[li][0]), host64(inputs[li][1])
        SA, SG, nt, ne = ok.factor_sums(A, B, maps[li][0], maps[li][1], lens)
        ea = rel_fro(host64(c.field(li, "sum_a")), SA)
        eg = rel_fro(host64(c.field(li, "sum_g")), SG)
        assert ea <= 1e-5 and eg <= 1e-5, (li, ea, eg)
        assert c.field(li, "counts").tolist() == [nt, ne, 0]


def test_factor_sums_accumulate_and_reset():
    n, T = 3, 40
    a = _inputs(LAYERS[:2], n, T, "f32", seed=31, batch=0)
    b = _inputs(LAYERS[:2], n, T, "f32", seed=31, batch=1)
    s = _session(LAYERS[:2], a, "f32", 9)
    c = Curvature(s)
    c.accumulate_factors()
    s.clear()
    for li, (A, B) in enumerate(b):
        s.capture(li, A, B)
    c.accumulate_factors()
    torch.cuda.synchronize()
    maps = oracle_maps(9, LAYERS[:2], "f32")
    for li in range(2):
        A = np.concatenate([host64(a[li][0]), host64(b[li][0])])
        B = np.concatenate([host64(a[li][1]), host64(b[li][1])])
        SA, SG, nt, ne = ok.factor_sums(A, B, maps[li][0], maps[li][1])
        assert rel_fro(host64(c.field(li, "sum_a")), SA) <= 1e-5
        assert rel_fro(host64(c.field(li, "sum_g")), SG) <= 1e-5
        assert c.field(li, "counts").tolist() == [2 * n * T, 2 * n, 0]
    c.reset()
    torch.cuda.synchronize()
    assert float(c.field(0, "sum_a").abs().sum()) == 0.0
    assert c.field(1, "counts").tolist() == [0, 0, 0]


def test_project_and_fit_repeated_batches_same_buffers():
    # the usual training loop: each batch written into the captured buffers and
    # fitted with an unchanged plan (its tables stay in the plan buffer); the
    # sums cover both batches and each phi matches its own batch
    n, T = 3, 70
    a = _inputs(LAYERS[:2], n, T, "bf16", seed=41, batch=0)
    b = _inputs(LAYERS[:2], n, T, "bf16", seed=41, batch=1)
    bufs = [(A.clone(), B.clone()) for A, B in a]
    s = _session(LAYERS[:2], bufs, "bf16", 11)
    c = Curvature(s)
    phis = []
    for data in (a, b):
        for (A, B), (A2, B2) in zip(bufs, data):
            A.copy_(A2)
            B.copy_(B2)
        phis.append(c.project_and_fit(n).clone())
    torch.cuda.synchronize()
    maps = oracle_maps(11, LAYERS[:2], "bf16")
    for data, phi in zip((a, b), phis):
        for li, L in enumerate(LAYERS[:2]):
            A, B = host64(data[li][0]), host64(data[li][1])
            o, w = s.offsets[li], L["k_in"] * L["k_out"]
            ref = np.stack([og.project_factored(A[i], B[i], maps[li][0], maps[li][1]).reshape(-1) for i in range(n)])
            assert rel_fro(host64(phi[:, o:o + w]), ref) <= 1e-5
    for li in range(2):
        A = np.concatenate([host64(a[li][0]), host64(b[li][0])])
        B = np.concatenate([host64(a[li][1]), host64(b[li][1])])
        SA, SG, nt, ne = ok.factor_sums(A, B, maps[li][0], maps[li][1])
        assert rel_fro(host64(c.field(li, "sum_a")), SA) <= 1e-5
        assert rel_fro(host64(c.field(li, "sum_g")), SG) <= 1e-5
        assert c.field(li, "counts").tolist() == [2 * n * T, 2 * n, 0]


def _spectrum_matrix(rng, k, lam):
    U, _ = np.linalg.qr(rng.standard_normal((k, k)))
    return (U * lam) @ U.T


def _eig_session(ks):
    layers = [dict(name=f"e{i}", d_in=8, d_out=8, k_in=ka, k_out=kg, a_group=f"e{i}") for i, (ka, kg) in enumerate(ks)]
    return layers, ProjectionSession(layers, dtype="f32", seed=0)


def test_eigen_against_oracle():
    rng = np.random.default_rng(3)
    ks = [(1, 2), (3, 17), (63, 64), (64, 5), (2, 64)]
    layers, s = _eig_session(ks)
    c = Curvature(s)
    mats = []
    for li, (ka, kg) in enumerate(ks):
        # spectra with relative gaps >= 1e-2: geometric ladders times a random basis
        Ma = _spectrum_matrix(rng, ka, 3.0 * 1.05 ** np.arange(ka))
        Mg = _spectrum_matrix(rng, kg, 0.2 * 1.04 ** np.arange(kg))
        na, ng = 1000 + li, 7 + li
        Sa = (Ma * na).astype(np.float32)
        Sg = (Mg * ng).astype(np.float32)
        c.field(li, "sum_a").copy_(torch.from_numpy(Sa))
        c.field(li, "sum_g").copy_(torch.from_numpy(Sg))
        c.field(li, "counts").copy_(torch.tensor([na, ng, 0]))
        mats.append((Sa.astype(np.float64) / na, Sg.astype(np.float64) / ng))
    c.eigen()
    torch.cuda.synchronize()
    for li, (ka, kg) in enumerate(ks):
        for side, M in zip(("a", "g"), mats[li]):
            k = M.shape[0]
            M = 0.5 * (M + M.T)
            lam_o, Q_o = ok.eigenbasis(M)
            lam = host64(c.field(li, "lam_" + side))
            Q = host64(c.field(li, "q_" + side))
            assert np.max(np.abs(lam - lam_o)) <= 1e-5 * np.max(np.abs(lam_o)), (li, side)
            assert np.all(np.diff(lam) >= 0)
            assert rel_fro(Q.T @ Q, np.eye(k)) <= 1e-5
            assert rel_fro((Q * lam) @ Q.T, M) <= 1e-5
            # columns equal up to sign
            dots = np.abs(np.sum(Q * Q_o, axis=0))
            assert np.max(np.abs(dots - 1.0)) <= 1e-4, (li, side, np.min(dots))


def test_eigen_degenerate_cases():
    ks = [(4, 3), (6, 6), (33, 1)]
    layers, s = _eig_session(ks)
    c = Curvature(s)
    rng = np.random.default_rng(4)
    # layer 0: zero counts -> zeros and identity
    # layer 1: a multiple of the identity (every basis is an eigenbasis) and a rank-2 factor
    c.field(1, "sum_a").copy_(torch.eye(6) * 12.0)
    v = rng.standard_normal((2, 6))
    R2 = (v.T @ v).astype(np.float32)
    c.field(1, "sum_g").copy_(torch.from_numpy(R2))
    c.field(1, "counts").copy_(torch.tensor([4, 2, 0]))
    # layer 2: k = 33 (odd: one padded index), plain random SPD; k = 1 side
    M = rng.standard_normal((33, 50))
    S33 = (M @ M.T).astype(np.float32)
    c.field(2, "sum_a").copy_(torch.from_numpy(S33))
    c.field(2, "sum_g").copy_(torch.tensor([[5.0]]))
    c.field(2, "counts").copy_(torch.tensor([10, 4, 0]))
    c.eigen()
    torch.cuda.synchronize()
    assert float(c.field(0, "lam_a").abs().max()) == 0.0
    assert torch.equal(c.field(0, "q_g").cpu(), torch.eye(3))
    assert np.allclose(host64(c.field(1, "lam_a")), 3.0, rtol=1e-6)
    Q = host64(c.field(1, "q_a"))
    assert rel_fro(Q.T @ Q, np.eye(6)) <= 1e-6
    lam_g, Q_g = host64(c.field(1, "lam_g")), host64(c.field(1, "q_g"))
    ref = R2.astype(np.float64) / 2
    assert rel_fro((Q_g * lam_g) @ Q_g.T, ref) <= 1e-5
    assert np.sum(np.abs(lam_g) > 1e-5 * np.max(lam_g)) == 2  # rank 2
    lam_o, _ = ok.eigenbasis(S33.astype(np.float64) / 10)
    assert np.max(np.abs(host64(c.field(2, "lam_a")) - lam_o)) <= 1e-5 * np.max(lam_o)
    assert np.isclose(float(c.field(2, "lam_g")[0]), 1.25, rtol=1e-7)


def _write_oracle_state(c, layers, curv, with_ekfac=True, n_e=None):
    """Oracle-fitted curvature (float32-rounded) into a state; returns the rounded copies."""
    out = []
    for li, C in enumerate(curv):
        Qa = C.Q_a.astype(np.float32)
        Qg = C.Q_g.astype(np.float32)
        la = C.lam_a.astype(np.float32)
        lg = C.lam_g.astype(np.float32)
        c.field(li, "q_a").copy_(torch.from_numpy(Qa))
        c.field(li, "q_g").copy_(torch.from_numpy(Qg))
        c.field(li, "lam_a").copy_(torch.from_numpy(la))
        c.field(li, "lam_g").copy_(torch.from_numpy(lg))
        se = None
        if with_ekfac:
            se = (C.E_ekfac * n_e).astype(np.float32)
            c.field(li, "sum_e").copy_(torch.from_numpy(se))
            c.field(li, "counts").copy_(torch.tensor([1, 1, n_e]))
        out.append((Qa.astype(np.float64), Qg.astype(np.float64), la.astype(np.float64),
                    lg.astype(np.float64), None if se is None else se.astype(np.float64) / n_e))
    return out


def _oracle_curvatures(layers, seed, n, T, dtype):
    inputs = _inputs(layers, n, T, dtype, seed=seed)
    maps = oracle_maps(seed, layers, dtype)
    host = [(host64(A), host64(B)) for A, B in inputs]
    oracle_layers = [dict(A=A, B=B, P_in=P[0], P_out=P[1]) for (A, B), P in zip(host, maps)]
    phi = np.stack([og.feature_vector([og.project_factored(A[i], B[i], P[0], P[1])
                                        for (A, B), P in zip(host, maps)]) for i in range(n)])
    offsets = list(np.cumsum([0] + [L["k_in"] * L["k_out"] for L in layers])[:-1])
    curv = ok.fit_layers(oracle_layers, phi, offsets)
    return inputs, phi, offsets, curv


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ekfac_sums_with_oracle_basis(dtype):
    print(f"[curvature] ekfac sums dtype={dtype}", flush=True)
    layers = LAYERS
    _, phi_fit, offsets, curv = _oracle_curvatures(layers, 41, 6, 24, "f32")
    s = ProjectionSession(layers, dtype="f32", seed=41)
    c = Curvature(s)
    rounded = _write_oracle_state(c, layers, curv, with_ekfac=False)
    rng = np.random.default_rng(5)
    F = s.F
    rows1 = rng.standard_normal((37, F))
    rows2 = rng.standard_normal((5, F))
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    t1 = W.strided_copy(torch.from_numpy(rows1).to(tdt).to(DEV), F + 24)
    t2 = torch.from_numpy(rows2).to(tdt).to(DEV)
    c.accumulate_ekfac(t1)
    c.accumulate_ekfac(t2)
    torch.cuda.synchronize()
    rows = np.concatenate([host64(t1), host64(t2)])
    for li, L in enumerate(layers):
        Qa, Qg = rounded[li][0], rounded[li][1]
        o, w = offsets[li], L["k_in"] * L["k_out"]
        psis = [r[o:o + w].reshape(L["k_in"], L["k_out"]) for r in rows]
        want = ok.ekfac_sums(psis, Qa, Qg)
        got = host64(c.field(li, "sum_e"))
        e = rel_fro(got, want)
        print(f"  layer {li}: {e:.2e}")
        assert e <= 1e-5, (li, e)
        assert int(c.field(li, "counts")[2]) == 42


@pytest.mark.parametrize("kind", ["kfac", "ekfac"])
@pytest.mark.parametrize("in_dt,out_dt", [("f32", "f32"), ("bf16", "f32"), ("f32", "bf16")])
@pytest.mark.parametrize("rel,abs_", [(0.1, 0.0), (0.0, 1e-3), (0.5, 0.2)])
def test_precondition_with_oracle_state(kind, in_dt, out_dt, rel, abs_):
    layers = LAYERS
    n_e = 6
    _, _, offsets, curv = _oracle_curvatures(layers, 43, n_e, 20, "f32")
    s = ProjectionSession(layers, dtype="f32", seed=43)
    c = Curvature(s)
    rounded = _write_oracle_state(c, layers, curv, n_e=n_e)
    rng = np.random.default_rng(6)
    q = rng.standard_normal((11, s.F))
    tq = torch.from_numpy(q).to(torch.float32 if in_dt == "f32" else torch.bfloat16).to(DEV)
    tq = W.strided_copy(tq, s.F + 8)
    out = c.precondition(tq, kind, rel, abs_, out_dtype=out_dt)
    torch.cuda.synchronize()
    qh = host64(tq)
    got = host64(out)
    for li, L in enumerate(layers):
        Qa, Qg, la, lg, Ee = rounded[li]
        E = ok.kfac_eigenvalues(la, lg) if kind == "kfac" else Ee
        delta = ok.damping(E, rel, abs_)
        o, w = offsets[li], L["k_in"] * L["k_out"]
        want = np.stack([ok.precondition(r[o:o + w].reshape(L["k_in"], L["k_out"]), Qa, Qg, E, delta).reshape(-1)
                         for r in qh])
        e = rel_fro(got[:, o:o + w], want)
        assert e <= (1e-5 if out_dt == "f32" else 1e-2), (li, e)


def _end_to_end(dtype, layers, seed, overrides, kinds, tol):
    """Fit on two capture batches, eigendecompose, correct, precondition the
    queries and score, against the oracle's curvature scores."""
    n, T = 12, 64
    # anisotropic factors (column scales 1.15^j and 1.12^j)
    batches = []
    for b in range(2):
        ins = _inputs(layers, n, T, dtype, seed=seed, batch=b)
        scaled = []
        for li, (A, B) in enumerate(ins):
            sa = (1.15 ** torch.arange(A.shape[2], device=DEV, dtype=torch.float32)).to(A.dtype)
            sb = (1.12 ** torch.arange(B.shape[2], device=DEV, dtype=torch.float32)).to(B.dtype)
            scaled.append(((A * sa).contiguous(), (B * sb).contiguous()))
        batches.append(scaled)
    s = ProjectionSession(layers, dtype=dtype, seed=seed, overrides=overrides)
    c = Curvature(s)
    phis = []
    for b in range(2):
        s.clear()
        for li, (A, B) in enumerate(batches[b]):
            s.capture(li, A, B)
        c.accumulate_factors()
        phis.append(s.project(n, phi_dtype="f32").clone())
    phi_t = torch.cat(phis)
    c.eigen()
    c.accumulate_ekfac(phi_t)
    rng = np.random.default_rng(7)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    queries = torch.from_numpy(rng.standard_normal((3, s.F))).to(tdt).to(DEV)
    if overrides:
        maps = [tuple(np.asarray(m, dtype=np.float64) for m in overrides[li]) for li in range(len(layers))]
    else:
        maps = oracle_maps(seed, layers, dtype)
    host = [[(host64(A), host64(B)) for A, B in batches[b]] for b in range(2)]
    oracle_layers = [dict(A=np.concatenate([host[0][li][0], host[1][li][0]]),
                          B=np.concatenate([host[0][li][1], host[1][li][1]]),
                          P_in=maps[li][0], P_out=maps[li][1]) for li in range(len(layers))]
    phi_o = np.stack([og.feature_vector([og.project_factored(L["A"][i], L["B"][i], L["P_in"], L["P_out"])
                                         for L in oracle_layers]) for i in range(2 * n)])
    offsets = list(np.cumsum([0] + [L["k_in"] * L["k_out"] for L in layers])[:-1])
    curv = ok.fit_layers(oracle_layers, phi_o, offsets)
    qh = host64(queries)
    gap = min(float(np.min(np.diff(lam)) / np.max(lam)) for C in curv for lam in (C.lam_a, C.lam_g))
    for kind in kinds:
        pq = c.precondition(queries, kind, out_dtype="f32")
        S, _, _ = score(pq, phi_t)
        torch.cuda.synchronize()
        want = ok.curvature_scores(qh, phi_o, curv, offsets, kind)
        e = rel_fro(host64(S), want)
        print(f"  {kind}: scores rel err {e:.2e} (smallest relative eigengap {gap:.1e})")
        assert e <= tol, (kind, e)
    return gap


E2E_LAYERS = [dict(name="x0", d_in=96, d_out=80, k_in=16, k_out=24, a_group="x0"),
              dict(name="x1", d_in=64, d_out=48, k_in=8, k_out=8, a_group="x1")]


def _leading_maps(layers):
    """Maps that keep the leading k coordinates: P = [I_k; 0] (d x k)."""
    out = {}
    for li, L in enumerate(layers):
        out[li] = tuple(np.ascontiguousarray(np.eye(d, k, dtype=np.float32))
                        for d, k in ((L["d_in"], L["k_in"]), (L["d_out"], L["k_out"])))
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_end_to_end_scores(dtype):
    """Both curvature kinds end to end.  The maps keep the leading coordinates
    of the anisotropic factors, so the fitted spectra have relative gaps of at
    least 1e-3 (checked), the condition the 1e-3 bound rests on."""
    print(f"[curvature] end to end dtype={dtype}", flush=True)
    gap = _end_to_end(dtype, E2E_LAYERS, 51, _leading_maps(E2E_LAYERS), ("kfac", "ekfac"),
                      1e-3 if dtype == "f32" else 2e-2)
    assert gap >= 1e-3


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_end_to_end_kfac_seeded_maps(dtype):
    """K-FAC end to end with the seeded Gaussian maps.  Its preconditioned block
    (A (x) S + delta I)^{-1} vec(Psi) is a smooth function of the factors (no
    eigenvector sensitivity), bounded by the damped condition number times the
    float32 error of the sums: 1e-4 for float32 captures."""
    print(f"[curvature] end to end seeded maps dtype={dtype}", flush=True)
    _end_to_end(dtype, E2E_LAYERS, 52, None, ("kfac",), 1e-4 if dtype == "f32" else 2e-2)


def test_curvature_full_size_sampled():
    """The Qwen2.5-7B-shaped batch of the curvature benchmark (196 layers,
    32 x 512 token rows, k = 64, bf16) through dattri_project_and_fit in the
    launch configuration bench.py times, then the eigendecompositions and the
    EK-FAC correction; sampled layers against the oracle:
    * phi blocks of two examples and the factor sums and counts: 1e-5;
    * eigenvalues (unique, unlike eigenvectors): 1e-4 of the largest;
    * EK-FAC: the total of the corrected sums equals sum_i ||Psi_i||_F^2 (the
      rotation keeps Frobenius norms; holds at any size): 1e-4;
    * K-FAC preconditioned query block against the oracle's own fit: 1e-3 (a
      smooth function of the factors, float32 sums)."""
    wl = W.WORKLOADS["curvature"]
    layers, n, T, seed = wl["layers"], wl["batch"], wl["T"], wl["seed"]
    print("[curvature] full-size sampled: building inputs", flush=True)
    cache, inputs = {}, []
    s = ProjectionSession(layers, dtype="bf16", seed=seed)
    for li in range(len(layers)):
        A, B = W.factor_blocks(wl, li, 0, n, T, DEV, "bf16", a_cache=cache)
        s.capture(li, A, B)
        inputs.append((A, B))
    c = Curvature(s)
    phi = c.project_and_fit(n)
    c.eigen()
    c.accumulate_ekfac(phi)
    rng = np.random.default_rng(11)
    q = torch.from_numpy(rng.standard_normal((1, s.F))).to(torch.float32).to(DEV)
    pq = c.precondition(q, "kfac")
    torch.cuda.synchronize()
    assert torch.isfinite(phi).all() and torch.isfinite(pq).all()
    sampled = [0, 6, 7 * 27 + 4]  # q_proj and down_proj of block 0, gate_proj of block 27
    for li in sampled:
        L = layers[li]
        print(f"[curvature] full-size sampled: layer {li} ({L['name']})", flush=True)
        P_in, P_out = orng.projection_pair(seed, li, L["d_in"], L["d_out"], L["k_in"], L["k_out"], "bf16")
        A, B = host64(inputs[li][0]), host64(inputs[li][1])
        SA, SG, nt, ne = ok.factor_sums(A, B, P_in, P_out)
        assert rel_fro(host64(c.field(li, "sum_a")), SA) <= 1e-5
        assert rel_fro(host64(c.field(li, "sum_g")), SG) <= 1e-5
        assert c.field(li, "counts").tolist() == [n * T, n, n]
        off, w = s.offsets[li], L["k_in"] * L["k_out"]
        psis = [og.project_factored(A[i], B[i], P_in, P_out) for i in range(n)]
        for i in (0, n - 1):
            assert rel_fro(host64(phi[i, off:off + w]), psis[i].reshape(-1)) <= 1e-5
        C = ok.LayerCurvature(SA, SG, nt, ne)
        for side, lam_o in (("a", C.lam_a), ("g", C.lam_g)):
            lam = host64(c.field(li, "lam_" + side))
            assert np.max(np.abs(lam - lam_o)) <= 1e-4 * np.max(np.abs(lam_o)), (li, side)
        tot = float(host64(c.field(li, "sum_e")).sum())
        want = sum(float(np.sum(P ** 2)) for P in psis)
        assert abs(tot - want) <= 1e-4 * want, (li, tot, want)
        Xq = host64(q[0, off:off + w]).reshape(L["k_in"], L["k_out"])
        ref = C.precondition(Xq, "kfac")
        e = rel_fro(host64(pq[0, off:off + w]).reshape(L["k_in"], L["k_out"]), ref)
        print(f"  layer {li}: K-FAC preconditioned block rel err {e:.2e}")
        assert e <= 1e-3, (li, e)
