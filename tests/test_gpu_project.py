"""GPU parity of per-example projected gradients (through the C ABI) against the
float64 oracle, element by element on the same seeded inputs.

Tolerance: relative Frobenius error per layer block over the checked examples,
1e-5 for float32 inputs and 2e-2 for bf16 inputs."""
import numpy as np
import pytest
import torch

import paper_2609_38767_amd as dt
import workloads as W
from gpu_util import host64, oracle_maps, oracle_phi_rows, per_layer_errors, rel_fro
from oracle import gradients as og
from oracle import rng as orng
from paper_2609_38767_amd.session import ProjectionSession

pytestmark = pytest.mark.gpu
TOL = {"f32": 1e-5, "bf16": 2e-2}
ROUTES = {"auto": dt.DATTRI_ROUTE_AUTO, "factored": dt.DATTRI_ROUTE_FACTORED,
          "materialized": dt.DATTRI_ROUTE_MATERIALIZED}
FORMS = {"fused": dt.DATTRI_FORM_FUSED, "split": dt.DATTRI_FORM_SPLIT, None: None}
DEV = "cuda"


def _session_inputs(wl, layers, n, T, dtype, device=DEV):
    cache, inputs = {}, []
    wl = dict(wl, layers=layers)
    for li in range(len(layers)):
        A, B = W.factor_blocks(wl, li, 0, n, T, device, dtype, a_cache=cache)
        inputs.append((A, B))
    return inputs


def _run(layers, inputs, dtype, seed, route, phi_dtype="f32", lengths=None, overrides=None, form=None):
    s = ProjectionSession(layers, dtype=dtype, seed=seed, overrides=overrides, form=FORMS[form])
    n = inputs[0][0].shape[0]
    for li, (A, B) in enumerate(inputs):
        s.capture(li, A, B, lengths)
    phi = s.project(n, route=ROUTES[route], phi_dtype=phi_dtype)
    torch.cuda.synchronize()
    return s, phi


def _check(layers, inputs, phi, seed, dtype, examples, lengths=None, tol=None):
    maps = oracle_maps(seed, layers, dtype)
    host = [(host64(A), host64(B)) for A, B in inputs]
    ref = oracle_phi_rows(layers, maps, host, examples, None if lengths is None else lengths.cpu().numpy())
    got = host64(phi)[examples]
    errs = per_layer_errors(got, ref, layers)
    assert np.all(np.isfinite(got))
    assert max(errs) <= (tol or TOL[dtype]), errs
    return errs


@pytest.mark.parametrize("route,form", [("auto", None), ("factored", "fused"), ("factored", "split"),
                                        ("materialized", None)])
def test_tiny_f32_all_routes(route, form):
    wl = W.WORKLOADS["tiny"]
    inputs = _session_inputs(wl, wl["layers"], wl["batch"], wl["T"], "f32")
    s, phi = _run(wl["layers"], inputs, "f32", wl["seed"], route, form=form)
    errs = _check(wl["layers"], inputs, phi, wl["seed"], "f32", list(range(wl["batch"])))
    print(f"tiny {route}: per-layer rel err {errs}")
    if route == "auto":
        assert s.routes()[0][0] == dt.DATTRI_ROUTE_FACTORED


RAGGED = [dict(name="r0", d_in=100, d_out=72, k_in=24, k_out=40, a_group="g0"),
          dict(name="r1", d_in=100, d_out=18, k_in=8, k_out=8, a_group="g0"),
          dict(name="r2", d_in=40, d_out=256, k_in=16, k_out=64, a_group="g2"),
          dict(name="r3", d_in=9, d_out=13, k_in=5, k_out=3, a_group="g3")]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("route,form", [("factored", "fused"), ("factored", "split"), ("materialized", None)])
def test_ragged_unaligned_lengths(dtype, route, form):
    wl = dict(W.WORKLOADS["tiny"], dist_a="normal", dist_b="normal", seed=11)
    n, T = 5, 37
    inputs = _session_inputs(wl, RAGGED, n, T, dtype)
    lengths = torch.tensor([37, 0, 1, 20, 33], dtype=torch.int32, device=DEV)
    s, phi = _run(RAGGED, inputs, dtype, 77, route, lengths=lengths, form=form)
    # example 1 has length 0: its whole row must be exactly zero
    assert torch.count_nonzero(phi[1]).item() == 0
    tol = 1e-5 if dtype == "f32" else 1e-5  # inputs are exact bf16 values; accumulation is float32
    _check(RAGGED, inputs, phi, 77, dtype, [0, 2, 3, 4], lengths=lengths, tol=tol)


@pytest.mark.parametrize("form", ["fused", "split"])
def test_token_chunks_and_lengths_at_chunk_edges(form):
    # T = 300 splits each example's tokens over several contraction chunks in
    # the split form; lengths fall on and beside chunk boundaries
    layers = [dict(name="c0", d_in=200, d_out=135, k_in=40, k_out=24, a_group="a"),
              dict(name="c1", d_in=200, d_out=64, k_in=16, k_out=64, a_group="a")]
    wl = dict(W.WORKLOADS["tiny"], dist_a="normal", dist_b="normal", seed=13)
    n, T = 3, 300
    for dtype in ("f32", "bf16"):
        inputs = _session_inputs(wl, layers, n, T, dtype)
        lengths = torch.tensor([300, 129, 64], dtype=torch.int32, device=DEV)
        _, phi = _run(layers, inputs, dtype, 9, "factored", lengths=lengths, form=form)
        _check(layers, inputs, phi, 9, dtype, [0, 1, 2], lengths=lengths, tol=1e-5)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fused_64_wide_maps(dtype):
    # k_in = k_out = 64: the 4 x 4-tile fused instance, several sub-chunks per
    # work item, ragged lengths
    layers = [dict(name="w0", d_in=264, d_out=200, k_in=64, k_out=64, a_group="a"),
              dict(name="w1", d_in=96, d_out=520, k_in=64, k_out=60, a_group="b")]
    wl = dict(W.WORKLOADS["tiny"], dist_a="normal", dist_b="normal", seed=17)
    n, T = 4, 700
    inputs = _session_inputs(wl, layers, n, T, dtype)
    lengths = torch.tensor([700, 513, 128, 1], dtype=torch.int32, device=DEV)
    _, phi = _run(layers, inputs, dtype, 19, "factored", lengths=lengths, form="fused")
    _check(layers, inputs, phi, 19, dtype, [0, 1, 2, 3], lengths=lengths, tol=1e-5)


def test_fused_direct_lds_path_ragged():
    # bf16 layers with 16-byte aligned rows and 17..32-wide maps on both sides
    # take the fused kernel's direct-to-LDS path (two map tiles per side):
    # d not a multiple of the 64-column stage (520: 17 k-blocks, the last
    # stage half empty; 200; 72), a member with one output tile, sub-chunks of
    # 256 rows ragged by length, a zero-length example
    layers = [dict(name="d0", d_in=520, d_out=200, k_in=32, k_out=32, a_group="a"),
              dict(name="d1", d_in=520, d_out=72, k_in=20, k_out=16, a_group="b"),
              dict(name="d2", d_in=64, d_out=40, k_in=32, k_out=24, a_group="c")]
    wl = dict(W.WORKLOADS["tiny"], dist_a="student_t4", dist_b="student_t4", seed=97)
    n, T = 4, 600
    inputs = _session_inputs(wl, layers, n, T, "bf16")
    lengths = torch.tensor([600, 0, 257, 1], dtype=torch.int32, device=DEV)
    _, phi = _run(layers, inputs, "bf16", 99, "factored", lengths=lengths, form="fused")
    assert torch.count_nonzero(phi[1]).item() == 0
    _check(layers, inputs, phi, 99, "bf16", [0, 2, 3], lengths=lengths, tol=1e-5)
    # the register path (split form's stage 1 streams the same rows) agrees to rounding
    _, phi_s = _run(layers, inputs, "bf16", 99, "factored", lengths=lengths, form="split")
    assert rel_fro(host64(phi_s), host64(phi)) < 1e-6


def test_grouped_direct_lds_path_ragged():
    # layers sharing an input block run as one work item of the direct-to-LDS
    # kernel when their input maps add up to 4 or 6 tiles and no output map
    # exceeds 2 tiles: a q/k/v-like group of 2 + 1 + 2 input tiles (instance of
    # 6, the last tile unused) and a gate/up-like pair of 2 + 2, d_in not a
    # multiple of the 64-column stage, ragged lengths and an empty example
    layers = [dict(name="q", d_in=520, d_out=200, k_in=32, k_out=32, a_group="a"),
              dict(name="k", d_in=520, d_out=72, k_in=16, k_out=16, a_group="a"),
              dict(name="v", d_in=520, d_out=136, k_in=24, k_out=32, a_group="a"),
              dict(name="gate", d_in=192, d_out=264, k_in=32, k_out=32, a_group="b"),
              dict(name="up", d_in=192, d_out=264, k_in=32, k_out=24, a_group="b"),
              dict(name="down", d_in=264, d_out=192, k_in=32, k_out=32, a_group="c")]
    wl = dict(W.WORKLOADS["tiny"], dist_a="student_t4", dist_b="student_t4", seed=101)
    n, T = 5, 600
    inputs = _session_inputs(wl, layers, n, T, "bf16")
    assert inputs[0][0] is inputs[2][0] and inputs[3][0] is inputs[4][0]
    lengths = torch.tensor([600, 0, 257, 1, 511], dtype=torch.int32, device=DEV)
    _, phi = _run(layers, inputs, "bf16", 103, "factored", lengths=lengths, form="fused")
    assert torch.count_nonzero(phi[1]).item() == 0
    _check(layers, inputs, phi, 103, "bf16", [0, 2, 3, 4], lengths=lengths, tol=1e-5)
    # the split form (register path, one factor block at a time) agrees to rounding
    _, phi_s = _run(layers, inputs, "bf16", 103, "factored", lengths=lengths, form="split")
    assert rel_fro(host64(phi_s), host64(phi)) < 1e-6


def test_wide_map_direct_lds_path_ragged():
    # 4-tile output maps (k_out 49..64) on the direct-to-LDS path: a (4, 4)
    # layer, a (2, 4) layer and a (4, 4) layer whose input block is shared
    # with a (2, 2) one (4 + 2 input tiles exceed the 4-tile instance, so
    # they stay apart); d not a multiple of the 64-column stage, ragged lengths
    # and an empty example, against the oracle and the split form
    layers = [dict(name="w0", d_in=584, d_out=200, k_in=64, k_out=64, a_group="a"),
              dict(name="w1", d_in=584, d_out=72, k_in=32, k_out=32, a_group="a"),
              dict(name="w2", d_in=136, d_out=520, k_in=24, k_out=56, a_group="b"),
              dict(name="w3", d_in=200, d_out=64, k_in=56, k_out=49, a_group="c")]
    wl = dict(W.WORKLOADS["tiny"], dist_a="student_t4", dist_b="student_t4", seed=107)
    n, T = 5, 600
    inputs = _session_inputs(wl, layers, n, T, "bf16")
    lengths = torch.tensor([600, 0, 257, 1, 511], dtype=torch.int32, device=DEV)
    _, phi = _run(layers, inputs, "bf16", 109, "factored", lengths=lengths, form="fused")
    assert torch.count_nonzero(phi[1]).item() == 0
    _check(layers, inputs, phi, 109, "bf16", [0, 2, 3, 4], lengths=lengths, tol=1e-5)
    _, phi_s = _run(layers, inputs, "bf16", 109, "factored", lengths=lengths, form="split")
    assert rel_fro(host64(phi_s), host64(phi)) < 1e-6


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("route,form", [("factored", "fused"), ("factored", "split"), ("materialized", None)])
def test_rademacher_maps(dtype, route, form):
    # App. A.2 "Random maps": +-1/sqrt(k) entries from the same per-layer seeds
    layers = RAGGED
    wl = dict(W.WORKLOADS["tiny"], dist_a="normal", dist_b="normal", seed=23)
    n, T = 4, 41
    inputs = _session_inputs(wl, layers, n, T, dtype)
    s = ProjectionSession(layers, dtype=dtype, seed=29, form=FORMS[form], map_kind=dt.DATTRI_MAP_RADEMACHER)
    for li, (A, B) in enumerate(inputs):
        s.capture(li, A, B)
    phi = s.project(n, route=ROUTES[route])
    torch.cuda.synchronize()
    maps = [orng.projection_pair(29, i, L["d_in"], L["d_out"], L["k_in"], L["k_out"], dtype, kind="rademacher")
            for i, L in enumerate(layers)]
    host = [(host64(A), host64(B)) for A, B in inputs]
    ref = oracle_phi_rows(layers, maps, host, list(range(n)))
    errs = per_layer_errors(host64(phi), ref, layers)
    assert max(errs) <= 1e-5, errs
    # switching a bound layer's kind unbinds it
    dt.dattri_set_map_kind(s.ctx, 0, dt.DATTRI_MAP_GAUSSIAN)
    with pytest.raises(dt.DattriError) as e:
        s.project(n, route=ROUTES[route])
    assert e.value.status_name == "E_STATE"


MASKED = [dict(name="m0", d_in=300, d_out=128, k_in=1, k_out=512, mask_size=512, mask_id=0, a_group="ma"),
          dict(name="m1", d_in=300, d_out=128, k_in=1, k_out=1536, mask_size=512, mask_id=3, mask_count=3,
               a_group="ma"),
          dict(name="m2", d_in=256, d_out=256, k_in=1, k_out=30000, mask_size=30000, mask_id=0, a_group="mb"),
          dict(name="m3", d_in=37, d_out=21, k_in=1, k_out=100, mask_size=100, mask_id=1, a_group="mc"),
          dict(name="m4", d_in=257, d_out=255, k_in=1, k_out=30000, mask_size=30000, mask_id=0, a_group="md"),
          dict(name="x", d_in=64, d_out=48, k_in=8, k_out=8, a_group="xa")]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("route", ["auto", "materialized"])
def test_mask_layers(dtype, route):
    # App. A.2 random masks: DW entries gathered from the factors; a whole
    # entry group plus a partial one (m = 30000, aligned and unaligned rows),
    # a small unaligned layer (37 x 21), ragged lengths over several token
    # chunks, an ordinary layer beside them (its route forced)
    from oracle import mask as om
    wl = dict(W.WORKLOADS["tiny"], dist_a="normal", dist_b="normal", seed=31)
    n, T = 4, 300
    inputs = _session_inputs(wl, MASKED, n, T, dtype)
    lengths = torch.tensor([300, 0, 17, 299], dtype=torch.int32, device=DEV)
    s = ProjectionSession(MASKED, dtype=dtype, seed=41)
    for li, (A, B) in enumerate(inputs):
        s.capture(li, A, B, lengths)
    phi = s.project(n, route=ROUTES[route])
    torch.cuda.synchronize()
    assert [r[0] for r in s.routes()[:5]] == [dt.DATTRI_ROUTE_MASK] * 5
    lens = lengths.cpu().numpy()
    got = host64(phi)
    assert np.count_nonzero(got[1]) == 0  # length 0
    for li, L in enumerate(MASKED):
        A, B = host64(inputs[li][0]), host64(inputs[li][1])
        off, w = s.offsets[li], L["k_in"] * L["k_out"]
        if "mask_size" in L:
            parts = [om.mask_indices(41, li, L["d_in"], L["d_out"], L["mask_size"], L["mask_id"] + j)
                     for j in range(L.get("mask_count", 1))]
            rows = np.concatenate([p[0] for p in parts])
            cols = np.concatenate([p[1] for p in parts])
            r_lib, c_lib = dt.dattri_get_mask(s.ctx, li)
            np.testing.assert_array_equal(r_lib, rows)
            ref = np.stack([om.masked_gradient(A[i], B[i], rows, cols, int(lens[i])) for i in range(n)])
        else:
            P_in, P_out = orng.projection_pair(41, li, L["d_in"], L["d_out"], L["k_in"], L["k_out"], dtype)
            ref = np.stack([og.project_factored(A[i], B[i], P_in, P_out, int(lens[i])).reshape(-1)
                            for i in range(n)])
        e = rel_fro(got[:, off:off + w], ref)
        assert e <= 1e-5, (li, e)


def test_mask_layer_wider_than_byte_offsets():
    # a bf16 mask layer with d_out = 33000 (its rows' byte offsets do not fit
    # 16 bits): the call's gather keeps element indices and float32 FMA for
    # every mask layer, the narrow one beside it included
    from oracle import mask as om
    layers = [dict(name="w", d_in=40, d_out=33000, k_in=1, k_out=5000, mask_size=5000, mask_id=0, a_group="wa"),
              dict(name="n", d_in=64, d_out=48, k_in=1, k_out=700, mask_size=700, mask_id=0, a_group="wb")]
    wl = dict(W.WORKLOADS["tiny"], dist_a="normal", dist_b="normal", seed=33)
    n, T = 2, 40
    inputs = _session_inputs(wl, layers, n, T, "bf16")
    lengths = torch.tensor([40, 23], dtype=torch.int32, device=DEV)
    s = ProjectionSession(layers, dtype="bf16", seed=43)
    for li, (A, B) in enumerate(inputs):
        s.capture(li, A, B, lengths)
    phi = s.project(n)
    torch.cuda.synchronize()
    got = host64(phi)
    lens = lengths.cpu().numpy()
    for li, L in enumerate(layers):
        A, B = host64(inputs[li][0]), host64(inputs[li][1])
        rows, cols = om.mask_indices(43, li, L["d_in"], L["d_out"], L["mask_size"], L["mask_id"])
        ref = np.stack([om.masked_gradient(A[i], B[i], rows, cols, int(lens[i])) for i in range(n)])
        off = s.offsets[li]
        e = rel_fro(got[:, off:off + L["k_out"]], ref)
        assert e <= 1e-5, (li, e)


SLICED = [dict(name="tall", d_in=512, d_out=2048, k_in=1, k_out=40000, mask_size=20000, mask_id=1, mask_count=2,
               a_group="sa"),
          dict(name="wide", d_in=3000, d_out=512, k_in=1, k_out=33000, mask_size=33000, mask_id=0, a_group="sb"),
          # bf16: the 4200-wide side's slice (8400 bytes) exceeds a fixed slot, so
          # its whole groups take the sliced direct-load gather instead
          dict(name="broad", d_in=4200, d_out=9000, k_in=1, k_out=40000, mask_size=20000, mask_id=0, mask_count=2,
               a_group="sc")]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_mask_groups_stage_row_slices(dtype):
    # App. A.2 random masks with several entry groups per layer: the table
    # deals entries to the groups along the wider side of DW (rows of the
    # tall layer, columns of the wide one), each group stages only its slice
    # of every token row; two whole groups and a partial one per layer,
    # ragged lengths
    from oracle import mask as om
    wl = dict(W.WORKLOADS["tiny"], dist_a="normal", dist_b="normal", seed=35)
    n, T = 2, 96
    inputs = _session_inputs(wl, SLICED, n, T, dtype)
    lengths = torch.tensor([96, 50], dtype=torch.int32, device=DEV)
    s = ProjectionSession(SLICED, dtype=dtype, seed=45)
    for li, (A, B) in enumerate(inputs):
        s.capture(li, A, B, lengths)
    phi = s.project(n)
    torch.cuda.synchronize()
    got, lens = host64(phi), lengths.cpu().numpy()
    group = 16384
    for li, L in enumerate(SLICED):
        m = L["k_out"]
        table = s.maps[li][0].view(torch.int32).cpu().numpy()
        t_rows, t_cols, t_pos = table[:m], table[m:2 * m], table[2 * m:3 * m]
        parts = [om.mask_indices(45, li, L["d_in"], L["d_out"], L["mask_size"], L["mask_id"] + j)
                 for j in range(L.get("mask_count", 1))]
        rows = np.concatenate([p[0] for p in parts])
        cols = np.concatenate([p[1] for p in parts])
        # the table is a permutation of the mask with each slot's position
        assert np.array_equal(np.sort(t_pos), np.arange(m))
        assert np.array_equal(t_rows, rows[t_pos]) and np.array_equal(t_cols, cols[t_pos])
        # groups follow each other along the wider side
        key = t_rows if L["d_out"] >= L["d_in"] else t_cols
        for g in range(0, m - group, group):
            assert key[g:g + group].max() <= key[g + group:g + 2 * group].min(), (li, g)
        A, B = host64(inputs[li][0]), host64(inputs[li][1])
        ref = np.stack([om.masked_gradient(A[i], B[i], rows, cols, int(lens[i])) for i in range(n)])
        off = s.offsets[li]
        e = rel_fro(got[:, off:off + m], ref)
        assert e <= 1e-5, (li, e)


def test_mask_full_size_sampled():
    # App. A.2 / App. B: ten masks of 8192 entries on Llama-3-8B-shaped layers
    # (q, k, gate, down of one block) at T = 2048, one ragged example, in the
    # launch configuration the benchmark times (whole groups on the
    # fixed-slot gather); 4096 sampled entries per layer against the oracle
    from oracle import mask as om
    wl = W.WORKLOADS["llama8b"]
    pick = [0, 1, 4, 6]  # q_proj, k_proj, gate_proj, down_proj of block 0
    layers = [dict(wl["layers"][i], k_in=1, k_out=81920, mask_size=8192, mask_count=10) for i in pick]
    n, T = 2, wl["T"]
    cache = {}
    inputs = [W.factor_blocks(dict(wl, layers=layers), li, 0, n, T, DEV, "bf16", a_cache=cache)
              for li in range(len(layers))]
    lengths = torch.tensor([T, 1531], dtype=torch.int32, device=DEV)
    s = ProjectionSession(layers, dtype="bf16", seed=wl["seed"])
    for li, (A, B) in enumerate(inputs):
        s.capture(li, A, B, lengths)
    phi = s.project(n)
    torch.cuda.synchronize()
    got, lens = host64(phi), lengths.cpu().numpy()
    rng = np.random.default_rng(5)
    for li, L in enumerate(layers):
        rows, cols = dt.dattri_get_mask(s.ctx, li)
        idx = np.sort(rng.choice(L["k_out"], 4096, replace=False))
        A, B = host64(inputs[li][0]), host64(inputs[li][1])
        ref = np.stack([om.masked_gradient(A[i], B[i], rows[idx], cols[idx], int(lens[i])) for i in range(n)])
        off = s.offsets[li]
        e = rel_fro(got[:, off + idx], ref)
        assert e <= 1e-5, (L["name"], e)


@pytest.mark.parametrize("form", ["fused", "split"])
def test_shared_input_group_matches_separate_inputs(form):
    # 16-wide maps: q and k share one fused work item (2 input tiles keep 4 row
    # tiles per wave); v would need 3 and runs alone, as does o
    layers = [dict(name="q", d_in=256, d_out=256, k_in=16, k_out=16, a_group="x"),
              dict(name="k", d_in=256, d_out=64, k_in=16, k_out=16, a_group="x"),
              dict(name="v", d_in=256, d_out=64, k_in=16, k_out=16, a_group="x"),
              dict(name="o", d_in=256, d_out=256, k_in=32, k_out=32, a_group="y")]
    wl = dict(W.WORKLOADS["llama8b"], seed=21)
    inputs = _session_inputs(wl, layers, 3, 96, "bf16")
    assert inputs[0][0] is inputs[1][0] is inputs[2][0]  # q/k/v share one A tensor
    _, phi = _run(layers, inputs, "bf16", 5, "factored", form=form)
    _check(layers, inputs, phi, 5, "bf16", [0, 1, 2], tol=1e-5)
    # the same values through separate A tensors (no sharing) agree within fp32 rounding
    sep = [(A.clone(), B) for A, B in inputs]
    _, phi2 = _run(layers, sep, "bf16", 5, "factored", form=form)
    assert rel_fro(host64(phi2), host64(phi)) < 1e-6


@pytest.mark.parametrize("form", ["fused", "split"])
def test_identity_maps_reproduce_eq4(form):
    # k = d and P = I: <phi_i, phi_j> is the factorized inner product of Eq. (4)
    d_in, d_out, T, n = 32, 16, 24, 4
    layers = [dict(name="id", d_in=d_in, d_out=d_out, k_in=d_in, k_out=d_out, a_group="a")]
    wl = dict(W.WORKLOADS["tiny"], seed=31)
    inputs = _session_inputs(wl, layers, n, T, "f32")
    eye_in = np.eye(d_in, dtype=np.float32)
    eye_out = np.eye(d_out, dtype=np.float32)
    _, phi = _run(layers, inputs, "f32", 0, "factored", overrides={0: (eye_in, eye_out)}, form=form)
    A, B = host64(inputs[0][0]), host64(inputs[0][1])
    gram = host64(phi) @ host64(phi).T
    ref = np.array([[og.ghost_dot(A[i], B[i], A[j], B[j]) for j in range(n)] for i in range(n)])
    assert rel_fro(gram, ref) < 1e-5


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_materialize_gradient_matches_eq1(dtype):
    layers = [dict(name="g", d_in=100, d_out=72, k_in=8, k_out=8, a_group="a")]
    wl = dict(W.WORKLOADS["tiny"], seed=41)
    n, T = 3, 45
    inputs = _session_inputs(wl, layers, n, T, dtype)
    lengths = torch.tensor([45, 17, 0], dtype=torch.int32, device=DEV)
    s = ProjectionSession(layers, dtype=dtype, seed=0)
    s.capture(0, inputs[0][0], inputs[0][1], lengths)
    G = torch.empty((2, 72, 100), dtype=torch.float32, device=DEV)
    dt.dattri_materialize_gradient(s.ctx, 0, 1, 2, G)
    torch.cuda.synchronize()
    A, B = host64(inputs[0][0]), host64(inputs[0][1])
    ref1 = og.weight_gradient(A[1], B[1], 17)
    assert rel_fro(host64(G[0]), ref1) < 1e-5
    assert torch.count_nonzero(G[1]).item() == 0  # length 0


# One AUTO plan that mixes routes (Eq. 2 / App. A.4 "Routing": the two forms
# are equal, so a call may route each layer its own way): two wide layers at a
# short sequence, where G costs 134 and 18 MB per example and the cost model
# sends them to the factored kernels, a layer with k_out = 128 and one with
# k_in = 160, which exceed the factored kernels' map widths and route
# materialized; k_in = 160 takes two passes of the G projection (8 input tiles
# per pass).  f0 and w_out share their input block, so the factored group and
# the materialized layer read the same A.  bf16 rows of 2048 and 300 elements
# take the transposing and the plain G kernel; rows of 3000 are unaligned.
MIXED = [dict(name="f0", d_in=2048, d_out=16384, k_in=32, k_out=32, a_group="a"),
         dict(name="w_out", d_in=2048, d_out=96, k_in=16, k_out=128, a_group="a"),
         dict(name="w_in", d_in=300, d_out=72, k_in=160, k_out=24, a_group="b"),
         dict(name="f1", d_in=3000, d_out=1500, k_in=8, k_out=16, a_group="c")]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_auto_mixed_routes_wide_maps(dtype):
    print(f"[project] mixed AUTO plan dtype={dtype}", flush=True)
    wl = dict(W.WORKLOADS["tiny"], dist_a="normal", dist_b="normal", seed=61)
    n, T = 5, 70
    inputs = _session_inputs(wl, MIXED, n, T, dtype)
    assert inputs[0][0] is inputs[1][0]
    lengths = torch.tensor([70, 0, 1, 33, 64], dtype=torch.int32, device=DEV)
    s, phi = _run(MIXED, inputs, dtype, 63, "auto", lengths=lengths)
    routes = [r[0] for r in s.routes()]
    assert routes[1] == dt.DATTRI_ROUTE_MATERIALIZED and routes[2] == dt.DATTRI_ROUTE_MATERIALIZED
    assert routes[0] == dt.DATTRI_ROUTE_FACTORED and routes[3] == dt.DATTRI_ROUTE_FACTORED
    assert torch.count_nonzero(phi[1]).item() == 0  # length 0
    # offsets are the running sums of k_in * k_out in registration order
    assert s.offsets == [0, 1024, 1024 + 2048, 1024 + 2048 + 3840]
    errs = _check(MIXED, inputs, phi, 63, dtype, [0, 2, 3, 4], lengths=lengths, tol=1e-5)
    print(f"[project] mixed AUTO per-layer rel err {errs}", flush=True)
    # forced materialized on every layer gives the same blocks
    _, phi_m = _run(MIXED, inputs, dtype, 63, "materialized", lengths=lengths)
    assert rel_fro(host64(phi_m), host64(phi)) < 1e-5


def test_factored_route_refuses_wide_maps():
    layers = [MIXED[1]]
    s = ProjectionSession(layers, dtype="f32", seed=0)
    A = torch.zeros((2, 4, 200), device=DEV)
    B = torch.zeros((2, 4, 96), device=DEV)
    s.capture(0, A, B)
    with pytest.raises(dt.DattriError) as e:
        s.project(2, route=dt.DATTRI_ROUTE_FACTORED)
    assert e.value.status_name == "E_UNSUPPORTED"


def test_gpt2_batch_bf16():
    wl = W.WORKLOADS["gpt2"]
    inputs = _session_inputs(wl, wl["layers"], wl["batch"], wl["T"], "bf16")
    s, phi = _run(wl["layers"], inputs, "bf16", wl["seed"], "auto")
    assert all(r[0] == dt.DATTRI_ROUTE_FACTORED for r in s.routes())
    errs = _check(wl["layers"], inputs, phi, wl["seed"], "bf16", [0, 13, 31])
    print(f"gpt2: max per-layer rel err {max(errs):.3e}")
    assert torch.isfinite(phi).all()


def test_llama8b_full_size_sampled():
    """Full Llama-3-8B-shaped batch (224 layers, T=2048, n=8) in the launch
    configuration the benchmark times; every layer block of examples 0 and 7
    against the oracle (factor blocks streamed to the host layer by layer)."""
    wl = W.WORKLOADS["llama8b"]
    layers, n, T = wl["layers"], wl["batch"], wl["T"]
    cache = {}
    s = ProjectionSession(layers, dtype="bf16", seed=wl["seed"])
    inputs = []
    for li in range(len(layers)):
        A, B = W.factor_blocks(wl, li, 0, n, T, DEV, "bf16", a_cache=cache)
        s.capture(li, A, B)
        inputs.append((A, B))
    phi = s.project(n)
    torch.cuda.synchronize()
    assert all(r[0] == dt.DATTRI_ROUTE_FACTORED for r in s.routes())
    assert torch.isfinite(phi).all()
    examples = (0, 7)
    got = host64(phi[list(examples)])
    print("[project] llama8b full size: oracle over 224 layers x 2 examples", flush=True)
    a_host = {}
    worst = 0.0
    for li, L in enumerate(layers):
        A, B = inputs[li]
        P_in, P_out = orng.projection_pair(wl["seed"], li, L["d_in"], L["d_out"], L["k_in"], L["k_out"], "bf16")
        if A.data_ptr() not in a_host:  # q/k/v and gate/up share one input block
            a_host = {A.data_ptr(): [A[i].cpu().to(torch.float64).numpy() for i in examples]}
        off, w = s.offsets[li], L["k_in"] * L["k_out"]
        for j, i in enumerate(examples):
            Bh = B[i].cpu().to(torch.float64).numpy()
            ref = og.project_factored(a_host[A.data_ptr()][j], Bh, P_in, P_out).reshape(-1)
            err = rel_fro(got[j, off:off + w], ref)
            worst = max(worst, err)
            assert err <= 1e-5, (li, i, err)
    print(f"[project] llama8b full size: worst block rel err {worst:.3e}", flush=True)


@pytest.mark.parametrize("form", ["fused", "split"])
@pytest.mark.parametrize("name", ["routing", "lora_b", "narrow"])
def test_switch_workloads_both_routes(name, form):
    wl = W.WORKLOADS[name]
    n = wl["batch"]
    inputs = _session_inputs(wl, wl["layers"], n, wl["T"], "bf16")
    _, phi_f = _run(wl["layers"], inputs, "bf16", wl["seed"], "factored", form=form)
    _, phi_m = _run(wl["layers"], inputs, "bf16", wl["seed"], "materialized")
    ex = [0, n // 2, n - 1]
    _check(wl["layers"], inputs, phi_f, wl["seed"], "bf16", ex, tol=1e-5)
    _check(wl["layers"], inputs, phi_m, wl["seed"], "bf16", ex, tol=1e-5)
    # the two exact routes agree on every example (Eq. (2))
    assert rel_fro(host64(phi_m), host64(phi_f)) < 1e-5


@pytest.mark.parametrize("name,expect", [("routing", "factored"), ("lora_b", "materialized"),
                                         ("narrow", "materialized")])
def test_switch_workloads_auto_route(name, expect):
    # the default (MI355X-fitted) cost model: the wide short-sequence layer
    # stays factored, the adapter's B matrix (8 -> 4096, T = 32) and the
    # narrow 128 -> 128 layer at T = 2048 switch to the one-pass materialized
    # kernel, as the forced-route timings do; the blocks AUTO produces match
    # the oracle on sampled examples
    wl = W.WORKLOADS[name]
    n = wl["batch"]
    inputs = _session_inputs(wl, wl["layers"], n, wl["T"], "bf16")
    s, phi = _run(wl["layers"], inputs, "bf16", wl["seed"], "auto")
    want = dt.DATTRI_ROUTE_FACTORED if expect == "factored" else dt.DATTRI_ROUTE_MATERIALIZED
    route, pf, pm = s.routes()[0]
    print(f"[project] {name}: AUTO -> {expect}? predicted factored {pf:.1f} us, materialized {pm:.1f} us", flush=True)
    assert route == want
    _check(wl["layers"], inputs, phi, wl["seed"], "bf16", [0, n // 2, n - 1], tol=1e-5)


@pytest.mark.parametrize("plan_buffer", [True, False])
def test_plan_reuse_follows_captures(plan_buffer):
    # launch plans are cached by the context state and kept in the bound plan
    # buffer: new contents in the same captured buffers reuse the plan, a
    # capture of other buffers (or another route) re-plans; every call matches
    # the oracle for the data it saw
    layers = [dict(name="p0", d_in=96, d_out=80, k_in=16, k_out=32, a_group="a"),
              dict(name="p1", d_in=96, d_out=40, k_in=8, k_out=8, a_group="a")]
    wl = dict(W.WORKLOADS["tiny"], dist_a="normal", dist_b="normal", seed=91)
    n, T = 3, 50
    s = ProjectionSession(layers, dtype="f32", seed=93, plan_buffer=plan_buffer)
    first = _session_inputs(wl, layers, n, T, "f32")
    bufs = [(A.clone(), B.clone()) for A, B in first]
    for li, (A, B) in enumerate(bufs):
        s.capture(li, A, B)
    for step, seed in enumerate((91, 92)):
        data = _session_inputs(dict(wl, seed=seed), layers, n, T, "f32")
        for (A, B), (A2, B2) in zip(bufs, data):  # same buffers, new contents
            A.copy_(A2)
            B.copy_(B2)
        for route in ("factored", "materialized"):
            phi = s.project(n, route=ROUTES[route])
            torch.cuda.synchronize()
            _check(layers, data, phi, 93, "f32", [0, 1, 2], tol=1e-5)
    # other buffers: the next call must plan for them
    other = _session_inputs(dict(wl, seed=95), layers, n, T, "f32")
    s.clear()
    for li, (A, B) in enumerate(other):
        s.capture(li, A, B)
    phi = s.project(n)
    torch.cuda.synchronize()
    _check(layers, other, phi, 93, "f32", [0, 1, 2], tol=1e-5)


def test_bf16_phi_output_and_ld():
    wl = W.WORKLOADS["tiny"]
    layers = wl["layers"] * 2
    inputs = _session_inputs(dict(wl, seed=51), layers, 6, 16, "f32")
    s = ProjectionSession(layers, dtype="f32", seed=3)
    for li, (A, B) in enumerate(inputs):
        s.capture(li, A, B)
    big = torch.full((6, s.F + 40), 7.0, dtype=torch.bfloat16, device=DEV)
    s.project(6, phi_dtype="bf16", phi=big)
    torch.cuda.synchronize()
    assert torch.all(big[:, s.F:] == 7.0)  # columns beyond F untouched
    _check(layers, inputs, big[:, :s.F], 3, "f32", list(range(6)), tol=2 ** -8)


@pytest.mark.parametrize("form", ["fused", "split"])
def test_empty_batch_and_zero_tokens(form):
    layers = [dict(name="e", d_in=64, d_out=32, k_in=16, k_out=16, a_group="a")]
    s = ProjectionSession(layers, dtype="bf16", seed=0, form=FORMS[form])
    A = torch.empty((0, 16, 64), dtype=torch.bfloat16, device=DEV)
    B = torch.empty((0, 16, 32), dtype=torch.bfloat16, device=DEV)
    s.capture(0, A, B)
    phi = s.project(0)
    assert phi.shape == (0, 256)
    A = torch.empty((3, 0, 64), dtype=torch.bfloat16, device=DEV)
    B = torch.empty((3, 0, 32), dtype=torch.bfloat16, device=DEV)
    for route in ("factored", "materialized"):
        s.clear()
        s.capture(0, A, B)
        phi = torch.full((3, 256), 5.0, device=DEV)
        s.project(3, route=ROUTES[route], phi=phi)
        torch.cuda.synchronize()
        assert torch.count_nonzero(phi).item() == 0


@pytest.mark.parametrize("form", ["fused", "split"])
def test_deterministic_bitwise(form):
    wl = W.WORKLOADS["gpt2"]
    layers = wl["layers"][:8]
    inputs = _session_inputs(wl, layers, 8, 256, "bf16")
    _, a = _run(layers, inputs, "bf16", 1, "factored", form=form)
    _, b = _run(layers, inputs, "bf16", 1, "factored", form=form)
    assert torch.equal(a, b)
    _, c = _run(layers[:2], [inputs[0], inputs[1]], "bf16", 1, "materialized")
    _, d = _run(layers[:2], [inputs[0], inputs[1]], "bf16", 1, "materialized")
    assert torch.equal(c, d)
