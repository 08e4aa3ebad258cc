"""Host-side tests of libdattri (no GPU): the library loads, exports every entry
point declared in include/dattri.h, rejects bad calls with the documented
status before any GPU work, and its host generator and operation counters
agree with the oracle."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2609_38767_amd as dt
from golden_io import load as load_golden
from oracle import cost as ocost
from oracle import rng as orng

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "dattri.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dattri_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = dt.load()
    declared = _declared()
    assert len(declared) >= 20
    for name in declared:
        assert hasattr(lib, name), name
    assert set(declared) == set(dt.EXPORTED)


def test_nm_shows_c_symbols():
    # exported with C linkage (unmangled)
    out = os.popen(f"nm -D --defined-only {dt.lib_path}").read()
    for name in _declared():
        assert re.search(rf"\bT {name}\b", out), name


@pytest.fixture
def ctx():
    c = dt.dattri_create(dt.DATTRI_F32, 0)
    yield c
    dt.dattri_destroy(c)


def _status(excinfo):
    return excinfo.value.status_name


def test_create_and_register_errors(ctx):
    lib = dt.load()
    assert lib.dattri_create(None, 0, 0) == -1
    out = ctypes.c_void_p()
    assert lib.dattri_create(ctypes.byref(out), 7, 0) == -3
    assert "neither" in dt.dattri_last_error()
    for bad in [(0, 4, 2, 2), (4, 0, 2, 2), (4, 4, 0, 2), (4, 4, 2, -1), (1 << 21, 4, 2, 2)]:
        with pytest.raises(dt.DattriError) as e:
            dt.dattri_register_layer(ctx, *bad)
        assert _status(e) == "E_INVALID_ARG"
    assert dt.dattri_num_layers(ctx) == 0
    dt.dattri_destroy(None)  # NULL-safe


def test_layer_offsets_and_feature_dim(ctx):
    ids = [dt.dattri_register_layer(ctx, d, e, ki, ko) for d, e, ki, ko in
           [(64, 64, 8, 8), (768, 2304, 16, 16), (8, 4096, 8, 64)]]
    assert ids == [0, 1, 2]
    assert dt.dattri_feature_dim(ctx) == 64 + 256 + 512
    assert [dt.dattri_layer_offset(ctx, i) for i in ids] == [0, 64, 320]
    assert dt.dattri_layer_dims(ctx, 2) == (8, 4096, 8, 64)
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_layer_offset(ctx, 3)
    assert _status(e) == "E_INVALID_ARG"


def test_state_and_workspace_errors(ctx):
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_workspace_bytes(ctx)
    assert _status(e) == "E_STATE"  # nothing registered
    dt.dattri_register_layer(ctx, 64, 64, 8, 8)
    dt.dattri_register_layer(ctx, 64, 32, 8, 8)
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_workspace_bytes(ctx)
    assert _status(e) == "E_STATE"  # not captured
    fake = 1 << 40  # never dereferenced: no GPU work is enqueued on these paths
    dt.dattri_capture_layer(ctx, 0, fake, fake, 4, 16)
    dt.dattri_capture_layer(ctx, 1, fake, fake, 5, 16)
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_workspace_bytes(ctx)
    assert _status(e) == "E_STATE" and "n=5" in str(e.value)
    dt.dattri_capture_layer(ctx, 1, fake, fake, 4, 16)
    assert dt.dattri_workspace_bytes(ctx) > 0
    # project before binding maps
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_project_per_example(ctx, fake, dt.DATTRI_F32, 128, fake, 1 << 20)
    assert _status(e) == "E_STATE" and "not bound" in str(e.value)
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_capture_layer(ctx, 0, None, None, 4, 16)
    assert _status(e) == "E_INVALID_ARG"
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_capture_layer(ctx, 0, fake, fake, -1, 16)
    assert _status(e) == "E_INVALID_ARG"
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_capture_layer(ctx, 0, fake, fake, 1, 1 << 26)  # 2^26 x 64 x 4 bytes > 4 GiB
    assert _status(e) == "E_SHAPE"
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_bind_projection(ctx, 0, None, fake)
    assert _status(e) == "E_INVALID_ARG"
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_bind_projection(ctx, 0, fake + 4, fake)
    assert _status(e) == "E_INVALID_ARG" and "aligned" in str(e.value)
    dt.dattri_clear_captures(ctx)
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_layer_route(ctx, 0)
    assert _status(e) == "E_STATE"


def test_factored_limits_and_auto_route(ctx):
    fake = 1 << 40
    dt.dattri_register_layer(ctx, 256, 256, 16, 128)  # k_out beyond the factored kernel
    dt.dattri_capture_layer(ctx, 0, fake, fake, 2, 64)
    route, f_us, m_us = dt.dattri_layer_route(ctx, 0)
    assert route == dt.DATTRI_ROUTE_MATERIALIZED and f_us == float("inf")
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_workspace_bytes(ctx, dt.DATTRI_ROUTE_FACTORED)
    assert _status(e) == "E_UNSUPPORTED"
    assert dt.dattri_workspace_bytes(ctx, dt.DATTRI_ROUTE_MATERIALIZED) > 0


def test_score_argument_errors():
    fake = 1 << 40
    f32 = dt.DATTRI_F32

    def call(n_q=4, ld_q=0, n_t=8, ld_t=0, F=64, dtype=f32, d=None, S=fake, k=0, idx=None, val=None,
             ws=None, wsb=0):
        dt.dattri_score(fake, n_q, ld_q, fake, n_t, ld_t, F, dtype, d, S, k, idx, val, ws, wsb)

    cases = [
        (dict(dtype=5), "E_DTYPE"),
        (dict(k=9, idx=fake, val=fake), "E_INVALID_ARG"),        # topk > n_train
        (dict(n_t=2000, k=1025, idx=fake, val=fake), "E_UNSUPPORTED"),  # topk > 1024
        (dict(S=None), "E_INVALID_ARG"),                         # nothing requested
        (dict(d=fake), "E_WORKSPACE"),         # preconditioner needs a scaled-query workspace
        (dict(F=63), "E_UNSUPPORTED"),                           # rows not 16-byte multiples
        (dict(ld_q=32), "E_INVALID_ARG"),                        # stride below F
        (dict(ld_t=63), "E_INVALID_ARG"),
        (dict(ld_t=66), "E_UNSUPPORTED"),                        # stride not a 16-byte multiple
        (dict(ld_q=-1), "E_INVALID_ARG"),
        (dict(ld_t=1 << 22), "E_UNSUPPORTED"),                   # 256 rows reach 4 GiB
    ]
    for kw, want in cases:
        with pytest.raises(dt.DattriError) as e:
            call(**kw)
        assert _status(e) == want, kw
    need = dt.dattri_score_workspace_bytes(4, 8, 64, dt.DATTRI_BF16, True, False, 3)
    assert need >= 4 * 64 * 2 + 4 * 8 * 4
    assert dt.dattri_score_workspace_bytes(4, 8, 64, dt.DATTRI_BF16, False, True, 3) == 256
    # the scaled query copy is stored at the recommended stride
    ld = dt.dattri_feature_ld(8192, dt.DATTRI_BF16)
    assert dt.dattri_score_workspace_bytes(2048, 8, 8192, dt.DATTRI_BF16, True, True, 0) >= 2048 * ld * 2


@pytest.mark.parametrize("F,dtype,ld", [
    (64, dt.DATTRI_F32, 64),          # 256-byte rows: unchanged
    (100, dt.DATTRI_BF16, 128),       # rounded up to 256 bytes
    (4096, dt.DATTRI_BF16, 4096),     # 8 KiB rows: below 16 KiB, unchanged
    (8192, dt.DATTRI_BF16, 8448),     # 16 KiB rows: + 512 bytes
    (8192, dt.DATTRI_F32, 8320),      # 32 KiB rows: + 512 bytes
    (12288, dt.DATTRI_BF16, 12544),   # 24 KiB (a multiple of 8 KiB): + 512 bytes
    (14336, dt.DATTRI_BF16, 14336),   # 28 KiB: not a multiple of 8 KiB
    (0, dt.DATTRI_BF16, 0),
])
def test_feature_ld_rule(F, dtype, ld):
    assert dt.dattri_feature_ld(F, dtype) == ld


def test_feature_ld_errors():
    for args, want in [((-1, dt.DATTRI_F32), "E_INVALID_ARG"), ((8, 7), "E_DTYPE")]:
        with pytest.raises(dt.DattriError) as e:
            dt.dattri_feature_ld(*args)
        assert _status(e) == want


@pytest.mark.parametrize("dtype_name,dtype", [("f32", dt.DATTRI_F32), ("bf16", dt.DATTRI_BF16)])
def test_host_generator_matches_oracle(dtype_name, dtype):
    c = dt.dattri_create(dtype, 12345)
    shapes = [(64, 48, 8, 4), (100, 37, 16, 32), (4096, 1024, 32, 32)]
    for s in shapes:
        dt.dattri_register_layer(c, *s)
    for layer, (d_in, d_out, k_in, k_out) in enumerate(shapes):
        lib_in, lib_out = dt.dattri_get_projection(c, layer)
        ora_in, ora_out = orng.projection_pair(12345, layer, d_in, d_out, k_in, k_out, dtype_name)
        for lib_m, ora_m in ((lib_in, ora_in), (lib_out, ora_out)):
            ora32 = ora_m.astype(np.float32)
            # identical up to one float32 ulp (libm log/cos may differ in the last bit)
            diff = np.abs(lib_m.view(np.int32).astype(np.int64) - ora32.view(np.int32).astype(np.int64))
            assert diff.max() <= (1 if dtype_name == "f32" else 1)
            assert np.mean(diff == 0) > 0.999
    dt.dattri_destroy(c)


@pytest.mark.parametrize("dtype_name,dtype", [("f32", dt.DATTRI_F32), ("bf16", dt.DATTRI_BF16)])
def test_rademacher_maps_match_oracle(dtype_name, dtype):
    c = dt.dattri_create(dtype, 777)
    shapes = [(64, 48, 8, 4), (300, 37, 64, 24)]
    for s in shapes:
        dt.dattri_register_layer(c, *s)
    dt.dattri_set_map_kind(c, 1, dt.DATTRI_MAP_RADEMACHER)
    assert dt.dattri_get_map_kind(c, 0) == dt.DATTRI_MAP_GAUSSIAN
    assert dt.dattri_get_map_kind(c, 1) == dt.DATTRI_MAP_RADEMACHER
    d_in, d_out, k_in, k_out = shapes[1]
    lib_in, lib_out = dt.dattri_get_projection(c, 1)
    ora_in, ora_out = orng.projection_pair(777, 1, d_in, d_out, k_in, k_out, dtype_name, kind="rademacher")
    np.testing.assert_array_equal(lib_in, ora_in.astype(np.float32))  # exact: no libm in the signs
    np.testing.assert_array_equal(lib_out, ora_out.astype(np.float32))
    for bad in (2, -1):
        with pytest.raises(dt.DattriError) as e:
            dt.dattri_set_map_kind(c, 0, bad)
        assert _status(e) == "E_INVALID_ARG"
    with pytest.raises(dt.DattriError):
        dt.dattri_set_map_kind(c, 5, dt.DATTRI_MAP_RADEMACHER)
    dt.dattri_destroy(c)


def test_override_maps_are_rounded_and_returned():
    c = dt.dattri_create(dt.DATTRI_BF16, 0)
    dt.dattri_register_layer(c, 8, 4, 8, 4)
    p_in, _ = dt.dattri_get_projection(c, 0)
    assert p_in.shape == (8, 8)
    dt.dattri_destroy(c)


@pytest.mark.parametrize("case", load_golden("route_counts.json")["cases"], ids=lambda c: c["name"])
def test_layer_cost_counters(case):
    c = dt.dattri_create(dt.DATTRI_BF16, 0)
    dt.dattri_register_layer(c, case["d_in"], case["d_out"], case["k_in"], case["k_out"])
    f, m, fb, mb = dt.dattri_layer_costs(c, 0, case["T"])
    assert f == case["factored"] == ocost.factored_flops(case["d_in"], case["d_out"], case["k_in"], case["k_out"], case["T"])
    # the library runs the (G P_in)-first association of the materialized form
    di, do, ki, ko, T = case["d_in"], case["d_out"], case["k_in"], case["k_out"], case["T"]
    assert m == 2 * T * di * do + 2 * do * di * ki + 2 * do * ki * ko
    assert m >= ocost.materialized_flops(di, do, ki, ko, T)
    assert fb == ocost.factor_bytes(di, do, T, 2)
    assert mb == fb + 2 * 4 * do * di
    dt.dattri_destroy(c)


FIELDS = ("factored_tflops", "factored_gbs", "gradient_tflops", "gradient_gbs",
          "gproject_tflops", "gproject_gbs", "launch_us", "call_us", "round_us")


def test_cost_model_roundtrip_and_validation(ctx):
    m = dt.dattri_get_cost_model(ctx)
    assert set(m) == set(FIELDS)
    m2 = dict(m, factored_gbs=1234.5, call_us=7.25)
    dt.dattri_set_cost_model(ctx, m2)
    assert dt.dattri_get_cost_model(ctx) == m2
    # rates must be positive, finite and within the published MI355X peaks
    bad = [dict(m, gradient_tflops=0.0), dict(m, factored_gbs=8000.5), dict(m, gradient_gbs=float("inf")),
           dict(m, factored_tflops=2501.0), dict(m, gproject_tflops=157.4), dict(m, launch_us=-1.0),
           dict(m, call_us=float("nan")), dict(m, round_us=-0.5)]
    for b in bad:
        with pytest.raises(dt.DattriError) as e:
            dt.dattri_set_cost_model(ctx, b)
        assert _status(e) == "E_INVALID_ARG"
    assert dt.dattri_get_cost_model(ctx) == m2  # unchanged by the rejected calls


def _write(tmp_path, name, text):
    p = tmp_path / name
    p.write_text(text)
    return str(p)


def test_cost_calibration_file_roundtrip(ctx, tmp_path):
    import json
    model = {"factored_tflops": 310.5, "factored_gbs": 5123.25, "gradient_tflops": 700.0, "gradient_gbs": 4999.0,
             "gproject_tflops": 61.0, "gproject_gbs": 4000.0, "launch_us": 4.5, "call_us": 1.25e1,
             "round_us": 3.0}
    # the layout the calibration script writes: the model beside per-shape records
    doc = {"model": model, "rms_log_error": 0.1, "device": "AMD Instinct MI355X",
           "shapes": [{"d_in": 8, "auto": "factored", "regret": 0.0, "nested": [1, -2.5e-3, True, None, {}]}],
           "note": "escapes \" \\ \u00e9 \n"}
    path = _write(tmp_path, "calib.json", json.dumps(doc, indent=2))
    dt.dattri_set_cost_calibration(ctx, path)
    got = dt.dattri_get_cost_model(ctx)
    assert got == model
    # a layer's predicted times follow the loaded model
    fake = 1 << 40
    dt.dattri_register_layer(ctx, 128, 128, 64, 64)
    dt.dattri_capture_layer(ctx, 0, fake, fake, 8, 2048)
    before = dt.dattri_layer_route(ctx, 0)
    dt.dattri_set_cost_calibration(ctx, _write(tmp_path, "c2.json", json.dumps({"model": dict(model, call_us=112.5)})))
    after = dt.dattri_layer_route(ctx, 0)
    assert after[1] == pytest.approx(before[1] + 100.0) and after[2] == pytest.approx(before[2] + 100.0)


@pytest.mark.parametrize("text,what", [
    (None, "cannot open"),
    ('{"model": {"factored_tflops": 1', "expected ',' or '}'"),
    ('{"model": {"factored_tflops": ', "unexpected end"),
    ('[1, 2]', "not a JSON object"),
    ('{"models": {}}', "no \"model\""),
    ('{"model": {"factored_tflops": 300}}', "factored_gbs missing"),
    ('{"model": {"factored_tflops": "300", "factored_gbs": 1, "gradient_tflops": 1, "gradient_gbs": 1, '
     '"gproject_tflops": 1, "gproject_gbs": 1, "launch_us": 1, "call_us": 1, "round_us": 1}}',
     "factored_tflops missing"),
    ('{"model": {"factored_tflops": 300, "factored_gbs": 9000, "gradient_tflops": 1, "gradient_gbs": 1, '
     '"gproject_tflops": 1, "gproject_gbs": 1, "launch_us": 1, "call_us": 1, "round_us": 1}}', "factored_gbs"),
    ('{"model": {"factored_tflops": 300, "factored_gbs": 1, "gradient_tflops": 1, "gradient_gbs": 1, '
     '"gproject_tflops": 1, "gproject_gbs": 1, "launch_us": 1, "call_us": 1}}', "round_us missing"),
    ('{"model": {"factored_tflops": 01}}', "expected"),
    ('{"model": {}} x', "trailing"),
])
def test_cost_calibration_file_errors(ctx, tmp_path, text, what):
    before = dt.dattri_get_cost_model(ctx)
    path = str(tmp_path / "missing.json") if text is None else _write(tmp_path, "bad.json", text)
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_set_cost_calibration(ctx, path)
    assert _status(e) == "E_INVALID_ARG"
    assert what in dt.dattri_last_error() or what in str(e.value)
    assert dt.dattri_get_cost_model(ctx) == before


def test_route_prediction_counts_launches(ctx):
    # with rates at the peaks the work terms are tiny next to a huge per-launch
    # cost, so the predictions count launches: the wide short-sequence layer
    # alone takes the split form (stage 1 for both maps of 4 tiles, slab sum,
    # contraction; one token chunk, so no reduction) = 3 launches; the
    # materialized form stages G of 2 examples at a time (2 GiB / 940 MB) =
    # 32 chunks of 3 launches
    fake = 1 << 40
    dt.dattri_register_layer(ctx, 8192, 28672, 64, 64)
    dt.dattri_capture_layer(ctx, 0, fake, fake + (1 << 36), 64, 32)
    peaks = dict(factored_tflops=2500.0, factored_gbs=8000.0, gradient_tflops=2500.0, gradient_gbs=8000.0,
                 gproject_tflops=157.3, gproject_gbs=8000.0)
    dt.dattri_set_cost_model(ctx, dict(peaks, launch_us=1e6, call_us=0.0, round_us=0.0))
    _, f_us, m_us = dt.dattri_layer_route(ctx, 0)
    assert round(f_us / 1e6) == 3
    assert round(m_us / 1e6) == 96
    # the fused form when forced: factored kernel + reduction
    dt.dattri_set_factored_form(ctx, dt.DATTRI_FORM_FUSED)
    assert round(dt.dattri_layer_route(ctx, 0)[1] / 1e6) == 2


def test_route_follows_cost_model(ctx):
    fake = 1 << 40
    dt.dattri_register_layer(ctx, 128, 128, 64, 64)
    dt.dattri_capture_layer(ctx, 0, fake, fake, 8, 2048)
    m = dt.dattri_get_cost_model(ctx)
    # a factored kernel made artificially slow must lose, a fast one must win
    dt.dattri_set_cost_model(ctx, dict(m, factored_tflops=1e-3, factored_gbs=1e-3))
    assert dt.dattri_layer_route(ctx, 0)[0] == dt.DATTRI_ROUTE_MATERIALIZED
    dt.dattri_set_cost_model(ctx, dict(m, gradient_tflops=1e-3))
    assert dt.dattri_layer_route(ctx, 0)[0] == dt.DATTRI_ROUTE_FACTORED


def test_call_routes_share_factored_launches():
    # App. A.4 "Routing" per layer, with the launches of a call shared: a
    # narrow layer that is faster materialized when projected alone joins the
    # factored route in a call that factors another layer anyway, as long as
    # its factored work without launches is no slower; its own predictions do
    # not change
    fake = 1 << 40
    alone = dt.dattri_create(dt.DATTRI_BF16, 0)
    pair = dt.dattri_create(dt.DATTRI_BF16, 0)
    try:
        dt.dattri_register_layer(alone, 128, 128, 64, 64)
        dt.dattri_capture_layer(alone, 0, fake, fake + (1 << 36), 8, 2048)
        for d_in, d_out in ((128, 128), (4096, 14336)):
            dt.dattri_register_layer(pair, d_in, d_out, 32 if d_in > 128 else 64, 32 if d_in > 128 else 64)
        dt.dattri_capture_layer(pair, 0, fake, fake + (1 << 36), 8, 2048)
        dt.dattri_capture_layer(pair, 1, fake + (2 << 36), fake + (3 << 36), 8, 2048)
        r0, pf0, pm0 = dt.dattri_layer_route(alone, 0)
        assert r0 == dt.DATTRI_ROUTE_MATERIALIZED and pf0 > pm0
        r1, pf1, pm1 = dt.dattri_layer_route(pair, 1)
        assert r1 == dt.DATTRI_ROUTE_FACTORED and pf1 < pm1
        r, pf, pm = dt.dattri_layer_route(pair, 0)
        assert (pf, pm) == (pf0, pm0)
        assert r == dt.DATTRI_ROUTE_FACTORED
        # with the factored route made slow, the narrow layer stays materialized
        m = dt.dattri_get_cost_model(pair)
        dt.dattri_set_cost_model(pair, dict(m, factored_gbs=m["factored_gbs"] / 100))
        assert dt.dattri_layer_route(pair, 0)[0] == dt.DATTRI_ROUTE_MATERIALIZED
    finally:
        dt.dattri_destroy(alone)
        dt.dattri_destroy(pair)


def test_factored_form_option(ctx):
    assert dt.dattri_get_factored_form(ctx) == dt.DATTRI_FORM_AUTO
    for f in (dt.DATTRI_FORM_FUSED, dt.DATTRI_FORM_SPLIT, dt.DATTRI_FORM_AUTO):
        dt.dattri_set_factored_form(ctx, f)
        assert dt.dattri_get_factored_form(ctx) == f
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_set_factored_form(ctx, 3)
    assert _status(e) == "E_INVALID_ARG"
    # a short-sequence capture: the split form stages its float32 projected
    # rows (at least n*T*(k_in + k_out) floats) in the workspace
    fake = 1 << 40
    dt.dattri_register_layer(ctx, 8192, 28672, 64, 64)
    dt.dattri_capture_layer(ctx, 0, fake, fake, 64, 32)
    dt.dattri_set_factored_form(ctx, dt.DATTRI_FORM_FUSED)
    fused = dt.dattri_workspace_bytes(ctx, dt.DATTRI_ROUTE_FACTORED)
    dt.dattri_set_factored_form(ctx, dt.DATTRI_FORM_SPLIT)
    split = dt.dattri_workspace_bytes(ctx, dt.DATTRI_ROUTE_FACTORED)
    dt.dattri_set_factored_form(ctx, dt.DATTRI_FORM_AUTO)
    auto = dt.dattri_workspace_bytes(ctx, dt.DATTRI_ROUTE_FACTORED)
    assert split >= 4 * 64 * 32 * (64 + 64)
    assert auto == split  # few fused work items and T <= 128: AUTO takes the split form


def test_probe_errors():
    FAKE = 1 << 20
    cases = [(lambda: dt.dattri_probe_read(None, 1024, FAKE, 4), "E_INVALID_ARG"),
             (lambda: dt.dattri_probe_read(FAKE + 8, 1024, FAKE, 4), "E_INVALID_ARG"),
             (lambda: dt.dattri_probe_read(FAKE, 1000, FAKE, 4), "E_INVALID_ARG"),
             (lambda: dt.dattri_probe_read(FAKE, 0, FAKE, 4), "E_INVALID_ARG"),
             (lambda: dt.dattri_probe_read(FAKE, 1024, None, 4), "E_INVALID_ARG"),
             (lambda: dt.dattri_probe_read(FAKE, 1024, FAKE, 0), "E_INVALID_ARG"),
             (lambda: dt.dattri_probe_mfma(None, 4, 10), "E_INVALID_ARG"),
             (lambda: dt.dattri_probe_mfma(FAKE, 0, 10), "E_INVALID_ARG"),
             (lambda: dt.dattri_probe_mfma(FAKE, 4, 0), "E_INVALID_ARG"),
             (lambda: dt.dattri_probe_mfma(FAKE, (1 << 20) + 1, 10), "E_INVALID_ARG")]
    for fn, want in cases:
        with pytest.raises(dt.DattriError) as e:
            fn()
        assert _status(e) == want
