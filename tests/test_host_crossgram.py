"""Host-side tests of the cross-Gram entry points (no GPU, no kernel launch):
argument and state validation, the exact operation counts against the oracle,
the time model's route choice and its settable rates."""
import pytest

import paper_2609_38767_amd as dt
from oracle import cost as ocost

FAKE = 1 << 40  # a device address that is recorded, never dereferenced here


def _ctx(dims, n, T, dtype=dt.DATTRI_BF16, capture=True):
    c = dt.dattri_create(dtype, 0)
    for d_in, d_out in dims:
        lid = dt.dattri_register_layer(c, d_in, d_out, 1, 1)
        if capture:
            dt.dattri_capture_layer(c, lid, FAKE, FAKE, n, T)
    return c


def _status(e):
    return e.value.status_name


@pytest.mark.parametrize("shape", [(1, 1, 2, 2, 3, 5), (8, 1, 512, 512, 1024, 4096), (3, 5, 7, 11, 13, 17),
                                   (64, 64, 2048, 2048, 4096, 14336), (0, 4, 16, 16, 8, 8)])
def test_costs_match_oracle(shape):
    na, nb, Ta, Tb, di, dq = shape
    f, m, fb, mb = dt.dattri_cross_gram_costs(na, nb, Ta, Tb, di, dq, 2)
    assert f == ocost.crossgram_flops_factorized(na, nb, Ta, Tb, di, dq)
    assert m == ocost.crossgram_flops_materialized(na, nb, Ta, Tb, di, dq)
    assert fb == (na * Ta + nb * Tb) * (di + dq) * 2
    assert mb == fb + 8 * (na + nb) * di * dq


def test_cost_errors():
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_cross_gram_costs(-1, 1, 1, 1, 1, 1, 2)
    assert _status(e) == "E_INVALID_ARG"
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_cross_gram_costs(1, 1, 1, 1, 1, 1, 3)
    assert _status(e) == "E_INVALID_ARG"


def test_validation_before_any_launch():
    a = _ctx([(64, 32), (16, 48)], 4, 8)
    b = _ctx([(64, 32), (16, 48)], 3, 5)
    other = _ctx([(64, 32)], 3, 5)
    wrong_dims = _ctx([(64, 32), (16, 40)], 3, 5)
    f32 = _ctx([(64, 32), (16, 48)], 3, 5, dtype=dt.DATTRI_F32)
    uncaptured = _ctx([(64, 32), (16, 48)], 3, 5, capture=False)
    try:
        for x, want in [(other, "E_SHAPE"), (wrong_dims, "E_SHAPE"), (f32, "E_SHAPE"),
                        (uncaptured, "E_STATE")]:
            with pytest.raises(dt.DattriError) as e:
                dt.dattri_cross_gram_workspace_bytes(a, x)
            assert _status(e) == want
            with pytest.raises(dt.DattriError) as e:
                dt.dattri_cross_gram(a, x, FAKE, 16, FAKE, 1 << 30)
            assert _status(e) == want
        with pytest.raises(dt.DattriError) as e:
            dt.dattri_cross_gram(a, b, FAKE, 2, FAKE, 1 << 30)   # ld_k < n_b
        assert _status(e) == "E_INVALID_ARG"
        with pytest.raises(dt.DattriError) as e:
            dt.dattri_cross_gram(a, b, None, 3, FAKE, 1 << 30)   # K NULL
        assert _status(e) == "E_INVALID_ARG"
        with pytest.raises(dt.DattriError) as e:
            dt.dattri_cross_gram(a, b, FAKE, 3, None, 0)         # workspace missing
        assert _status(e) == "E_WORKSPACE"
        need = dt.dattri_cross_gram_workspace_bytes(a, b)
        with pytest.raises(dt.DattriError) as e:
            dt.dattri_cross_gram(a, b, FAKE, 3, FAKE + 256, need - 1)
        assert _status(e) == "E_WORKSPACE"
        with pytest.raises(dt.DattriError) as e:
            dt.dattri_cross_gram_workspace_bytes(a, b, 7)
        assert _status(e) == "E_INVALID_ARG"
        with pytest.raises(dt.DattriError) as e:
            dt.dattri_cross_gram_route(a, b, 2)
        assert _status(e) == "E_INVALID_ARG"
        with pytest.raises(dt.DattriError) as e:
            dt.dattri_gradient_sq_norms(uncaptured, FAKE, FAKE, 1 << 30)
        assert _status(e) == "E_STATE"
        with pytest.raises(dt.DattriError) as e:
            dt.dattri_gradient_sq_norms(a, None, FAKE, 1 << 30)
        assert _status(e) == "E_INVALID_ARG"
        # both forced routes and AUTO size a workspace; the staged materialized
        # form holds DW of both batches
        model = dt.dattri_get_crossgram_cost_model(a)
        dt.dattri_set_crossgram_cost_model(a, dict(model, onepass_tflops=1e-9))
        wf = dt.dattri_cross_gram_workspace_bytes(a, b, dt.DATTRI_ROUTE_FACTORED)
        wm = dt.dattri_cross_gram_workspace_bytes(a, b, dt.DATTRI_ROUTE_MATERIALIZED)
        assert wm >= (4 + 3) * 64 * 32 * 4 and wf > 0
        assert dt.dattri_sq_norms_workspace_bytes(a, dt.DATTRI_ROUTE_MATERIALIZED) >= 4 * 64 * 32 * 4
        dt.dattri_set_crossgram_cost_model(a, model)
    finally:
        for c in (a, b, other, wrong_dims, f32, uncaptured):
            dt.dattri_destroy(c)


def test_route_regimes_and_cost_model():
    # App. A.4 "Regimes": short sequences and wide layers favour the
    # factorized route, long sequences the materialized one (with the MI355X
    # rates the crossover for 8 x 1 batches of this layer lies past T = 2048)
    short = _ctx([(1024, 4096)], 8, 32)
    q_short = _ctx([(1024, 4096)], 1, 32)
    long_ = _ctx([(1024, 4096)], 8, 8192)
    q_long = _ctx([(1024, 4096)], 1, 8192)
    try:
        r, f, m = dt.dattri_cross_gram_route(short, q_short, 0)
        assert r == dt.DATTRI_ROUTE_FACTORED and f < m
        r, f, m = dt.dattri_cross_gram_route(long_, q_long, 0)
        assert r == dt.DATTRI_ROUTE_MATERIALIZED and m < f
        model = dt.dattri_get_crossgram_cost_model(long_)
        assert all(v > 0 for v in model.values())
        slow_build = dict(model, build_tflops=1e-3, build_gbs=1e-3, onepass_tflops=1e-3)
        dt.dattri_set_crossgram_cost_model(long_, slow_build)
        assert dt.dattri_cross_gram_route(long_, q_long, 0)[0] == dt.DATTRI_ROUTE_FACTORED
        assert dt.dattri_get_crossgram_cost_model(long_) == pytest.approx(slow_build)
        for bad in (dict(model, ghost_tflops=0.0), dict(model, dot_gbs=float("nan")),
                    dict(model, launch_us=-1.0), dict(model, onepass_tflops=0.0)):
            with pytest.raises(dt.DattriError) as e:
                dt.dattri_set_crossgram_cost_model(long_, bad)
            assert _status(e) == "E_INVALID_ARG"
    finally:
        for c in (short, q_short, long_, q_long):
            dt.dattri_destroy(c)


def _ws(a, b, route=dt.DATTRI_ROUTE_MATERIALIZED):
    return dt.dattri_cross_gram_workspace_bytes(a, b, route)


def test_materialized_forms():
    # The materialized route takes the one-pass kernel (no DW in the workspace,
    # only one float per 128 x 128 tile of DW and example pair) for bf16 blocks
    # with 16-byte aligned rows when its predicted time is lower, else stages
    # DW of both batches; float32 and misaligned blocks always stage.
    a, q = _ctx([(1024, 4096)], 8, 2048), _ctx([(1024, 4096)], 1, 2048)
    a32, q32 = (_ctx([(1024, 4096)], 8, 2048, dtype=dt.DATTRI_F32),
                _ctx([(1024, 4096)], 1, 2048, dtype=dt.DATTRI_F32))
    mis, qmis = dt.dattri_create(dt.DATTRI_BF16, 0), _ctx([(1024, 4096)], 1, 2048)
    staged = (8 + 1) * 1024 * 4096 * 4
    try:
        lid = dt.dattri_register_layer(mis, 1024, 4096, 1, 1)
        dt.dattri_capture_layer(mis, lid, FAKE + 2, FAKE, 8, 2048)
        tiles = 8 * 32
        assert tiles * 8 * 4 <= _ws(a, q) < staged
        assert _ws(a32, q32) >= staged
        assert _ws(mis, qmis) >= staged
        # the route's predicted materialized time is the faster form
        r, f, m_one = dt.dattri_cross_gram_route(a, q, 0)
        model = dt.dattri_get_crossgram_cost_model(a)
        dt.dattri_set_crossgram_cost_model(a, dict(model, onepass_tflops=1e-9))
        r2, f2, m_staged = dt.dattri_cross_gram_route(a, q, 0)
        assert f2 == f and m_one < m_staged
        assert _ws(a, q) >= staged
        dt.dattri_set_crossgram_cost_model(a, model)
        # a square batch repeats the reference build per example: staged wins
        sq_a, sq_b = _ctx([(1024, 1024)], 16, 512), _ctx([(1024, 1024)], 16, 512)
        try:
            assert _ws(sq_a, sq_b) >= 32 * 1024 * 1024 * 4
            # the squared norms build every DW tile once either way: one-pass
            assert dt.dattri_sq_norms_workspace_bytes(sq_a, dt.DATTRI_ROUTE_MATERIALIZED) < 1024 * 1024 * 4
        finally:
            dt.dattri_destroy(sq_a)
            dt.dattri_destroy(sq_b)
    finally:
        for c in (a, q, a32, q32, mis, qmis):
            dt.dattri_destroy(c)
