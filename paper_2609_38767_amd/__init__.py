"""Python binding of libdattri (MI355X projected-gradient attribution).

Argument marshalling only: every function here has the name of a C entry point
declared in include/dattri.h, converts its arguments (torch tensors become
device pointers, ``stream=None`` becomes torch's current HIP stream), calls the
library, raises ``DattriError`` on a non-OK status, and returns the C
function's output parameters.  No computation happens in Python, and there is
no fallback: if libdattri.so is missing, every call raises.

Build the library with ``python -m paper_2609_38767_amd.build``.
"""
import ctypes
import os

__all__ = [
    "DattriError", "lib_path", "load",
    "DATTRI_F32", "DATTRI_BF16", "DATTRI_ROUTE_AUTO", "DATTRI_ROUTE_FACTORED",
    "DATTRI_ROUTE_MATERIALIZED", "STATUS_NAMES", "EXPORTED",
    "dattri_create", "dattri_destroy", "dattri_last_error", "dattri_register_layer",
    "dattri_num_layers", "dattri_layer_dims", "dattri_feature_dim", "dattri_layer_offset",
    "dattri_projection_bytes", "dattri_bind_projection", "dattri_get_projection",
    "dattri_capture_layer", "dattri_clear_captures", "dattri_workspace_bytes",
    "dattri_project_per_example", "dattri_materialize_gradient", "dattri_set_cost_model",
    "dattri_get_cost_model", "dattri_layer_costs", "dattri_layer_route",
    "dattri_score_workspace_bytes", "dattri_feature_ld", "dattri_score",
    "dattri_set_crossgram_cost_model", "dattri_get_crossgram_cost_model", "dattri_cross_gram_costs",
    "dattri_cross_gram_route", "dattri_cross_gram_workspace_bytes", "dattri_cross_gram",
    "dattri_sq_norms_workspace_bytes", "dattri_gradient_sq_norms",
    "DATTRI_CURV_KFAC", "DATTRI_CURV_EKFAC", "CurvatureLayout",
    "dattri_curvature_state_bytes", "dattri_curvature_layout_of", "dattri_curvature_reset",
    "dattri_curvature_fit_workspace_bytes", "dattri_curvature_accumulate_factors",
    "dattri_curvature_eigen", "dattri_curvature_ekfac_workspace_bytes",
    "dattri_curvature_accumulate_ekfac", "dattri_curvature_precondition",
    "dattri_project_fit_workspace_bytes", "dattri_project_and_fit",
    "DATTRI_MAP_GAUSSIAN", "DATTRI_MAP_RADEMACHER", "dattri_set_map_kind", "dattri_get_map_kind",
    "dattri_cosine_workspace_bytes", "dattri_score_cosine",
    "DATTRI_ROUTE_MASK", "dattri_register_mask_layer", "dattri_get_mask",
    "dattri_token_scores_workspace_bytes", "dattri_token_scores",
    "dattri_probe_read", "dattri_probe_mfma",
]

DATTRI_F32, DATTRI_BF16 = 0, 1
DATTRI_ROUTE_AUTO, DATTRI_ROUTE_FACTORED, DATTRI_ROUTE_MATERIALIZED, DATTRI_ROUTE_MASK = 0, 1, 2, 3
DATTRI_FORM_AUTO, DATTRI_FORM_FUSED, DATTRI_FORM_SPLIT = 0, 1, 2
DATTRI_CURV_KFAC, DATTRI_CURV_EKFAC = 0, 1
DATTRI_MAP_GAUSSIAN, DATTRI_MAP_RADEMACHER = 0, 1
STATUS_NAMES = {0: "OK", -1: "E_INVALID_ARG", -2: "E_SHAPE", -3: "E_DTYPE", -4: "E_STATE",
                -5: "E_WORKSPACE", -6: "E_HIP", -7: "E_UNSUPPORTED"}

_HERE = os.path.dirname(os.path.abspath(__file__))
# DATTRI_LIB selects another build of the library (e.g. the host-sanitizer
# build, for CPU-only tests); the default is the in-tree libdattri.so.
lib_path = os.environ.get("DATTRI_LIB") or os.path.join(_HERE, "libdattri.so")


class DattriError(RuntimeError):
    def __init__(self, status, message, func):
        self.status = status
        self.status_name = STATUS_NAMES.get(status, str(status))
        super().__init__(f"{func}: {self.status_name}: {message}")


class CostModel(ctypes.Structure):
    _fields_ = [("factored_tflops", ctypes.c_double), ("factored_gbs", ctypes.c_double),
                ("gradient_tflops", ctypes.c_double), ("gradient_gbs", ctypes.c_double),
                ("gproject_tflops", ctypes.c_double), ("gproject_gbs", ctypes.c_double),
                ("launch_us", ctypes.c_double), ("call_us", ctypes.c_double), ("round_us", ctypes.c_double)]


class CrossgramCostModel(ctypes.Structure):
    _fields_ = [("ghost_tflops", ctypes.c_double), ("ghost_gbs", ctypes.c_double),
                ("ghost_layer_us", ctypes.c_double), ("build_tflops", ctypes.c_double), ("build_gbs", ctypes.c_double),
                ("dot_gbs", ctypes.c_double), ("launch_us", ctypes.c_double), ("onepass_tflops", ctypes.c_double)]


class CurvatureLayout(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int64) for name in
                ("sum_a", "sum_g", "sum_e", "q_a", "lam_a", "q_g", "lam_g", "counts")]


_i32, _i64, _u64, _sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_size_t
_vp, _dbl = ctypes.c_void_p, ctypes.c_double
_P = ctypes.POINTER

# name -> (restype, argtypes); the complete exported C ABI.
_SIGS = {
    "dattri_create": (_i32, [_P(_vp), _i32, _u64]),
    "dattri_destroy": (None, [_vp]),
    "dattri_last_error": (ctypes.c_char_p, []),
    "dattri_register_layer": (_i32, [_vp, _i32, _i32, _i32, _i32, _P(_i32)]),
    "dattri_num_layers": (_i32, [_vp, _P(_i32)]),
    "dattri_layer_dims": (_i32, [_vp, _i32, _P(_i32), _P(_i32), _P(_i32), _P(_i32)]),
    "dattri_feature_dim": (_i32, [_vp, _P(_i64)]),
    "dattri_layer_offset": (_i32, [_vp, _i32, _P(_i64)]),
    "dattri_projection_bytes": (_i32, [_vp, _i32, _P(_sz), _P(_sz)]),
    "dattri_bind_projection": (_i32, [_vp, _i32, _vp, _vp, _vp, _vp, _vp]),
    "dattri_get_projection": (_i32, [_vp, _i32, _vp, _vp]),
    "dattri_capture_layer": (_i32, [_vp, _i32, _vp, _vp, _i32, _i32, _vp]),
    "dattri_clear_captures": (_i32, [_vp]),
    "dattri_workspace_bytes": (_i32, [_vp, _i32, _P(_sz)]),
    "dattri_plan_bytes": (_i32, [_vp, _i32, _P(_sz)]),
    "dattri_bind_plan_buffer": (_i32, [_vp, _vp, _sz]),
    "dattri_set_factored_form": (_i32, [_vp, _i32]),
    "dattri_get_factored_form": (_i32, [_vp, _P(_i32)]),
    "dattri_project_per_example": (_i32, [_vp, _vp, _i32, _i64, _vp, _sz, _i32, _vp]),
    "dattri_materialize_gradient": (_i32, [_vp, _i32, _i32, _i32, _vp, _vp]),
    "dattri_set_cost_model": (_i32, [_vp, _P(CostModel)]),
    "dattri_get_cost_model": (_i32, [_vp, _P(CostModel)]),
    "dattri_set_cost_calibration": (_i32, [_vp, ctypes.c_char_p]),
    "dattri_layer_costs": (_i32, [_vp, _i32, _i32, _P(_i64), _P(_i64), _P(_i64), _P(_i64)]),
    "dattri_layer_route": (_i32, [_vp, _i32, _P(_i32), _P(_dbl), _P(_dbl)]),
    "dattri_score_workspace_bytes": (_i32, [_i64, _i64, _i64, _i32, _i32, _i32, _i32, _P(_sz)]),
    "dattri_feature_ld": (_i32, [_i64, _i32, _P(_i64)]),
    "dattri_set_crossgram_cost_model": (_i32, [_vp, _P(CrossgramCostModel)]),
    "dattri_get_crossgram_cost_model": (_i32, [_vp, _P(CrossgramCostModel)]),
    "dattri_cross_gram_costs": (_i32, [_i64, _i64, _i32, _i32, _i32, _i32, _i32, _P(_i64), _P(_i64),
                                       _P(_i64), _P(_i64)]),
    "dattri_cross_gram_route": (_i32, [_vp, _vp, _i32, _P(_i32), _P(_dbl), _P(_dbl)]),
    "dattri_cross_gram_workspace_bytes": (_i32, [_vp, _vp, _i32, _P(_sz)]),
    "dattri_cross_gram": (_i32, [_vp, _vp, _vp, _i64, _vp, _sz, _i32, _vp]),
    "dattri_sq_norms_workspace_bytes": (_i32, [_vp, _i32, _P(_sz)]),
    "dattri_gradient_sq_norms": (_i32, [_vp, _vp, _vp, _sz, _i32, _vp]),
    "dattri_score": (_i32, [_vp, _i64, _i64, _vp, _i64, _i64, _i64, _i32, _vp, _vp, _i32, _vp, _vp,
                            _vp, _sz, _vp]),
    "dattri_score_noalloc": (_i32, [_vp, _i64, _i64, _vp, _i64, _i64, _i64, _i32, _vp, _vp, _i32, _vp, _vp, _vp]),
    "dattri_curvature_state_bytes": (_i32, [_vp, _P(_sz)]),
    "dattri_curvature_layout_of": (_i32, [_vp, _i32, _P(CurvatureLayout)]),
    "dattri_curvature_reset": (_i32, [_vp, _vp, _vp]),
    "dattri_curvature_fit_workspace_bytes": (_i32, [_vp, _P(_sz)]),
    "dattri_curvature_accumulate_factors": (_i32, [_vp, _vp, _vp, _sz, _vp]),
    "dattri_curvature_eigen": (_i32, [_vp, _vp, _vp]),
    "dattri_curvature_ekfac_workspace_bytes": (_i32, [_vp, _i64, _P(_sz)]),
    "dattri_curvature_accumulate_ekfac": (_i32, [_vp, _vp, _vp, _i32, _i64, _i64, _vp, _sz, _vp]),
    "dattri_project_fit_workspace_bytes": (_i32, [_vp, _i32, _P(_sz)]),
    "dattri_set_map_kind": (_i32, [_vp, _i32, _i32]),
    "dattri_register_mask_layer": (_i32, [_vp, _i32, _i32, _i32, _i32, _i32, _P(_i32)]),
    "dattri_get_mask": (_i32, [_vp, _i32, _vp, _vp]),
    "dattri_token_scores_workspace_bytes": (_i32, [_vp, _P(_sz)]),
    "dattri_token_scores": (_i32, [_vp, _vp, _i32, _i64, _i64, _vp, _vp, _i32, _i64, _vp, _sz, _vp]),
    "dattri_probe_read": (_i32, [_vp, _sz, _vp, _i32, _vp]),
    "dattri_probe_mfma": (_i32, [_vp, _i32, _i32, _P(_dbl), _vp]),
    "dattri_cosine_workspace_bytes": (_i32, [_i64, _i64, _i64, _i32, _i32, _i32, _i32, _P(_sz)]),
    "dattri_score_cosine": (_i32, [_vp, _i64, _i64, _vp, _i64, _i64, _i64, _i32, _vp, _vp, _i32, _vp, _vp,
                                   _vp, _sz, _vp]),
    "dattri_get_map_kind": (_i32, [_vp, _i32, _P(_i32)]),
    "dattri_project_and_fit": (_i32, [_vp, _vp, _i32, _i64, _vp, _vp, _sz, _i32, _vp]),
    "dattri_curvature_precondition": (_i32, [_vp, _vp, _i32, _dbl, _dbl, _vp, _i32, _i64, _i64, _vp, _i32,
                                             _i64, _vp]),
}
EXPORTED = tuple(_SIGS)

_lib = None


def load():
    """Load libdattri.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(lib_path):
            raise RuntimeError(f"{lib_path} is not built; run `python -m paper_2609_38767_amd.build`")
        lib = ctypes.CDLL(lib_path)
        for name, (res, args) in _SIGS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _check(status, func):
    if status != 0:
        raise DattriError(status, load().dattri_last_error().decode(), func)


def _ptr(x):
    """Device/host pointer of a tensor or array, an int address, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if hasattr(x, "ctypes"):
        return x.ctypes.data
    raise TypeError(f"cannot take a pointer of {type(x)}")


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def dattri_last_error():
    return load().dattri_last_error().decode()


def dattri_create(compute, seed):
    ctx = _vp()
    _check(load().dattri_create(ctypes.byref(ctx), compute, seed), "dattri_create")
    return ctx.value


def dattri_destroy(ctx):
    load().dattri_destroy(ctx)


def dattri_register_layer(ctx, d_in, d_out, k_in, k_out):
    lid = _i32()
    _check(load().dattri_register_layer(ctx, d_in, d_out, k_in, k_out, ctypes.byref(lid)),
           "dattri_register_layer")
    return lid.value


def dattri_num_layers(ctx):
    n = _i32()
    _check(load().dattri_num_layers(ctx, ctypes.byref(n)), "dattri_num_layers")
    return n.value


def dattri_layer_dims(ctx, layer):
    v = [_i32() for _ in range(4)]
    _check(load().dattri_layer_dims(ctx, layer, *[ctypes.byref(x) for x in v]), "dattri_layer_dims")
    return tuple(x.value for x in v)


def dattri_feature_dim(ctx):
    F = _i64()
    _check(load().dattri_feature_dim(ctx, ctypes.byref(F)), "dattri_feature_dim")
    return F.value


def dattri_layer_offset(ctx, layer):
    o = _i64()
    _check(load().dattri_layer_offset(ctx, layer, ctypes.byref(o)), "dattri_layer_offset")
    return o.value


def dattri_projection_bytes(ctx, layer):
    a, b = _sz(), _sz()
    _check(load().dattri_projection_bytes(ctx, layer, ctypes.byref(a), ctypes.byref(b)),
           "dattri_projection_bytes")
    return a.value, b.value


def dattri_bind_projection(ctx, layer, dev_P_in, dev_P_out, host_P_in_override=None,
                           host_P_out_override=None, stream=None):
    _check(load().dattri_bind_projection(ctx, layer, _ptr(dev_P_in), _ptr(dev_P_out),
                                         _ptr(host_P_in_override), _ptr(host_P_out_override),
                                         _stream(stream)), "dattri_bind_projection")


def dattri_get_projection(ctx, layer):
    """Returns (P_in [d_in, k_in], P_out [d_out, k_out]) as float32 numpy arrays."""
    import numpy as np
    d_in, d_out, k_in, k_out = dattri_layer_dims(ctx, layer)
    p_in = np.empty((d_in, k_in), dtype=np.float32)
    p_out = np.empty((d_out, k_out), dtype=np.float32)
    _check(load().dattri_get_projection(ctx, layer, p_in.ctypes.data, p_out.ctypes.data),
           "dattri_get_projection")
    return p_in, p_out


def dattri_capture_layer(ctx, layer, A, B, n, T, dev_lengths=None):
    _check(load().dattri_capture_layer(ctx, layer, _ptr(A), _ptr(B), n, T, _ptr(dev_lengths)),
           "dattri_capture_layer")


def dattri_clear_captures(ctx):
    _check(load().dattri_clear_captures(ctx), "dattri_clear_captures")


def dattri_workspace_bytes(ctx, route=DATTRI_ROUTE_AUTO):
    b = _sz()
    _check(load().dattri_workspace_bytes(ctx, route, ctypes.byref(b)), "dattri_workspace_bytes")
    return b.value


def dattri_plan_bytes(ctx, route=DATTRI_ROUTE_AUTO):
    b = _sz()
    _check(load().dattri_plan_bytes(ctx, route, ctypes.byref(b)), "dattri_plan_bytes")
    return b.value


def dattri_bind_plan_buffer(ctx, buf, nbytes=None):
    """Bind a device buffer (tensor or address; None unbinds) for launch tables."""
    if buf is not None and nbytes is None:
        nbytes = buf.numel() * buf.element_size()
    _check(load().dattri_bind_plan_buffer(ctx, _ptr(buf), nbytes or 0), "dattri_bind_plan_buffer")


def dattri_set_factored_form(ctx, form):
    _check(load().dattri_set_factored_form(ctx, form), "dattri_set_factored_form")


def dattri_get_factored_form(ctx):
    f = _i32()
    _check(load().dattri_get_factored_form(ctx, ctypes.byref(f)), "dattri_get_factored_form")
    return f.value


def dattri_project_per_example(ctx, phi, phi_dtype, ld_phi, workspace, ws_bytes,
                               route=DATTRI_ROUTE_AUTO, stream=None):
    _check(load().dattri_project_per_example(ctx, _ptr(phi), phi_dtype, ld_phi, _ptr(workspace),
                                             ws_bytes, route, _stream(stream)),
           "dattri_project_per_example")


def dattri_materialize_gradient(ctx, layer, ex_begin, ex_count, G_out, stream=None):
    _check(load().dattri_materialize_gradient(ctx, layer, ex_begin, ex_count, _ptr(G_out),
                                              _stream(stream)), "dattri_materialize_gradient")


def dattri_set_cost_model(ctx, model):
    m = CostModel(**model) if isinstance(model, dict) else model
    _check(load().dattri_set_cost_model(ctx, ctypes.byref(m)), "dattri_set_cost_model")


def dattri_set_cost_calibration(ctx, json_path):
    _check(load().dattri_set_cost_calibration(ctx, os.fsencode(json_path)), "dattri_set_cost_calibration")


def dattri_get_cost_model(ctx):
    m = CostModel()
    _check(load().dattri_get_cost_model(ctx, ctypes.byref(m)), "dattri_get_cost_model")
    return {name: getattr(m, name) for name, _ in CostModel._fields_}


def dattri_layer_costs(ctx, layer, T):
    v = [_i64() for _ in range(4)]
    _check(load().dattri_layer_costs(ctx, layer, T, *[ctypes.byref(x) for x in v]),
           "dattri_layer_costs")
    return tuple(x.value for x in v)


def dattri_layer_route(ctx, layer):
    r, f, m = _i32(), _dbl(), _dbl()
    _check(load().dattri_layer_route(ctx, layer, ctypes.byref(r), ctypes.byref(f), ctypes.byref(m)),
           "dattri_layer_route")
    return r.value, f.value, m.value


def dattri_score_workspace_bytes(n_q, n_train, F, dtype, has_precond, has_scores, topk):
    b = _sz()
    _check(load().dattri_score_workspace_bytes(n_q, n_train, F, dtype, int(bool(has_precond)),
                                               int(bool(has_scores)), topk, ctypes.byref(b)),
           "dattri_score_workspace_bytes")
    return b.value


def dattri_feature_ld(F, dtype):
    v = _i64()
    _check(load().dattri_feature_ld(F, dtype, ctypes.byref(v)), "dattri_feature_ld")
    return v.value


def dattri_score(phi_q, n_q, ld_q, phi_train, n_train, ld_train, F, dtype, dev_precond_diag, scores,
                 topk, topk_idx, topk_val, workspace, ws_bytes, stream=None):
    _check(load().dattri_score(_ptr(phi_q), n_q, ld_q, _ptr(phi_train), n_train, ld_train, F, dtype,
                               _ptr(dev_precond_diag), _ptr(scores), topk, _ptr(topk_idx),
                               _ptr(topk_val), _ptr(workspace), ws_bytes, _stream(stream)),
           "dattri_score")


def dattri_score_noalloc(phi_q, n_q, ld_q, phi_train, n_train, ld_train, F, dtype, dev_precond_diag, scores,
                         topk, topk_idx, topk_val, stream=None):
    _check(load().dattri_score_noalloc(_ptr(phi_q), n_q, ld_q, _ptr(phi_train), n_train, ld_train, F, dtype,
                                       _ptr(dev_precond_diag), _ptr(scores), topk, _ptr(topk_idx),
                                       _ptr(topk_val), _stream(stream)),
           "dattri_score_noalloc")


def dattri_set_crossgram_cost_model(ctx, model):
    m = CrossgramCostModel(**model) if isinstance(model, dict) else model
    _check(load().dattri_set_crossgram_cost_model(ctx, ctypes.byref(m)), "dattri_set_crossgram_cost_model")


def dattri_get_crossgram_cost_model(ctx):
    m = CrossgramCostModel()
    _check(load().dattri_get_crossgram_cost_model(ctx, ctypes.byref(m)), "dattri_get_crossgram_cost_model")
    return {name: getattr(m, name) for name, _ in CrossgramCostModel._fields_}


def dattri_cross_gram_costs(n_a, n_b, T_a, T_b, d_in, d_out, elt_bytes):
    v = [_i64() for _ in range(4)]
    _check(load().dattri_cross_gram_costs(n_a, n_b, T_a, T_b, d_in, d_out, elt_bytes,
                                          *[ctypes.byref(x) for x in v]), "dattri_cross_gram_costs")
    return tuple(x.value for x in v)


def dattri_cross_gram_route(a, b, layer):
    r, f, m = _i32(), _dbl(), _dbl()
    _check(load().dattri_cross_gram_route(a, b, layer, ctypes.byref(r), ctypes.byref(f), ctypes.byref(m)),
           "dattri_cross_gram_route")
    return r.value, f.value, m.value


def dattri_cross_gram_workspace_bytes(a, b, route=DATTRI_ROUTE_AUTO):
    v = _sz()
    _check(load().dattri_cross_gram_workspace_bytes(a, b, route, ctypes.byref(v)),
           "dattri_cross_gram_workspace_bytes")
    return v.value


def dattri_cross_gram(a, b, K, ld_k, workspace, ws_bytes, route=DATTRI_ROUTE_AUTO, stream=None):
    _check(load().dattri_cross_gram(a, b, _ptr(K), ld_k, _ptr(workspace), ws_bytes, route, _stream(stream)),
           "dattri_cross_gram")


def dattri_sq_norms_workspace_bytes(ctx, route=DATTRI_ROUTE_AUTO):
    v = _sz()
    _check(load().dattri_sq_norms_workspace_bytes(ctx, route, ctypes.byref(v)),
           "dattri_sq_norms_workspace_bytes")
    return v.value


def dattri_gradient_sq_norms(ctx, out, workspace, ws_bytes, route=DATTRI_ROUTE_AUTO, stream=None):
    _check(load().dattri_gradient_sq_norms(ctx, _ptr(out), _ptr(workspace), ws_bytes, route, _stream(stream)),
           "dattri_gradient_sq_norms")


def dattri_curvature_state_bytes(ctx):
    v = _sz()
    _check(load().dattri_curvature_state_bytes(ctx, ctypes.byref(v)), "dattri_curvature_state_bytes")
    return v.value


def dattri_curvature_layout_of(ctx, layer):
    f = CurvatureLayout()
    _check(load().dattri_curvature_layout_of(ctx, layer, ctypes.byref(f)), "dattri_curvature_layout_of")
    return {name: getattr(f, name) for name, _ in CurvatureLayout._fields_}


def dattri_curvature_reset(ctx, state, stream=None):
    _check(load().dattri_curvature_reset(ctx, _ptr(state), _stream(stream)), "dattri_curvature_reset")


def dattri_curvature_fit_workspace_bytes(ctx):
    v = _sz()
    _check(load().dattri_curvature_fit_workspace_bytes(ctx, ctypes.byref(v)),
           "dattri_curvature_fit_workspace_bytes")
    return v.value


def dattri_curvature_accumulate_factors(ctx, state, workspace, ws_bytes, stream=None):
    _check(load().dattri_curvature_accumulate_factors(ctx, _ptr(state), _ptr(workspace), ws_bytes,
                                                      _stream(stream)),
           "dattri_curvature_accumulate_factors")


def dattri_curvature_eigen(ctx, state, stream=None):
    _check(load().dattri_curvature_eigen(ctx, _ptr(state), _stream(stream)), "dattri_curvature_eigen")


def dattri_curvature_ekfac_workspace_bytes(ctx, n):
    v = _sz()
    _check(load().dattri_curvature_ekfac_workspace_bytes(ctx, n, ctypes.byref(v)),
           "dattri_curvature_ekfac_workspace_bytes")
    return v.value


def dattri_curvature_accumulate_ekfac(ctx, state, phi, dtype, n, ld, workspace, ws_bytes, stream=None):
    _check(load().dattri_curvature_accumulate_ekfac(ctx, _ptr(state), _ptr(phi), dtype, n, ld, _ptr(workspace),
                                                    ws_bytes, _stream(stream)),
           "dattri_curvature_accumulate_ekfac")


def dattri_curvature_precondition(ctx, state, kind, damping_rel, damping_abs, phi_q, in_dtype, n_q, ld_q,
                                  out, out_dtype, ld_out, stream=None):
    _check(load().dattri_curvature_precondition(ctx, _ptr(state), kind, damping_rel, damping_abs, _ptr(phi_q),
                                                in_dtype, n_q, ld_q, _ptr(out), out_dtype, ld_out,
                                                _stream(stream)),
           "dattri_curvature_precondition")


def dattri_project_fit_workspace_bytes(ctx, route=DATTRI_ROUTE_AUTO):
    v = _sz()
    _check(load().dattri_project_fit_workspace_bytes(ctx, route, ctypes.byref(v)),
           "dattri_project_fit_workspace_bytes")
    return v.value


def dattri_project_and_fit(ctx, phi, phi_dtype, ld_phi, state, workspace, ws_bytes, route=DATTRI_ROUTE_AUTO,
                           stream=None):
    _check(load().dattri_project_and_fit(ctx, _ptr(phi), phi_dtype, ld_phi, _ptr(state), _ptr(workspace), ws_bytes,
                                         route, _stream(stream)),
           "dattri_project_and_fit")


def dattri_set_map_kind(ctx, layer, kind):
    _check(load().dattri_set_map_kind(ctx, layer, kind), "dattri_set_map_kind")


def dattri_get_map_kind(ctx, layer):
    v = _i32()
    _check(load().dattri_get_map_kind(ctx, layer, ctypes.byref(v)), "dattri_get_map_kind")
    return v.value


def dattri_cosine_workspace_bytes(n_q, n_train, F, dtype, has_precond, has_scores, topk):
    v = _sz()
    _check(load().dattri_cosine_workspace_bytes(n_q, n_train, F, dtype, int(bool(has_precond)),
                                                int(bool(has_scores)), topk, ctypes.byref(v)),
           "dattri_cosine_workspace_bytes")
    return v.value


def dattri_score_cosine(phi_q, n_q, ld_q, phi_train, n_train, ld_train, F, dtype, dev_precond_diag, scores,
                        topk, topk_idx, topk_val, workspace, ws_bytes, stream=None):
    _check(load().dattri_score_cosine(_ptr(phi_q), n_q, ld_q, _ptr(phi_train), n_train, ld_train, F, dtype,
                                      _ptr(dev_precond_diag), _ptr(scores), topk, _ptr(topk_idx), _ptr(topk_val),
                                      _ptr(workspace), ws_bytes, _stream(stream)),
           "dattri_score_cosine")


def dattri_register_mask_layer(ctx, d_in, d_out, mask_size, mask_id=0, mask_count=1):
    lid = _i32()
    _check(load().dattri_register_mask_layer(ctx, d_in, d_out, mask_size, mask_id, mask_count, ctypes.byref(lid)),
           "dattri_register_mask_layer")
    return lid.value


def dattri_get_mask(ctx, layer):
    """(rows, cols) int32 numpy arrays of a mask layer's entries."""
    import numpy as np
    _, _, _, m = dattri_layer_dims(ctx, layer)
    rows = np.empty(m, dtype=np.int32)
    cols = np.empty(m, dtype=np.int32)
    _check(load().dattri_get_mask(ctx, layer, rows.ctypes.data, cols.ctypes.data), "dattri_get_mask")
    return rows, cols


def dattri_token_scores_workspace_bytes(ctx):
    v = _sz()
    _check(load().dattri_token_scores_workspace_bytes(ctx, ctypes.byref(v)), "dattri_token_scores_workspace_bytes")
    return v.value


def dattri_token_scores(ctx, phi_q, q_dtype, n_q, ld_q, scores, phi, phi_dtype, ld_phi, workspace, ws_bytes,
                        stream=None):
    _check(load().dattri_token_scores(ctx, _ptr(phi_q), q_dtype, n_q, ld_q, _ptr(scores), _ptr(phi), phi_dtype,
                                      ld_phi, _ptr(workspace), ws_bytes, _stream(stream)),
           "dattri_token_scores")


def dattri_probe_read(buf, nbytes, sink, workgroups, stream=None):
    _check(load().dattri_probe_read(_ptr(buf), nbytes, _ptr(sink), workgroups, _stream(stream)), "dattri_probe_read")


def dattri_probe_mfma(sink, workgroups, iters, stream=None):
    """Launch the MFMA probe; returns the launch's FLOP count."""
    f = _dbl()
    _check(load().dattri_probe_mfma(_ptr(sink), workgroups, iters, ctypes.byref(f), _stream(stream)),
           "dattri_probe_mfma")
    return f.value
