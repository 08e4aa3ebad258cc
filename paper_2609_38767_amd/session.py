"""Convenience wrappers over the C ABI that let torch own the device buffers.

``ProjectionSession`` registers layers, allocates and binds the projection
maps, captures factor blocks, sizes the workspace and calls
``dattri_project_per_example``; ``score`` sizes the scoring workspace and calls
``dattri_score``; ``Curvature`` owns a K-FAC / EK-FAC curvature state and runs
its fit, eigendecomposition, eigenvalue correction and query preconditioning.
All computation happens in libdattri's HIP kernels.
"""
import torch

from . import (DATTRI_BF16, DATTRI_F32, DATTRI_ROUTE_AUTO, dattri_bind_projection,
               dattri_cross_gram, dattri_cross_gram_workspace_bytes, dattri_gradient_sq_norms,
               dattri_sq_norms_workspace_bytes,
               dattri_capture_layer, dattri_clear_captures, dattri_create, dattri_destroy,
               dattri_feature_dim, dattri_feature_ld, dattri_layer_offset, dattri_layer_route,
               dattri_project_per_example, dattri_projection_bytes, dattri_register_layer,
               dattri_score, dattri_score_workspace_bytes, dattri_set_factored_form,
               dattri_workspace_bytes, DATTRI_CURV_KFAC, DATTRI_CURV_EKFAC,
               dattri_curvature_state_bytes, dattri_curvature_layout_of, dattri_curvature_reset,
               dattri_curvature_fit_workspace_bytes, dattri_curvature_accumulate_factors,
               dattri_curvature_eigen, dattri_curvature_ekfac_workspace_bytes,
               dattri_curvature_accumulate_ekfac, dattri_curvature_precondition,
               dattri_project_fit_workspace_bytes, dattri_project_and_fit, dattri_set_map_kind,
               dattri_cosine_workspace_bytes, dattri_score_cosine, dattri_register_mask_layer,
               dattri_token_scores_workspace_bytes, dattri_token_scores, dattri_bind_plan_buffer)

DTYPES = {"f32": (DATTRI_F32, torch.float32), "bf16": (DATTRI_BF16, torch.bfloat16)}
PLAN_BUFFER_BYTES = 8 << 20  # launch tables kept on the device between calls


def _dev_bytes(n, device):
    return torch.empty(max(int(n), 256), dtype=torch.uint8, device=device)


class ProjectionSession:
    """One library context with its layers and bound projection maps."""

    def __init__(self, layers, dtype="bf16", seed=0, device="cuda", overrides=None, form=None, map_kind=None,
                 plan_buffer=True):
        self.dtype = dtype
        self.code, self.torch_dtype = DTYPES[dtype]
        self.device = torch.device(device)
        self.ctx = dattri_create(self.code, seed)
        self.plan_buf = None
        if plan_buffer:  # repeated calls with unchanged captures then copy nothing to the device
            self.plan_buf = _dev_bytes(PLAN_BUFFER_BYTES, self.device)
            dattri_bind_plan_buffer(self.ctx, self.plan_buf)
        if form is not None:
            dattri_set_factored_form(self.ctx, form)
        self.layers = list(layers)
        self.maps = []
        overrides = overrides or {}
        for i, L in enumerate(self.layers):
            if L.get("mask_size"):  # a random-mask layer (entries of DW gathered from the factors)
                lid = dattri_register_mask_layer(self.ctx, L["d_in"], L["d_out"], L["mask_size"],
                                                 L.get("mask_id", 0), L.get("mask_count", 1))
            else:
                lid = dattri_register_layer(self.ctx, L["d_in"], L["d_out"], L["k_in"], L["k_out"])
                if map_kind is not None:
                    dattri_set_map_kind(self.ctx, lid, map_kind)
            assert lid == i
            b_in, b_out = dattri_projection_bytes(self.ctx, lid)
            p_in, p_out = _dev_bytes(b_in, self.device), _dev_bytes(b_out, self.device)
            o_in, o_out = overrides.get(i, (None, None))
            dattri_bind_projection(self.ctx, lid, p_in, p_out, o_in, o_out)
            self.maps.append((p_in, p_out))
        self.F = dattri_feature_dim(self.ctx)
        self.offsets = [dattri_layer_offset(self.ctx, i) for i in range(len(self.layers))]
        self._ws = None
        self._held = []

    def capture(self, layer, A, B, lengths=None):
        """A [n, T, d_in], B [n, T, d_out] contiguous device tensors of the compute dtype."""
        assert A.is_contiguous() and B.is_contiguous()
        assert A.dtype == self.torch_dtype and B.dtype == self.torch_dtype
        n, T = A.shape[0], A.shape[1]
        dattri_capture_layer(self.ctx, layer, A, B, n, T, lengths)
        self._held.append((A, B, lengths))

    def clear(self):
        dattri_clear_captures(self.ctx)
        self._held = []

    def workspace(self, route=DATTRI_ROUTE_AUTO):
        need = dattri_workspace_bytes(self.ctx, route)
        if self._ws is None or self._ws.numel() < need:
            self._ws = None
            self._ws = _dev_bytes(need, self.device)
        return self._ws

    def project(self, n, route=DATTRI_ROUTE_AUTO, phi_dtype="f32", phi=None, stream=None):
        code, tdt = DTYPES[phi_dtype]
        if phi is None:  # rows at the library's recommended stride (a view)
            phi = feature_rows(n, self.F, phi_dtype, self.device)
        ws = self.workspace(route)
        dattri_project_per_example(self.ctx, phi, code, phi.stride(0), ws, ws.numel(), route, stream)
        return phi

    def token_scores(self, phi_q, n, phi_dtype="f32", stream=None):
        """(scores [n_q, n, T] float32, phi) for the captures: per-token
        contributions of every training example to its score against each
        query row (GradDot rows, or rows preconditioned by a Curvature)."""
        T = self._held[0][0].shape[1]
        code, _ = DTYPES[phi_dtype]
        q_code = DATTRI_BF16 if phi_q.dtype == torch.bfloat16 else DATTRI_F32
        phi = feature_rows(n, self.F, phi_dtype, self.device)
        scores = torch.empty((phi_q.shape[0], n, T), dtype=torch.float32, device=self.device)
        need = dattri_token_scores_workspace_bytes(self.ctx)
        ws = _dev_bytes(need, self.device)
        dattri_token_scores(self.ctx, phi_q, q_code, phi_q.shape[0], phi_q.stride(0), scores, phi, code,
                            phi.stride(0), ws, ws.numel(), stream)
        return scores, phi

    def routes(self):
        return [dattri_layer_route(self.ctx, i) for i in range(len(self.layers))]

    def close(self):
        if self.ctx:
            dattri_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def feature_rows(n, F, dtype="bf16", device="cuda"):
    """Uninitialised [n, F] feature rows of `dtype` ("bf16" or "f32") whose
    row stride is the library's recommended one (a view into a padded buffer)."""
    code, tdt = DTYPES[dtype]
    ld = dattri_feature_ld(F, code)
    return torch.empty((n, ld), dtype=tdt, device=device)[:, :F]


def score(phi_q, phi_train, precond=None, topk=0, want_scores=True, stream=None, cosine=False):
    """(S or None, topk_idx or None, topk_val or None) for bf16/f32 feature
    rows; each operand may be row-strided (unit stride along features).
    cosine=True divides every score by the norms of its two rows."""
    code = DATTRI_BF16 if phi_q.dtype == torch.bfloat16 else DATTRI_F32
    n_q, F = phi_q.shape
    n_train = phi_train.shape[0]
    for t in (phi_q, phi_train):
        if t.shape[1] > 1 and t.stride(1) != 1:
            raise ValueError("feature rows must be contiguous along the feature axis")
    dev = phi_q.device
    S = torch.empty((n_q, n_train), dtype=torch.float32, device=dev) if want_scores else None
    idx = torch.empty((n_q, topk), dtype=torch.int32, device=dev) if topk else None
    val = torch.empty((n_q, topk), dtype=torch.float32, device=dev) if topk else None
    sizer, fn = ((dattri_cosine_workspace_bytes, dattri_score_cosine) if cosine
                 else (dattri_score_workspace_bytes, dattri_score))
    need = sizer(n_q, n_train, F, code, precond is not None, want_scores, topk)
    ws = _dev_bytes(need, dev)
    fn(phi_q, n_q, phi_q.stride(0), phi_train, n_train, phi_train.stride(0), F, code, precond,
       S, topk, idx, val, ws, ws.numel(), stream)
    return S, idx, val


def cross_gram(sess_a, sess_b, route=DATTRI_ROUTE_AUTO, K=None, stream=None):
    """K [n_a, n_b] float32: the cross-Gram of the unprojected gradients captured
    in two sessions over the same layers (sess_b may be sess_a)."""
    n_a = sess_a._held[0][0].shape[0]
    n_b = sess_b._held[0][0].shape[0]
    if K is None:
        K = torch.empty((n_a, n_b), dtype=torch.float32, device=sess_a.device)
    ws = _dev_bytes(dattri_cross_gram_workspace_bytes(sess_a.ctx, sess_b.ctx, route), sess_a.device)
    dattri_cross_gram(sess_a.ctx, sess_b.ctx, K, K.stride(0), ws, ws.numel(), route, stream)
    return K


def sq_norms(sess, route=DATTRI_ROUTE_AUTO, stream=None):
    """Per-example squared gradient norms [n] float32, summed over layers."""
    n = sess._held[0][0].shape[0]
    out = torch.empty(n, dtype=torch.float32, device=sess.device)
    ws = _dev_bytes(dattri_sq_norms_workspace_bytes(sess.ctx, route), sess.device)
    dattri_gradient_sq_norms(sess.ctx, out, ws, ws.numel(), route, stream)
    return out


KINDS = {"kfac": DATTRI_CURV_KFAC, "ekfac": DATTRI_CURV_EKFAC}


class Curvature:
    """K-FAC / EK-FAC curvature state of a session's layers in one device buffer."""

    def __init__(self, sess, stream=None):
        self.sess = sess
        self.nbytes = dattri_curvature_state_bytes(sess.ctx)
        self.state = _dev_bytes(self.nbytes, sess.device)
        self._ws = None
        self.reset(stream)

    def _workspace(self, need):
        if self._ws is None or self._ws.numel() < need:
            self._ws = None
            self._ws = _dev_bytes(need, self.sess.device)
        return self._ws

    def reset(self, stream=None):
        dattri_curvature_reset(self.sess.ctx, self.state, stream)

    def accumulate_factors(self, stream=None):
        """Adds the projected factor sums of the session's current captures."""
        ws = self._workspace(dattri_curvature_fit_workspace_bytes(self.sess.ctx))
        dattri_curvature_accumulate_factors(self.sess.ctx, self.state, ws, ws.numel(), stream)

    def project_and_fit(self, n, route=DATTRI_ROUTE_AUTO, phi_dtype="f32", phi=None, stream=None):
        """The session's projected gradients and, in the same pass, the factor
        sums of its captures."""
        code, _ = DTYPES[phi_dtype]
        if phi is None:
            phi = feature_rows(n, self.sess.F, phi_dtype, self.sess.device)
        ws = self._workspace(dattri_project_fit_workspace_bytes(self.sess.ctx, route))
        dattri_project_and_fit(self.sess.ctx, phi, code, phi.stride(0), self.state, ws, ws.numel(), route, stream)
        return phi

    def eigen(self, stream=None):
        dattri_curvature_eigen(self.sess.ctx, self.state, stream)

    def accumulate_ekfac(self, phi, stream=None):
        """EK-FAC's correction from training rows phi [n, F] (row-strided allowed)."""
        code = DATTRI_BF16 if phi.dtype == torch.bfloat16 else DATTRI_F32
        n = phi.shape[0]
        ws = self._workspace(dattri_curvature_ekfac_workspace_bytes(self.sess.ctx, n))
        dattri_curvature_accumulate_ekfac(self.sess.ctx, self.state, phi, code, n, phi.stride(0), ws,
                                          ws.numel(), stream)

    def precondition(self, phi_q, kind="ekfac", rel=0.1, abs_=0.0, out_dtype=None, out=None, stream=None):
        """Preconditioned query rows (rows at the library's recommended stride)."""
        in_code = DATTRI_BF16 if phi_q.dtype == torch.bfloat16 else DATTRI_F32
        if out is None:
            od = out_dtype or ("bf16" if in_code == DATTRI_BF16 else "f32")
            out = feature_rows(phi_q.shape[0], self.sess.F, od, self.sess.device)
        out_code = DATTRI_BF16 if out.dtype == torch.bfloat16 else DATTRI_F32
        dattri_curvature_precondition(self.sess.ctx, self.state, KINDS[kind], rel, abs_, phi_q, in_code,
                                      phi_q.shape[0], phi_q.stride(0), out, out_code, out.stride(0), stream)
        return out

    def layout(self, layer):
        return dattri_curvature_layout_of(self.sess.ctx, layer)

    def field(self, layer, name):
        """View of one field of a layer in the state: float32 matrices / vectors,
        int64 counts."""
        f = self.layout(layer)
        L = self.sess.layers[layer]
        ki, ko = L["k_in"], L["k_out"]
        shapes = {"sum_a": (ki, ki), "sum_g": (ko, ko), "sum_e": (ki, ko), "q_a": (ki, ki), "lam_a": (ki,),
                  "q_g": (ko, ko), "lam_g": (ko,), "counts": (3,)}
        shape = shapes[name]
        dt = torch.int64 if name == "counts" else torch.float32
        n = 1
        for v in shape:
            n *= v
        off = f[name]
        return self.state[off:off + n * dt.itemsize].view(dt).view(shape)
