"""The allocation-free scoring entry point (dattri_score_noalloc) through the C
ABI against dattri_score with a caller workspace: identical kernels, so the
scores and top-k must match bit for bit.  Two calls in a row, the second with
a smaller input (the static scratch keeps the first call's contents), and a
top-k-only call whose scores live in the scratch.  Run alone and after the
other GPU tests."""
import numpy as np
import pytest
import torch

import paper_2609_38767_amd as dt
from gpu_util import host64, rel_fro
from oracle import scoring as osc
from paper_2609_38767_amd.session import score

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _inputs(n_q, n_t, F, dtype, seed, precond):
    g = torch.Generator(device=DEV).manual_seed(seed)
    Q = torch.randn((n_q, F), generator=g, device=DEV).to(dtype)
    X = torch.randn((n_t, F), generator=g, device=DEV).to(dtype)
    d = torch.exp(torch.randn(F, generator=g, device=DEV)) if precond else None
    return Q, X, d


def _noalloc(Q, X, d, topk, want_scores=True):
    code = dt.DATTRI_BF16 if Q.dtype == torch.bfloat16 else dt.DATTRI_F32
    n_q, F = Q.shape
    n_t = X.shape[0]
    S = torch.full((n_q, n_t), float("nan"), device=DEV) if want_scores else None
    idx = torch.full((n_q, topk), -1, dtype=torch.int32, device=DEV) if topk else None
    val = torch.full((n_q, topk), float("nan"), device=DEV) if topk else None
    dt.dattri_score_noalloc(Q, n_q, Q.stride(0), X, n_t, X.stride(0), F, code, d, S, topk, idx, val)
    return S, idx, val


def test_noalloc_matches_workspace_entry_point_twice():
    # first call: bf16 through the 256 x 256 kernel (prepared queries in the
    # scratch) with the diagonal and top-k; second call: smaller, float32,
    # through the 128 x 128 kernel with the feature axis split (partial tiles
    # in the scratch)
    cases = [((300, 5000, 520), torch.bfloat16, True, 10), ((3, 200, 50008), torch.float32, False, 5)]
    for (n_q, n_t, F), dtype, precond, k in cases:
        print(f"[noalloc] n_q={n_q} n_train={n_t} F={F} {dtype} precond={precond} topk={k}", flush=True)
        Q, X, d = _inputs(n_q, n_t, F, dtype, 3 + n_q, precond)
        S_ref, i_ref, v_ref = score(Q, X, d, topk=k)
        S, idx, val = _noalloc(Q, X, d, k)
        torch.cuda.synchronize()
        assert torch.equal(S, S_ref)
        assert torch.equal(idx, i_ref) and torch.equal(val, v_ref)
        ref = osc.score(host64(Q), host64(X), None if d is None else host64(d))
        assert rel_fro(host64(S), ref) <= (5e-3 if precond and dtype == torch.bfloat16 else 1e-5)


def test_noalloc_topk_only_scores_in_scratch():
    Q, X, d = _inputs(7, 30000, 64, torch.float32, 11, True)  # 7 x 30000 scores: 840 KB of scratch
    _, i_ref, v_ref = score(Q, X, d, topk=50, want_scores=False)
    for _ in range(2):
        _, idx, val = _noalloc(Q, X, d, 50, want_scores=False)
        torch.cuda.synchronize()
        assert torch.equal(idx, i_ref) and torch.equal(val, v_ref)
    # every selected training row is among the oracle's best 50 up to float32 rounding
    S64 = osc.score(host64(Q), host64(X), host64(d))
    _, ref_val = osc.topk(S64, 50)
    picked = np.take_along_axis(S64, idx.cpu().numpy().astype(np.int64), axis=1)
    assert np.all(picked >= ref_val[:, -1:] - 1e-4 * np.abs(ref_val[:, :1]))


def test_noalloc_rejects_beyond_scratch():
    # top-k alone over 2048 x 10000 scores needs 82 MB of scratch: refused on
    # the host before any launch, outputs untouched
    Q, X, _ = _inputs(2048, 10000, 16, torch.float32, 5, False)
    idx = torch.full((2048, 4), -1, dtype=torch.int32, device=DEV)
    val = torch.zeros((2048, 4), device=DEV)
    with pytest.raises(dt.DattriError) as e:
        dt.dattri_score_noalloc(Q, 2048, 16, X, 10000, 16, 16, dt.DATTRI_F32, None, None, 4, idx, val)
    assert e.value.status_name == "E_UNSUPPORTED"
    torch.cuda.synchronize()
    assert torch.all(idx == -1)
