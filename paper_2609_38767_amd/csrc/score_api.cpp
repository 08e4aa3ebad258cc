// C ABI of scoring (GradDot with an optional diagonal preconditioner, Sec. 4.1;
// inner products of projected gradients, Eq. (4)) and per-query top-k:
// argument validation, workspace layout and kernel launches.
#include <algorithm>

#include "api_common.h"
#include "dattri.h"
#include "internal.h"

using namespace dattri;

namespace {
// Row stride (elements) for feature rows on MI355X: rows rounded up to 256
// bytes, plus 512 bytes when that leaves them a multiple of 8 KiB at 16 KiB or
// more.  Rows whose byte stride is such a multiple put the same column of
// many rows into the same few L2 sets, and a GEMM that reads one column chunk
// of 256 rows at a time then misses L2 on operands it should share (measured
// with 256 workgroups each reading 128-byte chunks of 256 rows: 13-14 B/clk per
// CU at strides of 16, 32, 48 and 128 KiB, 47-48.5 B/clk with 512 bytes added;
// 256 bytes added is not enough at 32 KiB).
int64_t feature_ld(int64_t F, int elt) {
  int64_t rb = (F * elt + 255) / 256 * 256;
  if (rb >= 16384 && rb % 8192 == 0) rb += 512;
  return rb / elt;
}

struct ScoreLayout {
  int64_t ldq;
  size_t off_q, q_bytes, off_s, s_bytes, off_p, p_bytes, off_n, n_bytes, total;
};

// Prepared queries: packed in MFMA fragment order for the 256 x 256 kernel
// (always), else a preconditioned row-major copy at the recommended stride.
ScoreLayout score_layout(int64_t n_q, int64_t n_train, int64_t F, int elt, bool precond,
                         bool has_scores, int32_t topk, bool cosine = false) {
  ScoreLayout L;
  size_t off = 0;
  L.ldq = feature_ld(F, elt);
  L.off_q = off;
  if (score_uses_big(elt, n_q, n_train))
    L.q_bytes = (size_t)score_qpack_bytes(n_q, F);
  else
    L.q_bytes = precond ? (size_t)(n_q * L.ldq * elt) : 0;
  off = align_up(off + L.q_bytes);
  L.off_s = off;
  L.s_bytes = (!has_scores && topk > 0) ? (size_t)(n_q * n_train * 4) : 0;
  off = align_up(off + L.s_bytes);
  L.off_p = off;
  L.p_bytes = (size_t)score_partial_floats(elt, n_q, n_train, F) * 4;
  off = align_up(off + L.p_bytes);
  L.off_n = off;  // cosine: inverse row norms of the queries, then of the training rows
  L.n_bytes = cosine ? (size_t)(n_q + n_train) * 4 : 0;
  off = align_up(off + L.n_bytes);
  L.total = std::max<size_t>(off, kAlign);
  return L;
}
}  // namespace

size_t dattri::score_workspace_need(int64_t n_q, int64_t n_train, int64_t F, int elt, bool precond,
                                    bool has_scores, int32_t topk, bool cosine) {
  return score_layout(n_q, n_train, F, elt, precond, has_scores, topk, cosine).total;
}

dattri_status dattri::score_impl(const void* phi_q, int64_t n_q, int64_t ld_q, const void* phi_train,
                         int64_t n_train, int64_t ld_train, int64_t F, dattri_dtype dtype,
                         const float* dev_precond_diag, float* scores, int32_t topk, int32_t* topk_idx,
                         float* topk_val, void* workspace, size_t ws_bytes, void* stream, bool cosine) {
  if (dtype != DATTRI_F32 && dtype != DATTRI_BF16)
    return fail(DATTRI_E_DTYPE, "dtype %d is neither F32 nor BF16", (int)dtype);
  if (n_q < 0 || n_train < 0 || F < 0 || topk < 0 || ld_q < 0 || ld_train < 0)
    return fail(DATTRI_E_INVALID_ARG, "sizes must be >= 0");
  if (ld_q == 0) ld_q = F;
  if (ld_train == 0) ld_train = F;
  if (ld_q < F || ld_train < F)
    return fail(DATTRI_E_INVALID_ARG, "row strides (ld_q=%lld, ld_train=%lld) must be >= F=%lld",
                (long long)ld_q, (long long)ld_train, (long long)F);
  if (n_q > INT32_MAX || n_train > INT32_MAX || F > INT32_MAX)
    return fail(DATTRI_E_UNSUPPORTED, "n_q, n_train and F must each fit in int32");
  if (topk > kTopkMax) return fail(DATTRI_E_UNSUPPORTED, "topk=%d exceeds %d", topk, kTopkMax);
  if (topk > n_train) return fail(DATTRI_E_INVALID_ARG, "topk=%d exceeds n_train=%lld", topk, (long long)n_train);
  if (!scores && topk == 0) return fail(DATTRI_E_INVALID_ARG, "nothing to compute: scores is NULL and topk is 0");
  if (topk > 0 && (!topk_idx || !topk_val))
    return fail(DATTRI_E_INVALID_ARG, "topk_idx and topk_val are required when topk > 0");
  if (n_q == 0 || n_train == 0) return DATTRI_OK;
  if (F > 0 && (!phi_q || !phi_train)) return fail(DATTRI_E_INVALID_ARG, "phi_q or phi_train is NULL");
  const int elt = dtype == DATTRI_BF16 ? 2 : 4;
  const ScoreLayout L = score_layout(n_q, n_train, F, elt, dev_precond_diag != nullptr,
                                     scores != nullptr, topk, cosine);
  const int64_t ld_max = std::max({ld_q, ld_train, L.ldq});
  if (ld_max * elt * 256 >= kMaxBlockBytes)
    return fail(DATTRI_E_UNSUPPORTED, "row stride %lld too large (256 rows must stay below 4 GiB)",
                (long long)ld_max);
  if ((uintptr_t)phi_q % 16 || (uintptr_t)phi_train % 16 || (F * elt) % 16 || (ld_q * elt) % 16 ||
      (ld_train * elt) % 16)
    return fail(DATTRI_E_UNSUPPORTED,
                "phi rows must be 16-byte aligned (pointers, F*%d and ld*%d multiples of 16)", elt, elt);
  if (L.q_bytes + L.s_bytes + L.p_bytes + L.n_bytes > 0) {
    if (!workspace) return fail(DATTRI_E_WORKSPACE, "workspace is NULL (needs %zu bytes)", L.total);
    if ((uintptr_t)workspace % kAlign) return fail(DATTRI_E_WORKSPACE, "workspace must be 256-byte aligned");
    if (ws_bytes < L.total)
      return fail(DATTRI_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, L.total);
  }
  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)workspace;
  float* S = scores ? scores : (float*)(ws + L.off_s);
  HIP_TRY(launch_score_gemm(elt, phi_q, ld_q, dev_precond_diag, phi_train, ld_train, S, n_q, n_train,
                            F, L.q_bytes ? ws + L.off_q : nullptr, L.ldq,
                            L.p_bytes ? (float*)(ws + L.off_p) : nullptr, s));
  if (cosine) {
    float* inv = (float*)(ws + L.off_n);
    HIP_TRY(launch_cosine_scale(elt, phi_q, ld_q, dev_precond_diag, phi_train, ld_train, S, n_q, n_train, F, inv,
                                inv + n_q, s));
  }
  if (topk > 0) HIP_TRY(launch_topk(S, n_q, n_train, topk, topk_idx, topk_val, s));
  return DATTRI_OK;
}

extern "C" {

dattri_status dattri_feature_ld(int64_t F, dattri_dtype dtype, int64_t* ld) {
  reset_error();
  if (!ld) return fail(DATTRI_E_INVALID_ARG, "ld is NULL");
  if (F < 0) return fail(DATTRI_E_INVALID_ARG, "F must be >= 0");
  if (dtype != DATTRI_F32 && dtype != DATTRI_BF16)
    return fail(DATTRI_E_DTYPE, "dtype %d is neither F32 nor BF16", (int)dtype);
  *ld = feature_ld(F, dtype == DATTRI_BF16 ? 2 : 4);
  return DATTRI_OK;
}

dattri_status dattri_score_workspace_bytes(int64_t n_q, int64_t n_train, int64_t F,
                                           dattri_dtype dtype, int32_t has_precond,
                                           int32_t has_scores, int32_t topk, size_t* bytes) {
  reset_error();
  if (!bytes) return fail(DATTRI_E_INVALID_ARG, "bytes is NULL");
  if (n_q < 0 || n_train < 0 || F < 0 || topk < 0)
    return fail(DATTRI_E_INVALID_ARG, "sizes must be >= 0");
  if (dtype != DATTRI_F32 && dtype != DATTRI_BF16)
    return fail(DATTRI_E_DTYPE, "dtype %d is neither F32 nor BF16", (int)dtype);
  *bytes = score_layout(n_q, n_train, F, dtype == DATTRI_BF16 ? 2 : 4, has_precond != 0,
                        has_scores != 0, topk).total;
  return DATTRI_OK;
}

dattri_status dattri_score(const void* phi_q, int64_t n_q, int64_t ld_q, const void* phi_train,
                           int64_t n_train, int64_t ld_train, int64_t F, dattri_dtype dtype,
                           const float* dev_precond_diag, float* scores, int32_t topk,
                           int32_t* topk_idx, float* topk_val, void* workspace, size_t ws_bytes,
                           void* stream) {
  reset_error();
  return score_impl(phi_q, n_q, ld_q, phi_train, n_train, ld_train, F, dtype, dev_precond_diag, scores, topk,
                    topk_idx, topk_val, workspace, ws_bytes, stream, false);
}

dattri_status dattri_cosine_workspace_bytes(int64_t n_q, int64_t n_train, int64_t F, dattri_dtype dtype,
                                            int32_t has_precond, int32_t has_scores, int32_t topk,
                                            size_t* bytes) {
  reset_error();
  if (!bytes) return fail(DATTRI_E_INVALID_ARG, "bytes is NULL");
  if (n_q < 0 || n_train < 0 || F < 0 || topk < 0)
    return fail(DATTRI_E_INVALID_ARG, "sizes must be >= 0");
  if (dtype != DATTRI_F32 && dtype != DATTRI_BF16)
    return fail(DATTRI_E_DTYPE, "dtype %d is neither F32 nor BF16", (int)dtype);
  *bytes = score_layout(n_q, n_train, F, dtype == DATTRI_BF16 ? 2 : 4, has_precond != 0, has_scores != 0, topk,
                        true).total;
  return DATTRI_OK;
}

dattri_status dattri_score_cosine(const void* phi_q, int64_t n_q, int64_t ld_q, const void* phi_train,
                                  int64_t n_train, int64_t ld_train, int64_t F, dattri_dtype dtype,
                                  const float* dev_precond_diag, float* scores, int32_t topk,
                                  int32_t* topk_idx, float* topk_val, void* workspace, size_t ws_bytes,
                                  void* stream) {
  reset_error();
  return score_impl(phi_q, n_q, ld_q, phi_train, n_train, ld_train, F, dtype, dev_precond_diag, scores, topk,
                    topk_idx, topk_val, workspace, ws_bytes, stream, true);
}

}  // extern "C"
