// Host-side pieces shared by the translation units that implement the C ABI:
// the thread-local error message, HIP error mapping and size constants.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "dattri.h"

namespace dattri {

// Records a formatted message for dattri_last_error() and returns `st`.
dattri_status fail(dattri_status st, const char* fmt, ...);
void reset_error();
const char* last_error_message();

constexpr int64_t kMaxBlockBytes = ((int64_t)1 << 32) - 4096;  // 32-bit buffer offsets
constexpr size_t kAlign = 256;                                  // workspace sub-buffer alignment
inline size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }

// MI355X-fitted defaults of the cross-Gram time model (crossgram_api.cpp).
dattri_crossgram_cost_model default_crossgram_cost_model();

// Scoring (score_api.cpp): the checks and launches behind dattri_score /
// dattri_score_cosine, and the workspace bytes they need.
dattri_status score_impl(const void* phi_q, int64_t n_q, int64_t ld_q, const void* phi_train,
                         int64_t n_train, int64_t ld_train, int64_t F, dattri_dtype dtype,
                         const float* dev_precond_diag, float* scores, int32_t topk, int32_t* topk_idx,
                         float* topk_val, void* workspace, size_t ws_bytes, void* stream, bool cosine);
size_t score_workspace_need(int64_t n_q, int64_t n_train, int64_t F, int elt, bool precond, bool has_scores,
                            int32_t topk, bool cosine);

}  // namespace dattri

#define HIP_TRY(expr)                                                                     \
  do {                                                                                    \
    hipError_t e_ = (expr);                                                               \
    if (e_ != hipSuccess)                                                                 \
      return ::dattri::fail(DATTRI_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_)); \
  } while (0)
