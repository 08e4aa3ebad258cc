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

}  // namespace dattri

#define HIP_TRY(expr)                                                                     \
  do {                                                                                    \
    hipError_t e_ = (expr);                                                               \
    if (e_ != hipSuccess)                                                                 \
      return ::dattri::fail(DATTRI_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_)); \
  } while (0)
