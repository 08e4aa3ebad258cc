// Scoring without a caller workspace (dattri_score_noalloc): the scratch the
// score kernels use (prepared queries, split-feature partial tiles, scores kept
// only for top-k) lives in a file-scope device array of fixed size that each
// GPU holds from the library's first use on it until the process ends.
//
// The array's name in host code is only a stand-in for the symbol: its device
// address differs per GPU and is looked up with hipGetSymbolAddress, once per
// device with that device current, and kept in g_scratch[]; only that address
// is ever passed to kernels or copies.
#include <mutex>

#include "api_common.h"
#include "dattri.h"
#include "internal.h"

namespace dattri {
namespace {

constexpr size_t kScratchBytes = DATTRI_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % kAlign == 0, "scratch size");

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` on each GPU, once looked up

// Address of the scratch array on the current device.
dattri_status scratch_address(void** out) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(DATTRI_E_UNSUPPORTED, "device %d beyond the %d this build tracks", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(DATTRI_E_HIP, "hipGetSymbolAddress returned NULL for the scratch array");
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return DATTRI_OK;
}

}  // namespace
}  // namespace dattri

using namespace dattri;

extern "C" dattri_status dattri_score_noalloc(const void* phi_q, int64_t n_q, int64_t ld_q, const void* phi_train,
                                              int64_t n_train, int64_t ld_train, int64_t F, dattri_dtype dtype,
                                              const float* dev_precond_diag, float* scores, int32_t topk,
                                              int32_t* topk_idx, float* topk_val, void* stream) {
  reset_error();
  // the scratch this call needs, from arguments dattri_score checks the same way
  if (dtype == DATTRI_F32 || dtype == DATTRI_BF16) {
    if (n_q > 0 && n_train > 0 && F >= 0 && topk >= 0 && n_q <= INT32_MAX && n_train <= INT32_MAX &&
        F <= INT32_MAX) {
      const size_t need = score_workspace_need(n_q, n_train, F, dtype == DATTRI_BF16 ? 2 : 4,
                                               dev_precond_diag != nullptr, scores != nullptr, topk, false);
      if (need > kScratchBytes)
        return fail(DATTRI_E_UNSUPPORTED,
                    "this call needs %zu bytes of scratch; the allocation-free entry point holds %zu",
                    need, kScratchBytes);
    }
  }
  void* ws = nullptr;
  dattri_status st = scratch_address(&ws);
  if (st != DATTRI_OK) return st;
  return score_impl(phi_q, n_q, ld_q, phi_train, n_train, ld_train, F, dtype, dev_precond_diag, scores, topk,
                    topk_idx, topk_val, ws, kScratchBytes, stream, false);
}
