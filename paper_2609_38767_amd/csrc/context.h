// Library context (host side): registered layers with their projection maps
// and captured factor blocks, the route cost models, and the host copy of the
// last uploaded launch plan.  Shared by the translation units of the C ABI.
#pragma once

#include <stdint.h>

#include <memory>
#include <utility>
#include <vector>

#include "dattri.h"

namespace dattri {

struct Plan;

// Kinds of launch tables a call uploads; each has at most one slot in the
// context's bound plan buffer.
enum TableKind { kTabProj = 0, kTabFit, kTabFsum, kTabEkfac, kTabTok, kTabCross, kTabKinds };

// One launch table resident in the bound plan buffer: where it sits, how much
// room it has and the bytes last copied there.
struct TableSlot {
  int kind = -1;
  size_t off = 0, cap = 0;
  std::vector<uint8_t> bytes;
};

struct Layer {
  int32_t d_in = 0, d_out = 0, k_in = 0, k_out = 0;
  int64_t offset = 0;  // first column of the layer's block in phi
  void* P_in = nullptr;
  void* P_out = nullptr;
  bool bound = false;
  int32_t map_kind = 0;  // dattri_map_kind of the seeded maps
  // mask layer when mask_size > 0: masks mask_id .. mask_id + mask_count - 1 of
  // mask_size entries each, back to back (k_in = 1, k_out = mask_size * mask_count)
  int32_t mask_size = 0, mask_id = 0, mask_count = 0;
  std::vector<int32_t> mask_slices;  // bound mask layer: the entry groups' row slices (as in its table)
  std::vector<float> override_in, override_out;  // rounded values when overridden
  const void* A = nullptr;  // captured [n, T, d_in]
  const void* B = nullptr;  // captured [n, T, d_out]
  int32_t n = 0, T = 0;
  const int32_t* lengths = nullptr;
  bool captured = false;
};

}  // namespace dattri

struct dattri_ctx {
  dattri_dtype dtype;
  int elt;
  uint64_t seed;
  std::vector<dattri::Layer> layers;
  int64_t F = 0;
  dattri_cost_model cost;
  dattri_crossgram_cost_model xcost;
  dattri_factored_form form = DATTRI_FORM_AUTO;
  // host copy of the last launch table copied into a workspace (fallback
  // path: no plan buffer bound, or a table larger than it); kept until the
  // next such copy
  mutable std::vector<uint8_t> blob;
  // caller-bound device buffer holding launch tables between calls
  // (dattri_bind_plan_buffer) and the tables resident in it
  uint8_t* plan_buf = nullptr;
  size_t plan_cap = 0;
  mutable std::vector<dattri::TableSlot> slots;
  mutable size_t slots_used = 0;
  // projection plans of recent calls with the context state each was built
  // from (captures, maps, route, form, cost model): an equal state reuses it
  mutable std::vector<std::pair<std::vector<uint64_t>, std::shared_ptr<const dattri::Plan>>> plans;
  mutable std::pair<std::vector<uint64_t>, std::vector<dattri_route>> route_cache;  // call_routes(AUTO)
};
