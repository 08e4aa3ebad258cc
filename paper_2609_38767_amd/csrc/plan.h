// Launch plan of the projection (all three kernel forms), shared by the
// projection entry point and the curvature fit that runs the projection with
// projected token rows kept.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <memory>
#include <vector>

#include "context.h"
#include "dattri.h"
#include "internal.h"

namespace dattri {

struct MatChunk {
  int layer, ex_begin, ex_count, n_ublocks, n_ksplit, kb_per_split, task;
  int fused = 0;                    // one-pass kernel (G on chip): its launch shape below
  int n_tchunks = 1, tok_chunk = 0, n_vsplit = 1, vt_per_split = 1;
};

// Where the projected token rows of one layer side sit after the projection
// ran with rows kept: byte offset in the workspace, floats per row, first
// column of the layer's k columns.
struct RowSrc { int layer, side; size_t off; int64_t ld; int col0; };

struct Plan {
  // host-side descriptors (device pointers inside)
  std::vector<FactItem> items;
  std::vector<FactGroup> groups;
  std::vector<FactMember> members;
  std::vector<ReduceTask> tasks;  // factored tasks first, then one per MatChunk
  int n_fact_tasks = 0;
  int fact_max_out = 0;            // largest k_in*k_out over the factored tasks
  struct Launch { int elt, na, nb, aligned, first, count; };
  std::vector<Launch> launches;
  std::vector<MatChunk> mat;
  // split form of the factored route (captures with few fused work items)
  std::vector<SplitOp> sops;
  std::vector<SplitItem> sitems;
  std::vector<ContractTask> ctasks;
  struct SplitLaunch { int elt, aligned, nt, first, count; };
  std::vector<SplitLaunch> slaunches;
  std::vector<ReduceTask> stasks;  // token-chunked contractions to reduce
  std::vector<SlabSumTask> slabsum;
  int64_t slabsum_max_n4 = 0;
  int split_max_tchunks = 0, split_max_out = 0;
  // mask layers (gathered DW entries)
  std::vector<MaskTask> mtasks;
  std::vector<MaskItem> mitems;
  // full: every item a whole entry group; fixed: the fixed-slot gather
  struct MaskLaunch { int aligned, full, fixed, first, count; };
  std::vector<MaskLaunch> mlaunches;
  std::vector<ReduceTask> mreduce;
  int mask_max_out = 0;
  size_t mask_lds = 0;
  bool mask_b16 = true;  // every mask layer bf16 with d_in, d_out <= 32768 (byte-offset gather)
  // projected token rows kept for the curvature fit (rows = true)
  bool rows = false;
  std::vector<size_t> member_rows;  // per fused member: byte offsets of its A rows, B rows (pairs)
  std::vector<RowSrc> row_srcs;     // every factored layer side
  std::vector<int> mat_layers;      // layers on the materialized route (no projected rows)
  // workspace layout (byte offsets)
  size_t off_items = 0, off_groups = 0, off_members = 0, off_tasks = 0;
  size_t off_sops = 0, off_sitems = 0, off_ctasks = 0, off_stasks = 0, off_slabsum = 0;
  size_t blob_bytes = 0;
  size_t off_fpart = 0, fpart_bytes = 0, off_g = 0, g_bytes = 0, off_mpart = 0, mpart_bytes = 0;
  size_t off_proj = 0, proj_bytes = 0, off_spart = 0, spart_bytes = 0;
  size_t off_rows = 0, rows_bytes = 0;
  size_t off_mtasks = 0, off_mitems = 0, off_mreduce = 0, off_maskpart = 0, maskpart_bytes = 0;
  size_t total = 0;
};

// Plans the projection of the current captures (route forced or AUTO); with
// `rows`, fused factored members also keep their projected token rows in the
// workspace and row_srcs lists where every factored layer side's rows sit.
dattri_status build_plan(const dattri_ctx* ctx, dattri_route forced, Plan& P, bool rows);
// The same plan, reused when the context state it depends on (layer sizes,
// captures, bound maps, factored form, cost model) and the arguments equal
// those of a recent call; otherwise built and remembered.
dattri_status get_plan(const dattri_ctx* ctx, dattri_route forced, bool rows, std::shared_ptr<const Plan>* out);

// Puts a launch table on the device.  With a plan buffer bound that can hold
// it, the table goes to its kind's slot there, and no copy is issued when that
// slot already holds the same bytes; otherwise it is copied to `fallback` (the
// head of the call's workspace).  *dev receives the table's device address.
hipError_t place_table(const dattri_ctx* ctx, TableKind kind, const std::vector<uint8_t>& blob,
                       uint8_t* fallback, hipStream_t s, uint8_t** dev);
// Validates phi / workspace arguments against a plan, uploads its descriptors
// and launches every kernel.  n = the captures' example count.
dattri_status run_plan(dattri_ctx* ctx, const Plan& P, void* phi, dattri_dtype phi_dtype, int64_t ld_phi,
                       void* workspace, size_t ws_bytes, hipStream_t s);

}  // namespace dattri
