// Internal interface between the host runtime (runtime.cpp) and the HIP
// kernels (*.hip).  Plain descriptors uploaded into the caller's workspace and
// launcher prototypes; nothing here is part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dattri {

// ---------------------------------------------------------------- layout
// Projection maps live on the device in a fragment-major layout: the d x k map
// is cut into k-blocks of KROWS rows and 16-column tiles; fragment (kb, nt) is
// 64 lanes x 16 bytes, lane l = 16*g + n holding the EPL consecutive rows
// kb*KROWS + g*EPL + j (j < EPL) of column nt*16 + n.  One wave reads one
// fragment with a single coalesced 1 KiB load, already in MFMA operand order.
//   bf16: EPL = 8, KROWS = 32 (operand of v_mfma_f32_16x16x32_bf16)
//   f32 : EPL = 4, KROWS = 16 (four v_mfma_f32_16x16x4f32, one per element)
constexpr int kFragBytes = 1024;
inline int epl_of(int elt_bytes) { return elt_bytes == 2 ? 8 : 4; }
inline int krows_of(int elt_bytes) { return 4 * epl_of(elt_bytes); }
inline int64_t packed_bytes(int d, int k, int elt_bytes) {
  const int64_t kb = (d + krows_of(elt_bytes) - 1) / krows_of(elt_bytes);
  const int64_t nt = (k + 15) / 16;
  return kb * nt * kFragBytes;
}
inline int64_t packed_offset(int v, int c, int k, int elt_bytes) {
  const int epl = epl_of(elt_bytes), kr = krows_of(elt_bytes);
  const int64_t nt_all = (k + 15) / 16;
  const int kb = v / kr, w = v % kr, g = w / epl, j = w % epl;
  const int nt = c / 16, n = c % 16, lane = 16 * g + n;
  return ((kb * nt_all + nt) * 64 + lane) * 16 + (int64_t)j * elt_bytes;
}

// ------------------------------------------------------- factored route
constexpr int kMaxGroupTiles = 8;   // input-side 16-column tiles per group
constexpr int kMaxMemberBTiles = 4; // output-side 16-column tiles per layer
constexpr int kWaves = 4;           // waves per workgroup (256 threads)

struct FactGroup {                  // layers sharing one input block A
  const void* A;                    // [n, T, d_in]
  const int32_t* lengths;           // [n] or null
  int32_t d_in, T, n;
  int32_t n_chunks, chunk_rows;     // token chunks per example
  int32_t n_members, member0;       // members: FactMember[member0 ...]
  int32_t na;                       // input-side tiles in use (<= 8)
  int32_t aligned;                  // 16-byte vector loads allowed
  int32_t pad0;
  const void* ptile[kMaxGroupTiles];    // packed P_in of the tile's layer
  int32_t ptile_local[kMaxGroupTiles];  // tile index inside that P_in
  int32_t ptile_nt[kMaxGroupTiles];     // 16-col tiles of that P_in
};

struct FactMember {                 // one layer of a group
  const void* B;                    // [n, T, d_out]
  const void* P_out;                // packed [d_out x k_out]
  int32_t d_out, k_in, k_out;
  int32_t a_tile0, na, nb;          // its input tiles [a_tile0, a_tile0+na), output tiles
  int32_t aligned, pad0;
  int64_t partial_base;             // float offset of (example 0, part 0)
  // When not null, the kernel also stores the layer's projected token rows
  // (float32 [n][T][k_in] and [n][T][k_out]; rows past an example's length
  // are not written) for the curvature fit.
  float* rows_a;
  float* rows_b;
};

struct FactItem { int32_t group, example, chunk, pad; };

// Partial blocks Psi (padded na*16 x nb*16 float32, row-major) are summed in a
// fixed order by the reduce kernel, which writes phi.
struct ReduceTask {
  int64_t partial_base;             // float offset of (example 0, part 0)
  int64_t phi_offset;               // column of the layer block in phi
  int32_t n_parts;                  // partial blocks per example
  int32_t k_in, k_out, ldp;         // ldp = nb*16 (row stride of a partial)
  int32_t part_floats;              // na*16*nb*16
  int32_t ex_begin;                 // first example of this task's rows
  int32_t pad0, pad1;
};

// Items with example < 0 are padding (the workgroup exits at once); they keep
// the XCD-interleaved order exact.
hipError_t launch_factored(int elt_bytes, int na, int nb, int aligned, const FactItem* items,
                           int n_items, const FactGroup* groups, const FactMember* members,
                           float* partials, hipStream_t s);
void factored_instance(int elt_bytes, int na_req, int nb_req, int aligned, int* na_inst,
                       int* nb_inst, int* rows_per_wave);
// Whether instance (na, nb) streams factor rows through LDS by direct loads.
bool factored_direct_loads(int elt_bytes, int na, int nb, int aligned);
constexpr int kXcds = 8;  // MI355X: workgroup i is dispatched to XCD i mod 8

// max_out: the largest k_in*k_out over the tasks (sets the grid's z extent)
hipError_t launch_reduce(const ReduceTask* tasks, int n_tasks, int n_examples, int max_out,
                         const float* partials, void* phi, int phi_bf16, int64_t ld_phi,
                         hipStream_t s);

// ------------------------------------------- factored route, split form
// For captures where the fused kernel has too few work items: stage 1
// projects the token rows of every factor block (all examples flattened,
// n*T rows) slab by slab over the feature dimension d, writing float32
// partial projections [slab][row][tile cols]; stage 2 sums the slabs and
// contracts each example's tokens into its layer block of phi.
// Rows per stage-1 workgroup of the instance with nt_inst tiles: 4 waves of
// 4 row tiles (2 at 8 tiles, where 4 would not fit the register file).
constexpr int split_rt_of(int nt_inst) { return nt_inst <= 4 ? 4 : 2; }
constexpr int split_rows_of(int nt_inst) { return 4 * split_rt_of(nt_inst) * 16; }
constexpr int kSplitSlabQuantum = 128;  // slab widths are multiples of this
struct SplitOp {                    // one factor block: a group's A or a member's B
  const void* X;                    // [rows, ld] row-major
  int32_t rows, ld;                 // n*T, d
  int32_t slab_cols, n_slabs;
  int32_t nt;                       // 16-column tiles of the projected rows
  int32_t aligned;                  // 16-byte vector loads allowed
  int64_t out_base;                 // float offset of [slab 0][row 0][col 0]
  const void* ptile[kMaxGroupTiles];    // packed map holding tile t
  int32_t ptile_local[kMaxGroupTiles];  // tile index inside that map
  int32_t ptile_nt[kMaxGroupTiles];     // 16-col tiles of that map
};
struct SplitItem { int32_t op, row_block, slab, pad; };
struct ContractTask {               // one layer
  int64_t a_base, b_base;           // out_base of its A op and B op
  int32_t a_ld, b_ld;               // floats per projected row of each op
  int32_t a_col0;                   // first column of this layer's tiles in the A op
  int32_t a_slabs, b_slabs;
  int32_t k_in, k_out, T, rows;     // rows = n*T (the slab stride in rows)
  int32_t tok_chunk, n_tchunks;     // tokens per workgroup, chunks per example
  int32_t pad0;
  int64_t phi_offset;               // used when n_tchunks == 1 (phi written directly)
  int64_t partial_base;             // else: float offset of [example][chunk][ki16 x ko16]
  const int32_t* lengths;           // [n] or null
};
// One launch per instance (elt, aligned, tiles); items of that instance only.
hipError_t launch_split_project(int elt_bytes, int aligned, int nt, const SplitItem* items,
                                int n_items, const SplitOp* ops, float* out, hipStream_t s);
int split_nt_instance(int nt_req);  // tiles of the instance that serves nt_req tiles
// In-place sum of a stage-1 op's slabs into slab 0 (slab order).
struct SlabSumTask {
  int64_t base;                     // float offset of slab 0 (16-byte aligned)
  int64_t n4;                       // float4s per slab
  int64_t stride4;                  // float4s between slabs
  int32_t n_slabs, pad0;
};
hipError_t launch_slab_sum(const SlabSumTask* tasks, int n_tasks, int64_t max_n4, float* out,
                           hipStream_t s);
// Grid (max_tchunks, n_examples, n_tasks); chunks past a task's n_tchunks exit.
hipError_t launch_split_contract(const ContractTask* tasks, int n_tasks, int n_examples,
                                 int max_tchunks, const float* proj, float* partials, void* phi,
                                 int phi_bf16, int64_t ld_phi, hipStream_t s);

// ---------------------------------------------------- materialized route
struct GradArgs {
  const void* A; const void* B; const int32_t* lengths;
  int32_t d_in, d_out, T, ex_begin, ex_count, aligned;
  float* G;                         // [ex_count, d_out, d_in]
};
hipError_t launch_gradient(int elt_bytes, const GradArgs& a, hipStream_t s);
// bf16 with 16-byte aligned rows (A, B bases and d_in, d_out multiples of 8): the
// LDS-transpose kernel; launch_gradient dispatches to it.
hipError_t launch_gradient_tr(const GradArgs& a, hipStream_t s);

struct GProjArgs {
  const float* G;                   // [ex_count, d_out, d_in]
  const void* P_in; const void* P_out;  // packed
  int32_t d_in, d_out, k_in, k_out, ex_count;
  int32_t n_ublocks;                // row blocks of kGProjRows rows of G
  int32_t n_ksplit, kb_per_split;   // d_in split into n_ksplit ranges of k-blocks
  float* partials;                  // [ex_count][n_ublocks * n_ksplit][na*16 x nb*16]
};
constexpr int kGProjRows = 128;     // rows of G per workgroup (4 waves x 2 row tiles)
constexpr int kGProjMaxTilesIn = 8; // input tiles per pass (larger k_in loops)
hipError_t launch_gproject(int elt_bytes, const GProjArgs& a, hipStream_t s);

// Fused materialized route (bf16, 16-byte aligned rows, k_in <= 128): each
// workgroup forms 128 rows of G over one token chunk, 128 columns at a time,
// and projects every tile from its accumulators, so G never goes to memory.
struct GFusedArgs {
  const void* A; const void* B; const int32_t* lengths;
  const void* P_in; const void* P_out;  // packed bf16
  int32_t d_in, d_out, T, k_in, k_out;
  int32_t ex_begin, ex_count;
  int32_t n_ublocks;                // row blocks of kGFusedRows rows of G
  int32_t n_vsplit, vt_per_split;   // 128-column tiles of G in n_vsplit ranges of vt_per_split
  int32_t n_tchunks, tok_chunk;     // token chunks per example (tok_chunk a multiple of 32)
  float* partials;                  // [ex_count][n_ublocks * n_vsplit * n_tchunks][na*16 x nb*16]
};
constexpr int kGFusedCols = 128;    // columns of G per tile
constexpr int kGFusedRows = 128;
constexpr int kGFusedMaxTilesIn = 8;
int gfused_tiles_in(int k_in);      // 16-column tiles of k_in the kernel instance serving k_in holds
int gfused_wgs_per_cu(int k_in);    // workgroups of that instance one CU holds
hipError_t launch_gfused(const GFusedArgs& a, hipStream_t s);

// ------------------------------------------------------ cross-Gram matrices
// One layer of the factorized route between batch 1 (n1 examples) and batch 2
// (n2 examples): factor blocks [n, T, d] row-major, token rows padded to
// Tp = T rounded up to 16 on the flattened token axes.
struct GhostEntry {
  const void* A1; const void* B1; const int32_t* len1;
  const void* A2; const void* B2; const int32_t* len2;
  int32_t d_in, d_out, n1, n2, T1, T2, Tp1, Tp2;
  int32_t nbr, nbc;                 // 16 x 16 blocks: n1*Tp1/16 rows, n2*Tp2/16 columns
  int32_t aligned;                  // rows and bases 16-byte aligned (vector loads)
  int32_t out0;                     // output row of its pair (i, j) is out0 + i
  int64_t part_off;                 // float offset of its block sums (nbr x nbc)
  int32_t dma;                      // bf16, aligned, and a tile's rows within 32-bit byte offsets:
                                    // token rows streamed into LDS by direct loads
  int32_t pad0;
};
struct GhostTile { int32_t entry, rt, ct, pad0; };  // 128 x 128 tile of an entry
constexpr int kGhostTile = 128;
hipError_t launch_ghost(int elt_bytes, const GhostEntry* entries, const GhostTile* tiles, int n_tiles,
                        float* parts, hipStream_t s);
// K[I*ld + J] (=, or += with accumulate) the sum over entries, in order, of the
// block sums of segment (I - out0, J) of every entry that has that pair; diag:
// K[I] from segments (I - out0, I - out0).  Cells: n_rows x n_cols (diag: n_rows).
hipError_t launch_ghost_reduce(const GhostEntry* entries, int n_entries, const float* parts,
                               int n_rows, int n_cols, float* K, int64_t ld, int diag, int accumulate,
                               hipStream_t s);
// One-pass materialized cross-Gram (bf16 blocks with 16-byte aligned rows),
// every one-pass layer of a call in one launch.  Layer e owns the nslots =
// (n_ub n_vt rounded up to 8) workgroup slots slot0 .. slot0 + nslots - 1 of
// grid x; grid y = examples j of batch b, grid z = runs of ipw examples of
// batch a.  parts[slot][i][j] (diag: parts[slot][i], the squared norms of
// batch a) = sum over the slot's 128 x 128 tile of DW_a[i0 + i] * DW_b[j0 + j]
// (0 for the padding slots).
constexpr int kXOneTile = 128;
struct XOneEntry {
  const void *A1, *B1, *A2, *B2;  // batch a and b factor blocks [n, T, d]
  const int32_t *len1, *len2;     // per-example lengths or NULL
  int32_t d_in, d_out, T1, T2;
  int32_t n_ub, n_vt;             // 128-row tiles of d_out, 128-column tiles of d_in
  int32_t slot0, nslots;          // its workgroup slots (nslots a multiple of 8)
};
struct XOneArgs {
  const XOneEntry* entries;
  const int32_t* slot_entry;      // entry of every slot
  int32_t n_slots;
  int32_t i0, ci, ipw;            // batch a examples i0 .. i0 + ci - 1, ipw per workgroup
  int32_t j0, cj;                 // batch b examples j0 .. j0 + cj - 1 (unused for diag)
  int32_t diag;
  float* parts;
};
hipError_t launch_xone(const XOneArgs& a, hipStream_t s);

// parts[c][i][j] (diag: parts[c][i]) = Frobenius product over chunk c of the
// flattened gradients G1[i], G2[j] (D floats each); chunk a multiple of 64
hipError_t launch_gdot(const float* G1, int n1, const float* G2, int n2, int64_t D, int64_t chunk,
                       int diag, float* parts, hipStream_t s);
// K[(r0+i)*ld + c0+j] (diag: K[r0+i]) = or += the sum over chunks of parts
hipError_t launch_kacc(const float* parts, int nchunks, int n1, int n2, float* K, int64_t ld, int r0,
                       int c0, int diag, int accumulate, hipStream_t s);
hipError_t launch_fill_rows(float* K, int rows, int cols, int64_t ld, hipStream_t s);

// ---------------------------------------------------------- random masks
// A mask layer keeps m entries (r_e, c_e) of DW, gathered from the factors:
// out[e] = sum_t B[t][r_e] A[t][c_e].  Work item = (task, example, token
// chunk, group of up to kMaskGroup entries); token rows of A and B are staged
// in LDS `stage_tokens` at a time (contiguous rows, moved as one block; two
// stage buffers of [A rows | B rows], each part rounded up to 1 KiB) and
// every thread sums the products of its entries; each item writes its entries'
// partial sums at partial_base + ((example * n_chunks + chunk) * m + entry),
// summed over chunks by the reduce kernel.
constexpr int kMaskPerThread = 64;
constexpr int kMaskGroup = 256 * kMaskPerThread;   // entries per work item
constexpr int64_t kMaskStageBudget = 40 * 1024;   // bytes of one stage (two stages per work item)
// Fixed-slot gather (bf16, 16-byte rows, whole groups whose A and B slices are
// at most kMaskSlot bytes): every stage holds kMaskSlotPairs token pairs, each
// side's slice as a row of bf16 pairs at a fixed offset.  LDS: 2 buffers of
// kMaskSlotPairs x [A pair row | B pair row], one workgroup per CU.
constexpr int kMaskSlot = 8192;
constexpr int kMaskSlotPairs = 2;
constexpr size_t kMaskSlotLds = (size_t)2 * kMaskSlotPairs * 2 * (2 * kMaskSlot);
// Byte offset of slice feature f in a fixed-slot pair row: 16-byte chunk
// g = f / 4 (four pairs) goes to half g % 2 (kMaskSlot bytes each) at
// 16 (g / 2), so the chunks 2k, 2k + 1 that one thread stages land in the two
// halves at 16 k and a wave's write of either is 1 KiB in a row (no bank
// conflicts).  Its 4-byte word falls in LDS bank (4 (f / 8) + f % 4) mod 32.
constexpr uint32_t mask_pair_offset(uint32_t f) {
  return ((f >> 2) & 1u) * (uint32_t)kMaskSlot + 16u * (f >> 3) + 4u * (f & 3u);
}
// whether a mask layer's whole groups qualify (slices: 4 per group, as in its table)
bool mask_fixed_layout(int elt, int d_in, int d_out, int m, const int32_t* slices);
struct MaskTask {
  const void* A; const void* B;      // [n, T, d_in], [n, T, d_out]
  const int32_t* lengths;            // [n] or null
  const int32_t* rows;               // [m] output feature of the entry in each slot
  const int32_t* cols;               // [m] input feature of the entry in each slot
  const int32_t* pos;                // [m] index of that entry in mask order
  const int32_t* slices;             // [4 per group] A slice (first byte, bytes), B slice (first byte, bytes)
  int32_t d_in, d_out, T, m;
  int32_t stage_tokens, chunk_tokens, n_chunks, aligned;  // aligned: 16-byte row blocks
  int32_t fixed, pad0;               // whole groups take the fixed-slot gather
  int64_t partial_base;
};
struct MaskItem { int32_t task, example, chunk, group; };  // task < 0: padding
// full: every item's group holds kMaskGroup entries; b16: bf16 layers with
// d_in, d_out <= 32768 only (entries as byte offsets, v_dot2_f32_bf16 gather)
hipError_t launch_mask(int elt_bytes, int aligned, int full, int b16, const MaskItem* items, int n_items,
                       const MaskTask* tasks, size_t lds_bytes, float* partials, hipStream_t s);
// whole groups of fixed-slot tasks (bf16, aligned), kMaskSlotLds bytes of LDS
hipError_t launch_mask_fixed(const MaskItem* items, int n_items, const MaskTask* tasks, float* partials,
                             hipStream_t s);

// ---------------------------------------------------------------- scoring
// dst rows ld_dst apart receive src rows (ld_src apart) times d, first F columns
hipError_t launch_scale_rows(int elt_bytes, const void* src, int64_t ld_src, const float* d,
                             void* dst, int64_t ld_dst, int64_t rows, int64_t F, hipStream_t s);
// partials: workspace of score_partial_floats(...) floats (may be null when 0)
// S = (Q diag(d)) X^T (d may be null): Q rows ldq elements apart, X rows ldx
// apart (both >= F, multiples of 16 bytes).  qws: workspace of
// score_query_ws_bytes(...) bytes for the prepared queries (ld_ws = row stride
// of the row-major form the small kernels use); partials: workspace of
// score_partial_floats(...) floats (may be null when 0).
hipError_t launch_score_gemm(int elt_bytes, const void* Q, int64_t ldq, const float* d, const void* X,
                             int64_t ldx, float* S, int64_t n_q, int64_t n_train, int64_t F,
                             void* qws, int64_t ld_ws, float* partials, hipStream_t s);
// bf16 problems at least this large (n_q * n_train) use the 256 x 256 kernel
constexpr int64_t kBigGemmMin = (int64_t)1 << 20;
inline bool score_uses_big(int elt_bytes, int64_t n_q, int64_t n_train) {
  return elt_bytes == 2 && n_q * n_train >= kBigGemmMin;
}
// bytes of queries packed in MFMA fragment order for the 256 x 256 kernel
int64_t score_qpack_bytes(int64_t n_q, int64_t F);
// Both GEMM kernels split K when their tiles alone would leave CUs idle:
// number of K splits (1 = none) and the float32 partial results it stages.
int score_ksplit(int elt_bytes, int64_t n_q, int64_t n_train, int64_t F);
// S[i] = sum over y < ks of part[y*n + i], in split order.
hipError_t launch_splitk_sum(const float* part, int ks, int64_t n, float* S, hipStream_t s);
inline int64_t score_partial_floats(int elt_bytes, int64_t n_q, int64_t n_train, int64_t F) {
  const int ks = score_ksplit(elt_bytes, n_q, n_train, F);
  return ks > 1 ? (int64_t)ks * n_q * n_train : 0;
}
// Packs (and scales by d, when given) the queries into qpack, then runs the
// 256 x 256 GEMM.
hipError_t launch_score_gemm_256(const void* Q, int64_t ldq, const float* d, const void* X,
                                 int64_t ldx, float* S, int64_t n_q, int64_t n_train, int64_t F,
                                 void* qpack, float* partials, hipStream_t s);
// Cosine scores: inv_q / inv_t receive 1 / row norms (queries times d when
// given; 0 for zero rows), then S[q][j] *= inv_q[q] * inv_t[j].
hipError_t launch_cosine_scale(int elt_bytes, const void* Q, int64_t ldq, const float* d, const void* X,
                               int64_t ldx, float* S, int64_t n_q, int64_t n_train, int64_t F, float* inv_q,
                               float* inv_t, hipStream_t s);
constexpr int kTopkMax = 1024;
hipError_t launch_topk(const float* S, int64_t n_q, int64_t n_train, int32_t k, int32_t* idx,
                       float* val, hipStream_t s);

// ---------------------------------------------------- K-FAC / EK-FAC curvature
constexpr int kCurvMaxK = 64;       // k_in, k_out limit of the curvature kernels

// Factor sums: one op per layer side (X = A with P_in, or X = B with P_out).
// Work item = a run of consecutive units u = example * n_chunks + chunk of one
// op; each wave of the item writes one partial (nt*16)^2 float32 sum.
struct FsumOp {
  const void* X;                    // [n, T, d]
  const int32_t* lengths;           // [n] or null
  const void* P;                    // packed [d x k] map
  int32_t d, T, n, nt;              // nt = 16-column tiles of the map
  int32_t chunk_rows, n_chunks, aligned, pad0;
  int64_t partial_base;             // float offset of the op's first partial
};
struct FsumItem { int32_t op, unit0, n_units, part; };  // n_units 0: padding item
// One launch per instance (elt, aligned, tiles); rows per wave from fsum_rt.
hipError_t launch_fsum(int elt_bytes, int aligned, int nt, const FsumItem* items, int n_items,
                       const FsumOp* ops, float* partials, hipStream_t s);
int fsum_nt_instance(int nt_req);   // tiles of the instance serving nt_req tiles
int fsum_rows_per_wave(int nt_inst);

// dst (float32 [rows][cols] at byte offset dst_off of the state) += the sum,
// in part order, of n_parts partials [rows][ldp] part_floats apart; one counter
// (int64 at count_off, if >= 0) += sum of lengths clamped to [0, T] over n
// entries, or count_add when lengths is null.
struct StatTask {
  int64_t part_base, dst_off, count_off, count_add;
  const int32_t* lengths;
  int32_t n_parts, part_floats, ldp, rows, cols, n_len, T, pad0;
};
hipError_t launch_stat_reduce(const StatTask* tasks, int n_tasks, int max_out, const float* parts,
                              uint8_t* state, hipStream_t s);

// Sums of outer products of stored projected token rows: for example i of an
// op, rows t < min(lengths[i], T) at rows + (i*T + t)*ld + col0, k columns.
// Work item (item, op) covers examples [item*ex_per_item, ...) and writes one
// k x k partial at partial_base + item*k*k.
struct RowOp {
  const float* rows;
  const int32_t* lengths;
  int64_t ld, partial_base;
  int32_t col0, k, T, n, ex_per_item, n_items;
};
hipError_t launch_rowcov(const RowOp* ops, int n_ops, int max_items, float* parts, hipStream_t s);

// Token-level scores: per layer, where its projected token rows sit (float32,
// row (i*T + t) at rows + (i*T + t)*ld + col0) and where its block sits in the
// query rows.  out[q][i][t] = sum over layers of a~_t^T R_q g~_t for t below
// the layer's length of example i.
struct TokTask {
  const float* a_rows; const float* b_rows;
  const int32_t* lengths;
  int64_t a_ld, b_ld, q_off;
  int32_t a_col0, b_col0, k_in, k_out;
};
constexpr int kTokTokens = 128;  // token positions per workgroup (32 per wave)
constexpr int kTokQueries = 4;   // queries per workgroup
hipError_t launch_token_scores(const TokTask* tasks, int n_tasks, const void* phi_q, int q_bf16, int64_t ld_q,
                               int64_t n_q, int64_t n, int T, float* out, hipStream_t s);

// Symmetric eigendecomposition of sum / count (k x k, k <= kCurvMaxK).
struct EigTask { int64_t sum_off, count_off, q_off, lam_off; int32_t k, pad0; };
hipError_t launch_eigen(const EigTask* tasks, int n_tasks, uint8_t* state, hipStream_t s);

// Rotated-block kernels: per layer, the block of phi at column col and the
// layer's fields in the state.
struct RotTask {
  int64_t col;                      // first column of the layer block in phi
  int64_t q_a, lam_a, q_g, lam_g, sum_e, counts;  // state byte offsets
  int64_t part_base;                // EK-FAC: float offset of the layer's partials
  int32_t k_in, k_out, n_blocks, pad0;
};
// parts[part_base + b*k_in*k_out ...] = sum over rows [b*rows_per_block, ...)
// of (Q_A^T Psi Q_G)^2; grid (max_blocks, n_tasks).
hipError_t launch_ekfac(const RotTask* tasks, int n_tasks, int max_blocks, const uint8_t* state,
                        const void* phi, int phi_bf16, int64_t ld, int64_t n, int rows_per_block,
                        float* parts, hipStream_t s);
// out rows = P(Psi_q) per layer; kind 0 K-FAC, 1 EK-FAC.
hipError_t launch_precondition(const RotTask* tasks, int n_tasks, const uint8_t* state, int kind,
                               double rel, double abs_, const void* phi_q, int in_bf16,
                               int64_t ld_q, int64_t n_q, void* out, int out_bf16, int64_t ld_out,
                               hipStream_t s);
// Zero `bytes` bytes (a multiple of 16, 16-byte aligned) with a fill kernel.
hipError_t launch_zero(void* p, int64_t bytes, hipStream_t s);

}  // namespace dattri
