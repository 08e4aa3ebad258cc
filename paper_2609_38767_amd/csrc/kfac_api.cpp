// C ABI of K-FAC / EK-FAC curvature on projected factors (Sec. 3.2: the
// preconditioned comparisons of K-FAC and EK-FAC on factorized gradients;
// App. A.2: the Kronecker-factored statistics apply unchanged to the projected
// pair; App. B: damping of 0.1 times the mean eigenvalue of each layer):
// state layout, validation, launch planning and execution.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "api_common.h"
#include "context.h"
#include "dattri.h"
#include "internal.h"
#include "plan.h"

using namespace dattri;

namespace {

inline int tiles16(int k) { return (k + 15) / 16; }
inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

constexpr int64_t kFsumTargetItems = 2048;   // factor-sum workgroups aimed for
constexpr int64_t kEkfacTargetBlocks = 2048; // EK-FAC workgroups aimed for
constexpr int kFsumChunkRows = 512;          // token rows per unit (rounded to a sub-chunk)

// Per-layer fields, then the descriptor tables the eigen and precondition
// kernels read (rewritten by each call that launches them).
struct CurvLayout {
  std::vector<dattri_curvature_layout> L;
  size_t off_eig = 0, off_rot = 0, total = 0;
};

dattri_status check_layers(const dattri_ctx* ctx) {
  if (!ctx) return fail(DATTRI_E_INVALID_ARG, "ctx is NULL");
  if (ctx->layers.empty()) return fail(DATTRI_E_STATE, "no layer registered");
  for (size_t l = 0; l < ctx->layers.size(); ++l) {
    const Layer& L = ctx->layers[l];
    if (L.mask_size > 0)
      return fail(DATTRI_E_UNSUPPORTED, "layer %zu is a mask layer: curvature needs the projected factors", l);
    if (L.k_in > kCurvMaxK || L.k_out > kCurvMaxK)
      return fail(DATTRI_E_UNSUPPORTED, "layer %zu: curvature needs k_in, k_out <= %d (got %d, %d)", l,
                  kCurvMaxK, L.k_in, L.k_out);
  }
  return DATTRI_OK;
}

void curv_layout(const dattri_ctx* ctx, CurvLayout& C) {
  size_t off = 0;
  C.L.resize(ctx->layers.size());
  for (size_t l = 0; l < ctx->layers.size(); ++l) {
    const size_t ki = ctx->layers[l].k_in, ko = ctx->layers[l].k_out;
    dattri_curvature_layout& f = C.L[l];
    f.sum_a = (int64_t)off; off = align_up(off + 4 * ki * ki);
    f.sum_g = (int64_t)off; off = align_up(off + 4 * ko * ko);
    f.sum_e = (int64_t)off; off = align_up(off + 4 * ki * ko);
    f.q_a = (int64_t)off;   off = align_up(off + 4 * ki * ki);
    f.lam_a = (int64_t)off; off = align_up(off + 4 * ki);
    f.q_g = (int64_t)off;   off = align_up(off + 4 * ko * ko);
    f.lam_g = (int64_t)off; off = align_up(off + 4 * ko);
    f.counts = (int64_t)off; off = align_up(off + 3 * 8);
  }
  C.off_eig = off;
  off = align_up(off + 2 * ctx->layers.size() * sizeof(EigTask));
  C.off_rot = off;
  off = align_up(off + ctx->layers.size() * sizeof(RotTask));
  C.total = off;
}

std::vector<RotTask> rot_tasks(const dattri_ctx* ctx, const CurvLayout& C) {
  std::vector<RotTask> R(ctx->layers.size());
  for (size_t l = 0; l < ctx->layers.size(); ++l) {
    const Layer& L = ctx->layers[l];
    const dattri_curvature_layout& f = C.L[l];
    RotTask& t = R[l];
    std::memset(&t, 0, sizeof(t));
    t.col = L.offset;
    t.q_a = f.q_a;
    t.lam_a = f.lam_a;
    t.q_g = f.q_g;
    t.lam_g = f.lam_g;
    t.sum_e = f.sum_e;
    t.counts = f.counts;
    t.k_in = L.k_in;
    t.k_out = L.k_out;
  }
  return R;
}

// Reduction of one layer side's factor sums into the state: destination,
// counter (A side: token rows, from the lengths when given; B side: examples)
// and size; the caller fills in the partial layout.
StatTask side_task(const dattri_ctx* ctx, const CurvLayout& C, int l, int side, int32_t n) {
  const Layer& L = ctx->layers[l];
  StatTask t;
  std::memset(&t, 0, sizeof(t));
  t.dst_off = side == 0 ? C.L[l].sum_a : C.L[l].sum_g;
  t.count_off = C.L[l].counts + 8 * side;
  if (side == 0 && L.lengths) {
    t.lengths = L.lengths;
    t.n_len = n;
    t.T = L.T;
  } else {
    t.count_add = side == 0 ? (int64_t)n * L.T : (int64_t)n;
  }
  t.rows = t.cols = side == 0 ? L.k_in : L.k_out;
  return t;
}

// ------------------------------------------------------ factor-sum planning
struct FsumPlan {
  std::vector<FsumOp> ops;
  std::vector<FsumItem> items;
  std::vector<StatTask> tasks;
  struct Launch { int elt, aligned, nt, first, count; };
  std::vector<Launch> launches;
  int max_out = 0;
  int32_t n = 0;
  size_t off_ops = 0, off_items = 0, off_tasks = 0, blob_bytes = 0, off_parts = 0, total = 0;
};

// Factor sums of every layer, or of the layers in `only`.
dattri_status plan_fsum(const dattri_ctx* ctx, const CurvLayout& C, FsumPlan& P,
                        const std::vector<int>* only = nullptr) {
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  int32_t n = -1;
  for (size_t l = 0; l < ctx->layers.size(); ++l) {
    const Layer& L = ctx->layers[l];
    if (!L.bound) return fail(DATTRI_E_STATE, "layer %zu: projection maps not bound", l);
    if (!L.captured) return fail(DATTRI_E_STATE, "layer %zu has no capture", l);
    if (n < 0) n = L.n;
    if (L.n != n) return fail(DATTRI_E_STATE, "layer %zu captured with n=%d but layer 0 with n=%d", l, L.n, n);
  }
  P.n = n;
  const int elt = ctx->elt;
  struct OpInfo { int inst_nt, aligned; int64_t units, unit_cost; int layer, side; };
  std::vector<OpInfo> info;
  double total_cost = 0.0;
  for (size_t l = 0; l < ctx->layers.size(); ++l) {
    if (only && std::find(only->begin(), only->end(), (int)l) == only->end()) continue;
    const Layer& L = ctx->layers[l];
    for (int side = 0; side < 2; ++side) {
      FsumOp O;
      std::memset(&O, 0, sizeof(O));
      O.X = side == 0 ? L.A : L.B;
      O.P = side == 0 ? L.P_in : L.P_out;
      O.lengths = L.lengths;
      O.d = side == 0 ? L.d_in : L.d_out;
      O.T = L.T;
      O.n = n;
      const int k = side == 0 ? L.k_in : L.k_out;
      O.nt = tiles16(k);
      O.aligned = ((uintptr_t)O.X % 16 == 0) && ((int64_t)O.d * elt) % 16 == 0;
      const int inst = fsum_nt_instance(O.nt);
      const int sub = kWaves * fsum_rows_per_wave(inst) * 16;
      int cr = std::max(sub, kFsumChunkRows / sub * sub);
      if (L.T <= cr) cr = std::max(sub, (L.T + sub - 1) / sub * sub);
      O.chunk_rows = cr;
      O.n_chunks = std::max(1, (L.T + cr - 1) / cr);
      OpInfo I{inst, O.aligned, (int64_t)n * O.n_chunks, (int64_t)cr * O.d, (int)l, side};
      total_cost += (double)I.units * I.unit_cost;
      info.push_back(I);
      P.ops.push_back(O);
    }
  }
  // work items: runs of units of one op, about kFsumTargetItems in total
  const double target = std::max(1.0, total_cost / (double)kFsumTargetItems);
  std::vector<int64_t> upi(P.ops.size()), nitems(P.ops.size());
  size_t part_floats_total = 0;
  for (size_t o = 0; o < P.ops.size(); ++o) {
    const OpInfo& I = info[o];
    upi[o] = std::min<int64_t>(std::max<int64_t>(1, (int64_t)std::llround(target / (double)I.unit_cost)),
                               std::max<int64_t>(1, I.units));
    nitems[o] = I.units > 0 ? cdiv(I.units, upi[o]) : 0;
    const int64_t kp = (int64_t)P.ops[o].nt * 16;
    P.ops[o].partial_base = (int64_t)part_floats_total;
    part_floats_total += (size_t)(nitems[o] * kWaves * kp * kp);
  }
  // reduction tasks: one per op (sum into sum_a / sum_g, counts N_tok / N)
  for (size_t o = 0; o < P.ops.size(); ++o) {
    const int l = info[o].layer, side = info[o].side;
    const int kp = P.ops[o].nt * 16;
    StatTask t = side_task(ctx, C, l, side, n);
    t.part_base = P.ops[o].partial_base;
    t.n_parts = (int32_t)(nitems[o] * kWaves);
    t.part_floats = kp * kp;
    t.ldp = kp;
    P.max_out = std::max(P.max_out, t.rows * t.cols);
    P.tasks.push_back(t);
  }
  // One launch per kernel instance.  Inside a launch every item of an op runs
  // on one XCD (the op's projection map then stays in that XCD's L2): ops are
  // dealt, costliest first, to the least-loaded of 8 per-XCD queues, and the
  // queues are interleaved (workgroup i goes to XCD i mod 8).
  struct Inst { int nt, aligned; std::vector<int> ops; };
  std::vector<Inst> insts;
  for (size_t o = 0; o < P.ops.size(); ++o) {
    if (nitems[o] == 0) continue;
    int found = -1;
    for (size_t i = 0; i < insts.size(); ++i)
      if (insts[i].nt == info[o].inst_nt && insts[i].aligned == info[o].aligned) found = (int)i;
    if (found < 0) {
      insts.push_back({info[o].inst_nt, info[o].aligned, {}});
      found = (int)insts.size() - 1;
    }
    insts[found].ops.push_back((int)o);
  }
  for (Inst& I : insts) {
    std::stable_sort(I.ops.begin(), I.ops.end(), [&](int a, int b) {
      return info[a].units * info[a].unit_cost > info[b].units * info[b].unit_cost;
    });
    std::vector<std::vector<FsumItem>> q(kXcds);
    double load[kXcds] = {0};
    for (int o : I.ops) {
      const int x = (int)(std::min_element(load, load + kXcds) - load);
      for (int64_t it = 0; it < nitems[o]; ++it) {
        const int64_t u0 = it * upi[o];
        const int64_t nu = std::min(upi[o], info[o].units - u0);
        q[x].push_back({o, (int32_t)u0, (int32_t)nu, (int32_t)it});
      }
      load[x] += (double)info[o].units * info[o].unit_cost;
    }
    size_t len = 0;
    for (const auto& v : q) len = std::max(len, v.size());
    const int first = (int)P.items.size();
    for (size_t s = 0; s < len; ++s)
      for (int x = 0; x < kXcds; ++x)
        P.items.push_back(s < q[x].size() ? q[x][s] : FsumItem{0, 0, 0, 0});
    P.launches.push_back({elt, I.aligned, I.nt, first, (int)P.items.size() - first});
  }
  size_t off = 0;
  P.off_ops = off;   off = align_up(off + P.ops.size() * sizeof(FsumOp));
  P.off_items = off; off = align_up(off + P.items.size() * sizeof(FsumItem));
  P.off_tasks = off; off = align_up(off + P.tasks.size() * sizeof(StatTask));
  P.blob_bytes = off;
  P.off_parts = off;
  off = align_up(off + part_floats_total * sizeof(float));
  P.total = off;
  return DATTRI_OK;
}

// ------------------------------------------------ projection with the fit
// The projection runs with projected token rows kept (fused factored members
// store them, the split form has them in its stage-1 buffer); the factor sums
// of those layers come from the stored rows, and only layers on the
// materialized route (which never form projected rows) take the separate
// factor-sum pass.  Workspace: [projection plan][row ops, row tasks, factor-sum
// descriptors][row partials][factor-sum partials].
constexpr int64_t kRowTargetItems = 2048;  // row-covariance workgroups aimed for

struct FitPlan {
  std::shared_ptr<const Plan> proj;
  std::vector<RowOp> rops;       // .rows set at run time from rop_off
  std::vector<size_t> rop_off;   // workspace byte offset of each op's rows
  std::vector<StatTask> rtasks;
  int max_items = 0, max_out = 0;
  FsumPlan mat;
  bool has_mat = false;
  size_t off_desc = 0, off_rops = 0, off_rtasks = 0, off_fdesc = 0, desc_bytes = 0;
  size_t off_rparts = 0, off_fparts = 0, total = 0;
};

dattri_status plan_fit(const dattri_ctx* ctx, const CurvLayout& C, dattri_route route, FitPlan& F) {
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  if (route < DATTRI_ROUTE_AUTO || route > DATTRI_ROUTE_MATERIALIZED)
    return fail(DATTRI_E_INVALID_ARG, "route %d unknown", (int)route);
  for (size_t l = 0; l < ctx->layers.size(); ++l)
    if (!ctx->layers[l].bound) return fail(DATTRI_E_STATE, "layer %zu: projection maps not bound", l);
  if ((st = get_plan(ctx, route, true, &F.proj)) != DATTRI_OK) return st;
  const int32_t n = ctx->layers[0].n;
  const int64_t n_ops = (int64_t)F.proj->row_srcs.size();
  const int epi = (int)std::max<int64_t>(1, cdiv((int64_t)n * n_ops, kRowTargetItems));
  size_t parts = 0;
  for (const RowSrc& R : F.proj->row_srcs) {
    const Layer& L = ctx->layers[R.layer];
    const int k = R.side ? L.k_out : L.k_in;
    RowOp o;
    std::memset(&o, 0, sizeof(o));
    o.lengths = L.lengths;
    o.ld = R.ld;
    o.col0 = R.col0;
    o.k = k;
    o.T = L.T;
    o.n = n;
    o.ex_per_item = epi;
    o.n_items = n > 0 ? (int)cdiv(n, epi) : 0;
    o.partial_base = (int64_t)parts;
    parts += (size_t)o.n_items * k * k;
    StatTask t = side_task(ctx, C, R.layer, R.side, n);
    t.part_base = o.partial_base;
    t.n_parts = o.n_items;
    t.part_floats = k * k;
    t.ldp = k;
    F.max_items = std::max(F.max_items, o.n_items);
    F.max_out = std::max(F.max_out, k * k);
    F.rops.push_back(o);
    F.rop_off.push_back(R.off);
    F.rtasks.push_back(t);
  }
  if (!F.proj->mat_layers.empty()) {
    if ((st = plan_fsum(ctx, C, F.mat, &F.proj->mat_layers)) != DATTRI_OK) return st;
    F.has_mat = true;
  }
  size_t off = align_up(F.proj->total);
  F.off_desc = off;
  F.off_rops = off;   off = align_up(off + F.rops.size() * sizeof(RowOp));
  F.off_rtasks = off; off = align_up(off + F.rtasks.size() * sizeof(StatTask));
  F.off_fdesc = off;  off = align_up(off + (F.has_mat ? F.mat.blob_bytes : 0));
  F.desc_bytes = off - F.off_desc;
  F.off_rparts = off; off = align_up(off + parts * sizeof(float));
  F.off_fparts = off; off = align_up(off + (F.has_mat ? F.mat.total - F.mat.off_parts : 0));
  F.total = off;
  return DATTRI_OK;
}

// ------------------------------------------------------------ EK-FAC plan
struct EkPlan {
  std::vector<RotTask> rot;
  std::vector<StatTask> tasks;
  int rows_per_block = 1, max_blocks = 0, max_out = 0;
  size_t off_rot = 0, off_tasks = 0, blob_bytes = 0, off_parts = 0, total = 0;
};

void plan_ekfac(const dattri_ctx* ctx, const CurvLayout& C, int64_t n, EkPlan& P) {
  const int64_t L = (int64_t)ctx->layers.size();
  P.rot = rot_tasks(ctx, C);
  const int64_t rpb = std::max<int64_t>(1, cdiv(n * L, kEkfacTargetBlocks));
  P.rows_per_block = (int)std::min<int64_t>(rpb, std::max<int64_t>(n, 1));
  const int64_t nb = n > 0 ? cdiv(n, P.rows_per_block) : 0;
  P.max_blocks = (int)nb;
  size_t part = 0;
  for (int64_t l = 0; l < L; ++l) {
    const Layer& Ly = ctx->layers[l];
    RotTask& r = P.rot[l];
    r.part_base = (int64_t)part;
    r.n_blocks = (int32_t)nb;
    part += (size_t)(nb * Ly.k_in * Ly.k_out);
    StatTask t;
    std::memset(&t, 0, sizeof(t));
    t.part_base = r.part_base;
    t.dst_off = C.L[l].sum_e;
    t.count_off = C.L[l].counts + 16;
    t.count_add = n;
    t.n_parts = (int32_t)nb;
    t.part_floats = Ly.k_in * Ly.k_out;
    t.ldp = Ly.k_out;
    t.rows = Ly.k_in;
    t.cols = Ly.k_out;
    P.max_out = std::max(P.max_out, Ly.k_in * Ly.k_out);
    P.tasks.push_back(t);
  }
  size_t off = 0;
  P.off_rot = off;   off = align_up(off + P.rot.size() * sizeof(RotTask));
  P.off_tasks = off; off = align_up(off + P.tasks.size() * sizeof(StatTask));
  P.blob_bytes = off;
  P.off_parts = off;
  off = align_up(off + part * sizeof(float));
  P.total = off;
}

dattri_status check_state(const void* state) {
  if (!state) return fail(DATTRI_E_INVALID_ARG, "state is NULL");
  if ((uintptr_t)state % kAlign) return fail(DATTRI_E_INVALID_ARG, "state must be 256-byte aligned");
  return DATTRI_OK;
}

dattri_status check_ws(const void* ws, size_t ws_bytes, size_t need) {
  if (!ws) return fail(DATTRI_E_WORKSPACE, "workspace is NULL (needs %zu bytes)", need);
  if ((uintptr_t)ws % kAlign) return fail(DATTRI_E_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < need) return fail(DATTRI_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  return DATTRI_OK;
}

// Host tables gathered into one blob at the given byte offsets.
std::vector<uint8_t> gather(const std::vector<const void*>& srcs, const std::vector<size_t>& offs,
                            const std::vector<size_t>& sizes, size_t total) {
  std::vector<uint8_t> blob(total, 0);
  for (size_t i = 0; i < srcs.size(); ++i)
    if (sizes[i]) std::memcpy(blob.data() + offs[i], srcs[i], sizes[i]);
  return blob;
}

// Launch tables of one call on the device (the bound plan buffer, else
// `fallback` in the workspace); *dev receives their base address.
hipError_t put_tables(const dattri_ctx* ctx, TableKind kind, uint8_t* fallback, const std::vector<const void*>& srcs,
                      const std::vector<size_t>& offs, const std::vector<size_t>& sizes, size_t total,
                      hipStream_t s, uint8_t** dev) {
  return place_table(ctx, kind, gather(srcs, offs, sizes, total), fallback, s, dev);
}

// Tables that live in the curvature state itself, copied to `dst` through a
// host buffer kept in the context until the next copy.
hipError_t copy_tables(const dattri_ctx* ctx, uint8_t* dst, const std::vector<const void*>& srcs,
                       const std::vector<size_t>& offs, const std::vector<size_t>& sizes, size_t total,
                       hipStream_t s) {
  ctx->blob = gather(srcs, offs, sizes, total);
  return hipMemcpyAsync(dst, ctx->blob.data(), total, hipMemcpyHostToDevice, s);
}

}  // namespace

extern "C" {

dattri_status dattri_curvature_state_bytes(const dattri_ctx* ctx, size_t* bytes) {
  reset_error();
  if (!bytes) return fail(DATTRI_E_INVALID_ARG, "bytes is NULL");
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  CurvLayout C;
  curv_layout(ctx, C);
  *bytes = C.total;
  return DATTRI_OK;
}

dattri_status dattri_curvature_layout_of(const dattri_ctx* ctx, int32_t layer,
                                         dattri_curvature_layout* out) {
  reset_error();
  if (!out) return fail(DATTRI_E_INVALID_ARG, "out is NULL");
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  if (layer < 0 || layer >= (int32_t)ctx->layers.size())
    return fail(DATTRI_E_INVALID_ARG, "layer %d out of range", layer);
  CurvLayout C;
  curv_layout(ctx, C);
  *out = C.L[layer];
  return DATTRI_OK;
}

dattri_status dattri_curvature_reset(const dattri_ctx* ctx, void* state, void* stream) {
  reset_error();
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  if ((st = check_state(state)) != DATTRI_OK) return st;
  CurvLayout C;
  curv_layout(ctx, C);
  HIP_TRY(launch_zero(state, (int64_t)C.total, (hipStream_t)stream));
  return DATTRI_OK;
}

dattri_status dattri_curvature_fit_workspace_bytes(const dattri_ctx* ctx, size_t* bytes) {
  reset_error();
  if (!bytes) return fail(DATTRI_E_INVALID_ARG, "bytes is NULL");
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  CurvLayout C;
  curv_layout(ctx, C);
  FsumPlan P;
  if ((st = plan_fsum(ctx, C, P)) != DATTRI_OK) return st;
  *bytes = P.total;
  return DATTRI_OK;
}

dattri_status dattri_curvature_accumulate_factors(dattri_ctx* ctx, void* state, void* workspace,
                                                  size_t ws_bytes, void* stream) {
  reset_error();
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  if ((st = check_state(state)) != DATTRI_OK) return st;
  CurvLayout C;
  curv_layout(ctx, C);
  FsumPlan P;
  if ((st = plan_fsum(ctx, C, P)) != DATTRI_OK) return st;
  if (P.n == 0) return DATTRI_OK;
  if ((st = check_ws(workspace, ws_bytes, P.total)) != DATTRI_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)workspace;
  uint8_t* tab = nullptr;
  HIP_TRY(put_tables(ctx, kTabFsum, ws, {P.ops.data(), P.items.data(), P.tasks.data()},
                     {P.off_ops, P.off_items, P.off_tasks},
                     {P.ops.size() * sizeof(FsumOp), P.items.size() * sizeof(FsumItem),
                      P.tasks.size() * sizeof(StatTask)},
                     P.blob_bytes, s, &tab));
  const FsumOp* d_ops = (const FsumOp*)(tab + P.off_ops);
  const FsumItem* d_items = (const FsumItem*)(tab + P.off_items);
  float* parts = (float*)(ws + P.off_parts);
  for (const FsumPlan::Launch& L : P.launches)
    HIP_TRY(launch_fsum(L.elt, L.aligned, L.nt, d_items + L.first, L.count, d_ops, parts, s));
  HIP_TRY(launch_stat_reduce((const StatTask*)(tab + P.off_tasks), (int)P.tasks.size(), P.max_out, parts,
                             (uint8_t*)state, s));
  return DATTRI_OK;
}

dattri_status dattri_curvature_eigen(const dattri_ctx* ctx, void* state, void* stream) {
  reset_error();
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  if ((st = check_state(state)) != DATTRI_OK) return st;
  CurvLayout C;
  curv_layout(ctx, C);
  std::vector<EigTask> E;
  for (size_t l = 0; l < ctx->layers.size(); ++l) {
    const dattri_curvature_layout& f = C.L[l];
    EigTask a, g;
    std::memset(&a, 0, sizeof(a));
    std::memset(&g, 0, sizeof(g));
    a.sum_off = f.sum_a; a.count_off = f.counts;     a.q_off = f.q_a; a.lam_off = f.lam_a;
    a.k = ctx->layers[l].k_in;
    g.sum_off = f.sum_g; g.count_off = f.counts + 8; g.q_off = f.q_g; g.lam_off = f.lam_g;
    g.k = ctx->layers[l].k_out;
    E.push_back(a);
    E.push_back(g);
  }
  hipStream_t s = (hipStream_t)stream;
  uint8_t* base = (uint8_t*)state;
  HIP_TRY(copy_tables(ctx, base + C.off_eig, {E.data()}, {0}, {E.size() * sizeof(EigTask)},
                      E.size() * sizeof(EigTask), s));
  HIP_TRY(launch_eigen((const EigTask*)(base + C.off_eig), (int)E.size(), base, s));
  return DATTRI_OK;
}

dattri_status dattri_curvature_ekfac_workspace_bytes(const dattri_ctx* ctx, int64_t n, size_t* bytes) {
  reset_error();
  if (!bytes) return fail(DATTRI_E_INVALID_ARG, "bytes is NULL");
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  if (n < 0) return fail(DATTRI_E_INVALID_ARG, "n=%lld < 0", (long long)n);
  CurvLayout C;
  curv_layout(ctx, C);
  EkPlan P;
  plan_ekfac(ctx, C, n, P);
  *bytes = P.total;
  return DATTRI_OK;
}

dattri_status dattri_curvature_accumulate_ekfac(const dattri_ctx* ctx, void* state, const void* phi,
                                                dattri_dtype dtype, int64_t n, int64_t ld,
                                                void* workspace, size_t ws_bytes, void* stream) {
  reset_error();
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  if ((st = check_state(state)) != DATTRI_OK) return st;
  if (dtype != DATTRI_F32 && dtype != DATTRI_BF16)
    return fail(DATTRI_E_DTYPE, "phi dtype %d is neither F32 nor BF16", (int)dtype);
  if (n < 0) return fail(DATTRI_E_INVALID_ARG, "n=%lld < 0", (long long)n);
  if (ld < ctx->F) return fail(DATTRI_E_SHAPE, "ld=%lld < F=%lld", (long long)ld, (long long)ctx->F);
  if (n == 0) return DATTRI_OK;
  if (!phi) return fail(DATTRI_E_INVALID_ARG, "phi is NULL");
  if (n > INT32_MAX) return fail(DATTRI_E_UNSUPPORTED, "n=%lld beyond 2^31 - 1", (long long)n);
  CurvLayout C;
  curv_layout(ctx, C);
  EkPlan P;
  plan_ekfac(ctx, C, n, P);
  if ((st = check_ws(workspace, ws_bytes, P.total)) != DATTRI_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)workspace;
  uint8_t* tab = nullptr;
  HIP_TRY(put_tables(ctx, kTabEkfac, ws, {P.rot.data(), P.tasks.data()}, {P.off_rot, P.off_tasks},
                     {P.rot.size() * sizeof(RotTask), P.tasks.size() * sizeof(StatTask)}, P.blob_bytes, s, &tab));
  float* parts = (float*)(ws + P.off_parts);
  HIP_TRY(launch_ekfac((const RotTask*)(tab + P.off_rot), (int)P.rot.size(), P.max_blocks,
                       (const uint8_t*)state, phi, dtype == DATTRI_BF16, ld, n, P.rows_per_block, parts, s));
  HIP_TRY(launch_stat_reduce((const StatTask*)(tab + P.off_tasks), (int)P.tasks.size(), P.max_out, parts,
                             (uint8_t*)state, s));
  return DATTRI_OK;
}

dattri_status dattri_curvature_precondition(const dattri_ctx* ctx, const void* state,
                                            dattri_curvature kind, double damping_rel,
                                            double damping_abs, const void* phi_q,
                                            dattri_dtype in_dtype, int64_t n_q, int64_t ld_q,
                                            void* out, dattri_dtype out_dtype, int64_t ld_out,
                                            void* stream) {
  reset_error();
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  if ((st = check_state(state)) != DATTRI_OK) return st;
  if (kind != DATTRI_CURV_KFAC && kind != DATTRI_CURV_EKFAC)
    return fail(DATTRI_E_INVALID_ARG, "curvature kind %d unknown", (int)kind);
  if (!(damping_rel >= 0.0) || !(damping_abs >= 0.0) || !std::isfinite(damping_rel) ||
      !std::isfinite(damping_abs) || (damping_rel == 0.0 && damping_abs == 0.0))
    return fail(DATTRI_E_INVALID_ARG, "damping needs rel >= 0, abs >= 0, finite, not both zero (got %g, %g)",
                damping_rel, damping_abs);
  if ((in_dtype != DATTRI_F32 && in_dtype != DATTRI_BF16) || (out_dtype != DATTRI_F32 && out_dtype != DATTRI_BF16))
    return fail(DATTRI_E_DTYPE, "dtypes must be F32 or BF16");
  if (n_q < 0) return fail(DATTRI_E_INVALID_ARG, "n_q=%lld < 0", (long long)n_q);
  if (ld_q < ctx->F || ld_out < ctx->F)
    return fail(DATTRI_E_SHAPE, "ld_q=%lld, ld_out=%lld must be >= F=%lld", (long long)ld_q, (long long)ld_out,
                (long long)ctx->F);
  if (n_q == 0) return DATTRI_OK;
  if (!phi_q || !out) return fail(DATTRI_E_INVALID_ARG, "phi_q or out is NULL");
  {  // out must not overlap phi_q
    const int64_t eq = in_dtype == DATTRI_BF16 ? 2 : 4, eo = out_dtype == DATTRI_BF16 ? 2 : 4;
    const uintptr_t a0 = (uintptr_t)phi_q, a1 = a0 + (uintptr_t)(((n_q - 1) * ld_q + ctx->F) * eq);
    const uintptr_t b0 = (uintptr_t)out, b1 = b0 + (uintptr_t)(((n_q - 1) * ld_out + ctx->F) * eo);
    if (a0 < b1 && b0 < a1) return fail(DATTRI_E_INVALID_ARG, "out overlaps phi_q");
  }
  CurvLayout C;
  curv_layout(ctx, C);
  std::vector<RotTask> R = rot_tasks(ctx, C);
  hipStream_t s = (hipStream_t)stream;
  uint8_t* base = (uint8_t*)const_cast<void*>(state);
  HIP_TRY(copy_tables(ctx, base + C.off_rot, {R.data()}, {0}, {R.size() * sizeof(RotTask)},
                      R.size() * sizeof(RotTask), s));
  HIP_TRY(launch_precondition((const RotTask*)(base + C.off_rot), (int)R.size(), base, (int)kind, damping_rel,
                              damping_abs, phi_q, in_dtype == DATTRI_BF16, ld_q, n_q, out,
                              out_dtype == DATTRI_BF16, ld_out, s));
  return DATTRI_OK;
}

dattri_status dattri_project_fit_workspace_bytes(const dattri_ctx* ctx, dattri_route route, size_t* bytes) {
  reset_error();
  if (!bytes) return fail(DATTRI_E_INVALID_ARG, "bytes is NULL");
  CurvLayout C;
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  curv_layout(ctx, C);
  FitPlan F;
  if ((st = plan_fit(ctx, C, route, F)) != DATTRI_OK) return st;
  *bytes = F.total;
  return DATTRI_OK;
}

dattri_status dattri_project_and_fit(dattri_ctx* ctx, void* phi, dattri_dtype phi_dtype, int64_t ld_phi,
                                     void* state, void* workspace, size_t ws_bytes, dattri_route route,
                                     void* stream) {
  reset_error();
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  if ((st = check_state(state)) != DATTRI_OK) return st;
  if (phi_dtype != DATTRI_F32 && phi_dtype != DATTRI_BF16)
    return fail(DATTRI_E_DTYPE, "phi dtype %d is neither F32 nor BF16", (int)phi_dtype);
  CurvLayout C;
  curv_layout(ctx, C);
  FitPlan F;
  if ((st = plan_fit(ctx, C, route, F)) != DATTRI_OK) return st;
  const int32_t n = ctx->layers[0].n;
  if (ld_phi < ctx->F) return fail(DATTRI_E_SHAPE, "ld_phi=%lld < F=%lld", (long long)ld_phi, (long long)ctx->F);
  if (n == 0) return DATTRI_OK;
  if (!phi) return fail(DATTRI_E_INVALID_ARG, "phi is NULL");
  if ((st = check_ws(workspace, ws_bytes, F.total)) != DATTRI_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)workspace;
  if ((st = run_plan(ctx, *F.proj, phi, phi_dtype, ld_phi, workspace, ws_bytes, s)) != DATTRI_OK) return st;
  std::vector<RowOp> rops = F.rops;
  for (size_t i = 0; i < rops.size(); ++i) rops[i].rows = (const float*)(ws + F.rop_off[i]);
  std::vector<const void*> srcs = {rops.data(), F.rtasks.data()};
  std::vector<size_t> offs = {F.off_rops - F.off_desc, F.off_rtasks - F.off_desc};
  std::vector<size_t> sizes = {rops.size() * sizeof(RowOp), F.rtasks.size() * sizeof(StatTask)};
  if (F.has_mat) {
    const size_t b = F.off_fdesc - F.off_desc;
    srcs.insert(srcs.end(), {F.mat.ops.data(), F.mat.items.data(), F.mat.tasks.data()});
    offs.insert(offs.end(), {b + F.mat.off_ops, b + F.mat.off_items, b + F.mat.off_tasks});
    sizes.insert(sizes.end(), {F.mat.ops.size() * sizeof(FsumOp), F.mat.items.size() * sizeof(FsumItem),
                               F.mat.tasks.size() * sizeof(StatTask)});
  }
  uint8_t* tab = nullptr;
  HIP_TRY(put_tables(ctx, kTabFit, ws + F.off_desc, srcs, offs, sizes, F.desc_bytes, s, &tab));
  float* rparts = (float*)(ws + F.off_rparts);
  HIP_TRY(launch_rowcov((const RowOp*)(tab + (F.off_rops - F.off_desc)), (int)rops.size(), F.max_items, rparts, s));
  HIP_TRY(launch_stat_reduce((const StatTask*)(tab + (F.off_rtasks - F.off_desc)), (int)F.rtasks.size(), F.max_out,
                             rparts, (uint8_t*)state, s));
  if (F.has_mat) {
    const uint8_t* fd = tab + (F.off_fdesc - F.off_desc);
    float* fparts = (float*)(ws + F.off_fparts);
    for (const FsumPlan::Launch& L : F.mat.launches)
      HIP_TRY(launch_fsum(L.elt, L.aligned, L.nt, (const FsumItem*)(fd + F.mat.off_items) + L.first, L.count,
                          (const FsumOp*)(fd + F.mat.off_ops), fparts, s));
    HIP_TRY(launch_stat_reduce((const StatTask*)(fd + F.mat.off_tasks), (int)F.mat.tasks.size(), F.mat.max_out,
                               fparts, (uint8_t*)state, s));
  }
  return DATTRI_OK;
}

// ---------------------------------------------------------- token scores
// Workspace: [projection plan with rows kept][token tasks][phi when not given].
struct TokPlan {
  std::shared_ptr<const Plan> proj;
  std::vector<TokTask> tasks;
  std::vector<std::pair<size_t, size_t>> rows_off;  // workspace offsets of each layer's A and B rows
  size_t off_tasks = 0, off_phi = 0, total = 0;
  int T = 0;
};

dattri_status plan_tokens(const dattri_ctx* ctx, TokPlan& K) {
  dattri_status st = check_layers(ctx);
  if (st != DATTRI_OK) return st;
  for (size_t l = 0; l < ctx->layers.size(); ++l) {
    const Layer& L = ctx->layers[l];
    if (!L.bound) return fail(DATTRI_E_STATE, "layer %zu: projection maps not bound", l);
    if (L.captured && L.T != ctx->layers[0].T)
      return fail(DATTRI_E_SHAPE, "layer %zu captured with T=%d but layer 0 with T=%d", l, L.T, ctx->layers[0].T);
  }
  // every layer on the factored route, whose kernels form the projected rows
  if ((st = get_plan(ctx, DATTRI_ROUTE_FACTORED, true, &K.proj)) != DATTRI_OK) return st;
  K.T = ctx->layers[0].T;
  K.tasks.assign(ctx->layers.size(), TokTask{});
  K.rows_off.assign(ctx->layers.size(), {0, 0});
  for (const RowSrc& R : K.proj->row_srcs) {
    TokTask& t = K.tasks[R.layer];
    const Layer& L = ctx->layers[R.layer];
    t.lengths = L.lengths;
    t.q_off = L.offset;
    t.k_in = L.k_in;
    t.k_out = L.k_out;
    if (R.side == 0) {
      K.rows_off[R.layer].first = R.off;
      t.a_ld = R.ld;
      t.a_col0 = R.col0;
    } else {
      K.rows_off[R.layer].second = R.off;
      t.b_ld = R.ld;
      t.b_col0 = R.col0;
    }
  }
  size_t off = align_up(K.proj->total);
  K.off_tasks = off;
  off = align_up(off + K.tasks.size() * sizeof(TokTask));
  K.off_phi = off;
  off = align_up(off + (size_t)ctx->layers[0].n * ctx->F * 4);
  K.total = off;
  return DATTRI_OK;
}

dattri_status dattri_token_scores_workspace_bytes(const dattri_ctx* ctx, size_t* bytes) {
  reset_error();
  if (!bytes) return fail(DATTRI_E_INVALID_ARG, "bytes is NULL");
  TokPlan K;
  dattri_status st = plan_tokens(ctx, K);
  if (st != DATTRI_OK) return st;
  *bytes = K.total;
  return DATTRI_OK;
}

dattri_status dattri_token_scores(dattri_ctx* ctx, const void* phi_q, dattri_dtype q_dtype, int64_t n_q, int64_t ld_q,
                                  float* scores, void* phi, dattri_dtype phi_dtype, int64_t ld_phi, void* workspace,
                                  size_t ws_bytes, void* stream) {
  reset_error();
  TokPlan K;
  dattri_status st = plan_tokens(ctx, K);
  if (st != DATTRI_OK) return st;
  if (q_dtype != DATTRI_F32 && q_dtype != DATTRI_BF16)
    return fail(DATTRI_E_DTYPE, "query dtype %d is neither F32 nor BF16", (int)q_dtype);
  if (phi && phi_dtype != DATTRI_F32 && phi_dtype != DATTRI_BF16)
    return fail(DATTRI_E_DTYPE, "phi dtype %d is neither F32 nor BF16", (int)phi_dtype);
  if (n_q < 0) return fail(DATTRI_E_INVALID_ARG, "n_q=%lld < 0", (long long)n_q);
  if (ld_q < ctx->F) return fail(DATTRI_E_SHAPE, "ld_q=%lld < F=%lld", (long long)ld_q, (long long)ctx->F);
  if (phi && ld_phi < ctx->F)
    return fail(DATTRI_E_SHAPE, "ld_phi=%lld < F=%lld", (long long)ld_phi, (long long)ctx->F);
  const int64_t n = ctx->layers[0].n;
  if (n == 0 || n_q == 0 || K.T == 0) return DATTRI_OK;
  if (!phi_q || !scores) return fail(DATTRI_E_INVALID_ARG, "phi_q or scores is NULL");
  if (n > 65535 || n_q > 65535)
    return fail(DATTRI_E_UNSUPPORTED, "n=%lld examples or n_q=%lld queries beyond the grid limits", (long long)n,
                (long long)n_q);
  if ((st = check_ws(workspace, ws_bytes, K.total)) != DATTRI_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)workspace;
  void* phi_out = phi ? phi : (void*)(ws + K.off_phi);
  const dattri_dtype pd = phi ? phi_dtype : DATTRI_F32;
  const int64_t pld = phi ? ld_phi : ctx->F;
  if ((st = run_plan(ctx, *K.proj, phi_out, pd, pld, workspace, ws_bytes, s)) != DATTRI_OK) return st;
  std::vector<TokTask> tasks = K.tasks;
  for (size_t l = 0; l < tasks.size(); ++l) {
    tasks[l].a_rows = (const float*)(ws + K.rows_off[l].first);
    tasks[l].b_rows = (const float*)(ws + K.rows_off[l].second);
  }
  uint8_t* tab = nullptr;
  HIP_TRY(put_tables(ctx, kTabTok, ws + K.off_tasks, {tasks.data()}, {0}, {tasks.size() * sizeof(TokTask)},
                     tasks.size() * sizeof(TokTask), s, &tab));
  HIP_TRY(launch_token_scores((const TokTask*)tab, (int)tasks.size(), phi_q, q_dtype == DATTRI_BF16,
                              ld_q, n_q, n, K.T, scores, s));
  return DATTRI_OK;
}

}  // extern "C"
