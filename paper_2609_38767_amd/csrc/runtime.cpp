// Host runtime of libdattri: context, layer registry, validation, the MI355X
// cost model that routes each layer (Sec. 3.2 "FLOP-aware routing", App. A.4),
// launch planning and the C ABI declared in include/dattri.h.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "api_common.h"
#include "context.h"
#include "dattri.h"
#include "internal.h"
#include "plan.h"
#include "runtime.h"

using namespace dattri;

namespace dattri {

static thread_local std::string g_err;

dattri_status fail(dattri_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

void reset_error() { g_err.clear(); }
const char* last_error_message() { return g_err.c_str(); }

}  // namespace dattri

namespace {

constexpr int kMaxDim = 1 << 20;
constexpr int64_t kGBudgetBytes = (int64_t)2 << 30;   // staged G per materialized chunk

inline int tiles16(int k) { return (k + 15) / 16; }

bool factored_supported(const Layer& L) {
  return tiles16(L.k_in) <= kMaxGroupTiles && tiles16(L.k_out) <= kMaxMemberBTiles;
}

dattri_cost_model default_cost_model() {
  // Fitted on MI355X (bf16 inputs; the calibration script's sweep of 28
  // single-layer shapes: transformer, adapter-shaped and narrow layers,
  // T = 16..4096, both forced routes timed with launch plans kept on the
  // device), every rate held below its bound: AUTO picks the faster route on
  // all 28 shapes, root-mean-square log error of the predictions 0.15.
  // gproject_gbs and gproject_tflops serve only the staged-G route, which
  // that sweep does not run.
  dattri_cost_model m;
  m.factored_tflops = 175.9;
  m.factored_gbs = 6450.0;
  m.gradient_tflops = 837.2;
  m.gradient_gbs = 6450.0;
  m.gproject_tflops = 157.3;
  m.gproject_gbs = 5000.0;
  m.launch_us = 10.74;
  m.call_us = 0.0;
  m.round_us = 0.674;
  return m;
}

// Published MI355X peaks that bound the model's effective rates.
constexpr double kPeakGbs = 8000.0, kPeakBf16Tflops = 2500.0, kPeakF32Tflops = 157.3;

dattri_status check_cost_model(const dattri_cost_model& m) {
  const struct { const char* name; double v, cap; } rates[] = {
      {"factored_tflops", m.factored_tflops, kPeakBf16Tflops}, {"factored_gbs", m.factored_gbs, kPeakGbs},
      {"gradient_tflops", m.gradient_tflops, kPeakBf16Tflops}, {"gradient_gbs", m.gradient_gbs, kPeakGbs},
      {"gproject_tflops", m.gproject_tflops, kPeakF32Tflops}, {"gproject_gbs", m.gproject_gbs, kPeakGbs}};
  for (const auto& r : rates)
    if (!(r.v > 0.0) || !std::isfinite(r.v) || r.v > r.cap)
      return fail(DATTRI_E_INVALID_ARG, "%s = %g must be finite, > 0 and at most the peak %g", r.name, r.v, r.cap);
  if (!(m.launch_us >= 0.0) || !std::isfinite(m.launch_us))
    return fail(DATTRI_E_INVALID_ARG, "launch_us = %g must be finite and >= 0", m.launch_us);
  if (!(m.call_us >= 0.0) || !std::isfinite(m.call_us))
    return fail(DATTRI_E_INVALID_ARG, "call_us = %g must be finite and >= 0", m.call_us);
  if (!(m.round_us >= 0.0) || !std::isfinite(m.round_us))
    return fail(DATTRI_E_INVALID_ARG, "round_us = %g must be finite and >= 0", m.round_us);
  return DATTRI_OK;
}

}  // namespace


namespace {

// ------------------------------------------------------------- cost model
struct Counts {
  int64_t f_flops, m_flops, f_bytes, m_bytes, g_flops, g_bytes, p_flops, p_bytes;
};

Counts layer_counts(const Layer& L, int64_t T, int elt) {
  Counts c;
  const int64_t di = L.d_in, dq = L.d_out, ki = L.k_in, ko = L.k_out;
  c.f_flops = 2 * T * (di * ki + dq * ko + ki * ko);
  c.g_flops = 2 * T * di * dq;
  c.p_flops = 2 * dq * di * ki + 2 * dq * ki * ko;
  c.m_flops = c.g_flops + c.p_flops;
  c.f_bytes = T * (di + dq) * elt;
  c.g_bytes = c.f_bytes + 4 * dq * di;
  c.p_bytes = 4 * dq * di;
  c.m_bytes = c.g_bytes + c.p_bytes;
  return c;
}

// Kernel launches of a layer's factored route if it were projected alone: the
// launch plan of a one-layer context decides fused or split form and stages.
int factored_launches(const dattri_ctx* ctx, const Layer& L) {
  dattri_ctx one;
  one.dtype = ctx->dtype;
  one.elt = ctx->elt;
  one.seed = ctx->seed;
  one.form = ctx->form;
  one.cost = ctx->cost;
  one.xcost = ctx->xcost;
  Layer C;  // the plan needs sizes, captures and map pointers only
  C.d_in = L.d_in; C.d_out = L.d_out; C.k_in = L.k_in; C.k_out = L.k_out;
  C.P_in = L.P_in; C.P_out = L.P_out; C.bound = L.bound;
  C.A = L.A; C.B = L.B; C.n = L.n; C.T = L.T; C.lengths = L.lengths; C.captured = L.captured;
  one.layers.push_back(C);
  one.F = (int64_t)L.k_in * L.k_out;
  Plan P;
  if (build_plan(&one, DATTRI_ROUTE_FACTORED, P, false) != DATTRI_OK) {
    reset_error();  // not a failure of the caller's request: count the fused form
    return 2;
  }
  return (int)(P.launches.size() + (P.n_fact_tasks ? 1 : 0) + P.slaunches.size() + (P.slabsum.empty() ? 0 : 1) +
               (P.ctasks.empty() ? 0 : 1) + (P.stasks.empty() ? 0 : 1));
}

// Example chunks of the materialized route: G of a chunk fits the staging budget.
int64_t materialized_chunk(const Layer& L, int64_t n) {
  const int64_t g_per_ex = (int64_t)L.d_out * L.d_in;
  return std::max<int64_t>(1, std::min<int64_t>({n, kGBudgetBytes / (4 * g_per_ex), (int64_t)65535}));
}

// The one-pass materialized kernel serves bf16 layers with 16-byte aligned
// rows and k_in <= 128; others stage G in the workspace.
bool fused_materialized(const Layer& L, int elt) {
  return elt == 2 && (uintptr_t)L.A % 16 == 0 && (uintptr_t)L.B % 16 == 0 && (L.d_in * 2) % 16 == 0 &&
         (L.d_out * 2) % 16 == 0 && tiles16(L.k_in) <= kGFusedMaxTilesIn;
}

// Launch shape of the one-pass kernel and its predicted time.  A workgroup
// runs, per 128-column tile of G in its range, tok_chunk / 32 token stages
// and a projection of the tile from its accumulators (three bf16 MFMA terms
// per product, against 32 tiles_in / 2 columns of P_in), then one closing
// H^T P_out the same way.  occ workgroups share a CU (36 KiB of LDS each; two
// when k_in <= 64, where the registers allow it).  Token chunks and column
// ranges add workgroups but the chunks repeat the projections; the shape
// minimising rounds of 256 occ workgroups x occ x per-workgroup time wins.
// Times use the model's rates: a round of 256 workgroups each running one
// stage is 256 x 2 x 32 x 128 x 128 FLOP, one tile projection per workgroup
// 256 x 3 x 2 x 128 x 128 x 16 x tiles_in FLOP, the closing product
// 256 x 3 x 2 x 128 x 16 tiles_in x 32 tiles32(k_out) FLOP, all bf16 MFMA at
// gradient_tflops; each round also costs round_us (load latencies and
// barriers, whatever the work).
struct FusedShape { int n_tchunks, tok_chunk, n_vsplit, vt_per_split; double us; };
FusedShape fused_shape(const Layer& L, int64_t n, const dattri_cost_model& m) {
  const int64_t T = std::max<int64_t>(L.T, 1);
  const int64_t n_ub = (L.d_out + kGFusedRows - 1) / kGFusedRows;
  const int64_t n_vt = (L.d_in + kGFusedCols - 1) / kGFusedCols;
  const int occ = gfused_wgs_per_cu(L.k_in);
  const double stage_us = 256.0 * 2 * 32 * kGFusedRows * kGFusedCols / (m.gradient_tflops * 1e6);
  const double proj_us = 256.0 * 3 * 2 * kGFusedRows * kGFusedCols * 16 * gfused_tiles_in(L.k_in) /
                         (m.gradient_tflops * 1e6);
  const double epi_us = 256.0 * 3 * 2 * kGFusedRows * 16 * gfused_tiles_in(L.k_in) * 32 *
                        ((L.k_out + 31) / 32) / (m.gradient_tflops * 1e6);
  FusedShape best{1, (int)((T + 31) / 32 * 32), 1, (int)n_vt, -1.0};
  for (int64_t c = 1; c <= (T + 31) / 32; c *= 2) {
    const int64_t tok_chunk = ((T + c - 1) / c + 31) / 32 * 32;
    const int64_t chunks = (T + tok_chunk - 1) / tok_chunk;
    for (int64_t v = 1; v <= n_vt; v *= 2) {
      const int64_t vps = (n_vt + v - 1) / v;
      const int64_t splits = (n_vt + vps - 1) / vps;
      const int64_t slots = 256 * (int64_t)occ;
      const int64_t rounds = (std::max<int64_t>(n, 1) * n_ub * splits * chunks + slots - 1) / slots;
      const double us = (double)rounds * ((double)occ * ((double)vps * ((double)(tok_chunk / 32) * stage_us + proj_us) +
                                                         epi_us) +
                                          m.round_us);
      if (best.us < 0 || us < best.us)
        best = FusedShape{(int)chunks, (int)tok_chunk, (int)splits, (int)vps, us};
    }
  }
  return best;
}

// Predicted times (us) of both routes for the layer's capture (n, T).
// f_launch_us (optional) receives the launch part of the factored time.
void predict(const dattri_ctx* ctx, const Layer& L, double* f_us, double* m_us, double* f_launch_us = nullptr) {
  const dattri_cost_model& m = ctx->cost;
  const int64_t n = L.n;
  const Counts c = layer_counts(L, L.T, ctx->elt);
  auto t = [](double flops, double tflops, double bytes, double gbs) {
    return std::max(flops / (tflops * 1e6), bytes / (gbs * 1e3));  // microseconds
  };
  *f_us = m.call_us + t((double)c.f_flops * n, m.factored_tflops, (double)c.f_bytes * n, m.factored_gbs);
  const double fl = n > 0 ? factored_launches(ctx, L) * m.launch_us : 0.0;
  *f_us += fl;
  if (f_launch_us) *f_launch_us = fl;
  if (fused_materialized(L, ctx->elt)) {
    // one pass: factor blocks read once, G on chip; time from its launch shape.
    // One launch is charged for the pair of kernels: the small reduction of
    // the partial products dispatches behind the one-pass kernel, and on
    // MI355X the pair's fixed cost measures about one launch (13.6 us in all
    // for the smallest layers).
    const int64_t chunks = n > 0 ? (n + 65534) / 65535 : 0;
    const double work = n > 0 ? fused_shape(L, n, m).us : 0.0;
    *m_us = m.call_us + std::max(work, (double)c.f_bytes * n / (m.gradient_gbs * 1e3)) +
            chunks * m.launch_us;
    return;
  }
  const int64_t chunks = n > 0 ? (n + materialized_chunk(L, n) - 1) / materialized_chunk(L, n) : 0;
  *m_us = m.call_us + t((double)c.g_flops * n, m.gradient_tflops, (double)c.g_bytes * n, m.gradient_gbs) +
          t((double)c.p_flops * n, m.gproject_tflops, (double)c.p_bytes * n, m.gproject_gbs) +
          3.0 * chunks * m.launch_us;
}

dattri_route choose_route(const dattri_ctx* ctx, const Layer& L, dattri_route forced) {
  if (L.mask_size > 0) return DATTRI_ROUTE_MASK;  // gathered from the factors, whatever the request
  if (forced != DATTRI_ROUTE_AUTO) return forced;
  if (!factored_supported(L)) return DATTRI_ROUTE_MATERIALIZED;
  double f, m;
  predict(ctx, L, &f, &m);
  return f <= m ? DATTRI_ROUTE_FACTORED : DATTRI_ROUTE_MATERIALIZED;
}

std::vector<uint64_t> plan_key(const dattri_ctx* ctx, dattri_route forced, bool rows);

// Routes of a call over all captured layers.  Each layer is first decided on
// its own (choose_route).  Under AUTO, once some layer is factored the
// factored launches are paid anyway and shared by every factored layer, while
// each materialized layer adds launches of its own; so a layer AUTO sent to
// the materialized route joins the factored one when its factored time
// without launches is no more than its materialized time.  (A stack of 196
// Qwen-shaped layers with one example: 56 k/v layers would otherwise run
// materialized, 2.4 ms per call against 0.8 ms.)  Cached by the plan key.
const std::vector<dattri_route>& call_routes(const dattri_ctx* ctx, dattri_route forced) {
  std::vector<uint64_t> key = plan_key(ctx, forced, false);
  if (ctx->route_cache.first == key) return ctx->route_cache.second;
  std::vector<dattri_route> route(ctx->layers.size(), DATTRI_ROUTE_FACTORED);
  std::vector<double> f_work(ctx->layers.size(), 0.0), m_us(ctx->layers.size(), 0.0);
  bool any_factored = false;
  for (size_t l = 0; l < ctx->layers.size(); ++l) {
    const Layer& L = ctx->layers[l];
    route[l] = choose_route(ctx, L, forced);
    if (forced == DATTRI_ROUTE_AUTO && route[l] == DATTRI_ROUTE_MATERIALIZED && factored_supported(L)) {
      double f, fl;
      predict(ctx, L, &f, &m_us[l], &fl);
      f_work[l] = f - fl;
    }
    any_factored = any_factored || route[l] == DATTRI_ROUTE_FACTORED;
  }
  if (forced == DATTRI_ROUTE_AUTO && any_factored)
    for (size_t l = 0; l < ctx->layers.size(); ++l)
      if (route[l] == DATTRI_ROUTE_MATERIALIZED && factored_supported(ctx->layers[l]) && f_work[l] <= m_us[l])
        route[l] = DATTRI_ROUTE_FACTORED;
  ctx->route_cache = {std::move(key), std::move(route)};
  return ctx->route_cache.second;
}

// ---------------------------------------------------------------- planning
// The split form serves every factored group when the fused kernel would have
// fewer than kSplitMinFusedItems work items.
constexpr int64_t kSplitMinFusedItems = 1024;
constexpr int64_t kSplitTargetItems = 1024;   // stage-1 workgroups aimed for
constexpr int64_t kContractTargetItems = 512; // stage-2 workgroups aimed for
constexpr int64_t kGProjTargetBlocks = 1024;  // G-projection workgroups aimed for

dattri_status check_captures(const dattri_ctx* ctx, int32_t* n_out) {
  if (ctx->layers.empty()) return fail(DATTRI_E_STATE, "no layer registered");
  int32_t n = -1;
  for (size_t l = 0; l < ctx->layers.size(); ++l) {
    const Layer& L = ctx->layers[l];
    if (!L.captured) return fail(DATTRI_E_STATE, "layer %zu has no capture", l);
    if (n < 0) n = L.n;
    if (L.n != n)
      return fail(DATTRI_E_STATE, "layer %zu captured with n=%d but layer 0 with n=%d", l, L.n, n);
  }
  *n_out = n;
  return DATTRI_OK;
}

}  // namespace

dattri_status dattri::build_plan(const dattri_ctx* ctx, dattri_route forced, Plan& P, bool rows) {
  int32_t n = 0;
  dattri_status st = check_captures(ctx, &n);
  if (st != DATTRI_OK) return st;
  const int elt = ctx->elt;

  // ---- factored layers: group by shared input block A.  A layer joins a
  // group only while the grouped kernel instance keeps the token rows per wave
  // of the layer alone: on MI355X the register-path kernel streams markedly
  // faster at 4 row tiles per wave than at 2 or 1, more than the cost of
  // reading A once per layer (Llama-3-8B stack: 15.8 ms per batch ungrouped vs
  // 17.4 ms with q/k/v and gate/up grouped).  The direct-load instances (bf16,
  // aligned rows, output maps of 2 tiles) keep 4 row tiles per wave with up to
  // 6 input tiles, so there q/k/v and gate/up do group and A is read once per
  // block: 85.5 -> 74.0 GB and 13.08 -> 12.33 ms per batch of 8.
  auto rows_per_wave = [&](int na, int nb) {
    int nai, nbi, rt;
    factored_instance(elt, na, nb, 1, &nai, &nbi, &rt);
    return rt;
  };
  const std::vector<dattri_route> route = call_routes(ctx, forced);
  std::vector<std::vector<int>> group_layers;
  for (size_t l = 0; l < ctx->layers.size(); ++l) {
    const Layer& L = ctx->layers[l];
    const dattri_route r = route[l];
    if (r == DATTRI_ROUTE_MATERIALIZED || r == DATTRI_ROUTE_MASK) continue;
    if (!factored_supported(L))
      return fail(DATTRI_E_UNSUPPORTED,
                  "layer %zu: factored route needs k_in <= %d and k_out <= %d (got %d, %d)", l,
                  16 * kMaxGroupTiles, 16 * kMaxMemberBTiles, L.k_in, L.k_out);
    int found = -1;
    for (size_t g = 0; g < group_layers.size() && found < 0; ++g) {
      const Layer& H = ctx->layers[group_layers[g][0]];
      int na = 0, nb = 0;
      for (int m : group_layers[g]) {
        na += tiles16(ctx->layers[m].k_in);
        nb = std::max(nb, tiles16(ctx->layers[m].k_out));
      }
      const int na2 = na + tiles16(L.k_in), nb2 = std::max(nb, tiles16(L.k_out));
      if (H.A == L.A && H.d_in == L.d_in && H.T == L.T && H.lengths == L.lengths &&
          L.A != nullptr && na2 <= kMaxGroupTiles &&
          rows_per_wave(na2, nb2) >= rows_per_wave(tiles16(L.k_in), tiles16(L.k_out)))
        found = (int)g;
    }
    if (found < 0) {
      group_layers.push_back({(int)l});
    } else {
      group_layers[found].push_back((int)l);
    }
  }

  // Fused-kernel shape of each group: input tiles, widest member, 16-byte
  // alignment, token chunking.
  struct GShape { int na, nb_max, aligned, na_inst, nb_inst, rt, chunk_rows, n_chunks; };
  std::vector<GShape> gshape(group_layers.size());
  int64_t fused_items_total = 0;
  for (size_t g = 0; g < group_layers.size(); ++g) {
    const Layer& H = ctx->layers[group_layers[g][0]];
    GShape& S = gshape[g];
    S.aligned = ((uintptr_t)H.A % 16 == 0) && (H.d_in * elt) % 16 == 0;
    S.na = 0;
    S.nb_max = 0;
    for (int li : group_layers[g]) {
      const Layer& L = ctx->layers[li];
      S.aligned = S.aligned && ((uintptr_t)L.B % 16 == 0) && (L.d_out * elt) % 16 == 0;
      S.na += tiles16(L.k_in);
      S.nb_max = std::max(S.nb_max, tiles16(L.k_out));
    }
    factored_instance(elt, S.na, S.nb_max, S.aligned, &S.na_inst, &S.nb_inst, &S.rt);
    const int sub_rows = kWaves * S.rt * 16;
    int cr = std::max(sub_rows, 512 / sub_rows * sub_rows);
    if (H.T <= cr) cr = std::max(sub_rows, (H.T + sub_rows - 1) / sub_rows * sub_rows);
    S.chunk_rows = cr;
    S.n_chunks = std::max(1, (H.T + cr - 1) / cr);
    fused_items_total += (int64_t)n * S.n_chunks;
  }
  const bool few_items = fused_items_total < kSplitMinFusedItems;
  // Wide maps (4 x 4 input x output tiles and more, k > 48 on both sides)
  // leave the register-path fused kernel 2 row tiles per wave and 2 waves per
  // SIMD; the split form, which projects one factor at a time, streams faster
  // there (Qwen2.5-7B-shaped stack, k = 64, T = 512, 32 examples: 19.2 ms vs
  // 26.8 ms per batch on MI355X).  The direct-load instances keep 4 row tiles
  // per wave with 4-tile maps and stay fused.
  auto use_split = [&](size_t g) {
    const Layer& H = ctx->layers[group_layers[g][0]];
    if ((int64_t)n * H.T > (int64_t)INT32_MAX / 2 || n > 65535) return false;  // index / grid range
    if (ctx->form != DATTRI_FORM_AUTO) return ctx->form == DATTRI_FORM_SPLIT;
    const GShape& S = gshape[g];
    return few_items ||
           (S.na_inst * S.nb_inst >= 16 && !factored_direct_loads(elt, S.na_inst, S.nb_inst, S.aligned));
  };

  size_t fpart_floats = 0;
  std::vector<int> member_layer;  // layer of each fused member
  struct SplitRows { int layer, a_op, b_op, a_col0; };
  std::vector<SplitRows> split_rows;  // split-form layers: their stage-1 ops
  struct Inst { int na, nb, aligned; std::vector<int> groups; };
  std::vector<Inst> insts;
  std::vector<double> group_cost;
  std::vector<size_t> split_groups;
  for (size_t g = 0; g < group_layers.size(); ++g) {
    if (use_split(g)) {
      split_groups.push_back(g);
      continue;
    }
    const int fg = (int)P.groups.size();  // index among fused groups
    const Layer& H = ctx->layers[group_layers[g][0]];
    FactGroup G;
    std::memset(&G, 0, sizeof(G));
    G.A = H.A;
    G.lengths = H.lengths;
    G.d_in = H.d_in;
    G.T = H.T;
    G.n = n;
    G.n_members = (int)group_layers[g].size();
    G.member0 = (int)P.members.size();
    const bool aligned = gshape[g].aligned;
    int na = 0;
    double bytes_per_row = (double)H.d_in;
    for (int li : group_layers[g]) {
      const Layer& L = ctx->layers[li];
      FactMember M;
      std::memset(&M, 0, sizeof(M));
      member_layer.push_back(li);
      M.B = L.B;
      M.P_out = L.P_out;
      M.d_out = L.d_out;
      M.k_in = L.k_in;
      M.k_out = L.k_out;
      M.a_tile0 = na;
      M.na = tiles16(L.k_in);
      M.nb = tiles16(L.k_out);
      for (int t = 0; t < M.na; ++t) {
        G.ptile[na + t] = L.P_in;
        G.ptile_local[na + t] = t;
        G.ptile_nt[na + t] = M.na;
      }
      na += M.na;
      bytes_per_row += L.d_out;
      P.members.push_back(M);
    }
    G.na = na;
    G.aligned = aligned;
    for (int m = 0; m < G.n_members; ++m) P.members[G.member0 + m].aligned = aligned;
    const int na_inst = gshape[g].na_inst, nb_inst = gshape[g].nb_inst;
    G.chunk_rows = gshape[g].chunk_rows;
    G.n_chunks = gshape[g].n_chunks;
    // partial blocks of each member: [n][n_chunks * waves][na*16 x nb*16]
    for (int m = 0; m < G.n_members; ++m) {
      FactMember& M = P.members[G.member0 + m];
      M.partial_base = (int64_t)fpart_floats;
      const int64_t part = (int64_t)M.na * 16 * M.nb * 16;
      fpart_floats += (size_t)n * G.n_chunks * kWaves * part;
      ReduceTask R;
      std::memset(&R, 0, sizeof(R));
      R.partial_base = M.partial_base;
      R.phi_offset = ctx->layers[group_layers[g][m]].offset;
      R.n_parts = G.n_chunks * kWaves;
      R.k_in = M.k_in;
      R.k_out = M.k_out;
      R.ldp = M.nb * 16;
      R.part_floats = (int32_t)part;
      R.ex_begin = 0;
      P.tasks.push_back(R);
      P.fact_max_out = std::max(P.fact_max_out, M.k_in * M.k_out);
    }
    int inst = -1;
    for (size_t i = 0; i < insts.size(); ++i)
      if (insts[i].na == na_inst && insts[i].nb == nb_inst && insts[i].aligned == (int)aligned)
        inst = (int)i;
    if (inst < 0) {
      insts.push_back({na_inst, nb_inst, (int)aligned, {}});
      inst = (int)insts.size() - 1;
    }
    insts[inst].groups.push_back(fg);
    group_cost.push_back((double)n * H.T * bytes_per_row);
    P.groups.push_back(G);
  }
  P.n_fact_tasks = (int)P.tasks.size();
  // One launch per kernel instance.  Inside a launch, every item of a group
  // runs on one XCD (its projection maps then stay in that XCD's L2).  Groups
  // of one launch that read the same input block (layers kept apart above,
  // e.g. q/k/v) form a unit: the unit goes to one XCD with its items
  // interleaved per (example, chunk), so the workgroups that read the same A
  // rows run side by side and share them through that XCD's L2.  Units are
  // dealt by the bytes their workgroups stream (A counted per group: an L2
  // hit still crosses from L2 to the CU), costliest first, to the
  // least-loaded of 8 per-XCD queues, and the queues are interleaved so that
  // position 8*s + x holds queue x's s-th item (workgroups are dispatched
  // round-robin over the XCDs).  Short queues are padded with items that exit
  // at once.  Launches with fewer than 4 units per XCD spread their items over
  // all XCDs instead (a few groups would otherwise leave XCDs idle).
  for (const Inst& I : insts) {
    std::vector<std::vector<int>> units;
    std::vector<double> unit_cost;
    for (int g : I.groups) {
      const FactGroup& G = P.groups[g];
      size_t u = 0;
      for (; u < units.size(); ++u) {
        const FactGroup& H = P.groups[units[u][0]];
        if (H.A == G.A && H.d_in == G.d_in && H.T == G.T && H.lengths == G.lengths &&
            H.n_chunks == G.n_chunks && H.chunk_rows == G.chunk_rows)
          break;
      }
      if (u == units.size()) {
        units.push_back({});
        unit_cost.push_back(0.0);
      }
      units[u].push_back(g);
      unit_cost[u] += group_cost[g];
    }
    std::vector<int> order(units.size());
    for (size_t u = 0; u < units.size(); ++u) order[u] = (int)u;
    if (units.size() < (size_t)4 * kXcds) {
      // too few units to keep every XCD busy with whole units: the items of a
      // unit, interleaved as above, spread over all XCDs
      const int first = (int)P.items.size();
      for (int u : order) {
        const FactGroup& H = P.groups[units[u][0]];
        for (int e = 0; e < n; ++e)
          for (int c = 0; c < H.n_chunks; ++c)
            for (int g : units[u]) P.items.push_back({g, e, c, 0});
      }
      P.launches.push_back({elt, I.na, I.nb, I.aligned, first, (int)P.items.size() - first});
      continue;
    }
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return unit_cost[a] > unit_cost[b]; });
    std::vector<std::vector<FactItem>> q(kXcds);
    double load[kXcds] = {0};
    for (int u : order) {
      const int x = (int)(std::min_element(load, load + kXcds) - load);
      const FactGroup& H = P.groups[units[u][0]];
      for (int e = 0; e < n; ++e)
        for (int c = 0; c < H.n_chunks; ++c)
          for (int g : units[u]) q[x].push_back({g, e, c, 0});
      load[x] += unit_cost[u];
    }
    size_t len = 0;
    for (const auto& v : q) len = std::max(len, v.size());
    const int first = (int)P.items.size();
    for (size_t s = 0; s < len; ++s)
      for (int x = 0; x < kXcds; ++x)
        P.items.push_back(s < q[x].size() ? q[x][s] : FactItem{0, -1, 0, 0});
    P.launches.push_back({elt, I.na, I.nb, I.aligned, first, (int)P.items.size() - first});
  }

  // ---- split form: one stage-1 op per factor block (a group's A, each
  // member's B) over all n*T token rows; one contraction task per layer.
  if (!split_groups.empty()) {
    struct Pending { int a_op, b_op; };
    std::vector<Pending> pend;
    const size_t op0 = P.sops.size();
    for (size_t g : split_groups) {
      const Layer& H = ctx->layers[group_layers[g][0]];
      const int rows = n * H.T;
      SplitOp A;
      std::memset(&A, 0, sizeof(A));
      A.X = H.A;
      A.rows = rows;
      A.ld = H.d_in;
      A.aligned = ((uintptr_t)H.A % 16 == 0) && (H.d_in * elt) % 16 == 0;
      std::vector<SplitOp> Bs;
      int na = 0;
      const int a_op = (int)P.sops.size();
      for (int li : group_layers[g]) {
        const Layer& L = ctx->layers[li];
        const int mt = tiles16(L.k_in);
        for (int t = 0; t < mt; ++t) {
          A.ptile[na + t] = L.P_in;
          A.ptile_local[na + t] = t;
          A.ptile_nt[na + t] = mt;
        }
        SplitOp B;
        std::memset(&B, 0, sizeof(B));
        B.X = L.B;
        B.rows = rows;
        B.ld = L.d_out;
        B.aligned = ((uintptr_t)L.B % 16 == 0) && (L.d_out * elt) % 16 == 0;
        B.nt = tiles16(L.k_out);
        for (int t = 0; t < B.nt; ++t) {
          B.ptile[t] = L.P_out;
          B.ptile_local[t] = t;
          B.ptile_nt[t] = B.nt;
        }
        ContractTask C;
        std::memset(&C, 0, sizeof(C));
        C.a_col0 = na * 16;
        C.k_in = L.k_in;
        C.k_out = L.k_out;
        C.T = H.T;
        C.rows = rows;
        C.phi_offset = L.offset;
        C.lengths = L.lengths;
        P.ctasks.push_back(C);
        pend.push_back({a_op, a_op + 1 + (int)Bs.size()});
        split_rows.push_back({li, a_op, a_op + 1 + (int)Bs.size(), na * 16});
        Bs.push_back(B);
        na += mt;
      }
      A.nt = na;
      P.sops.push_back(A);
      for (const SplitOp& B : Bs) P.sops.push_back(B);
    }
    // slab width: about kSplitTargetItems stage-1 workgroups in total
    int64_t work = 0;
    for (size_t o = op0; o < P.sops.size(); ++o)
      work += (int64_t)((P.sops[o].rows + split_rows_of(split_nt_instance(P.sops[o].nt)) - 1) /
                        split_rows_of(split_nt_instance(P.sops[o].nt))) * P.sops[o].ld;
    int64_t slab = (work + kSplitTargetItems - 1) / kSplitTargetItems;
    slab = std::max<int64_t>(kSplitSlabQuantum, (slab + kSplitSlabQuantum - 1) / kSplitSlabQuantum * kSplitSlabQuantum);
    size_t proj_floats = 0;
    for (size_t o = op0; o < P.sops.size(); ++o) {
      SplitOp& O = P.sops[o];
      O.slab_cols = (int32_t)std::min<int64_t>(slab, (O.ld + kSplitSlabQuantum - 1) / kSplitSlabQuantum * kSplitSlabQuantum);
      O.n_slabs = (O.ld + O.slab_cols - 1) / O.slab_cols;
      O.out_base = (int64_t)proj_floats;
      proj_floats += (size_t)O.n_slabs * O.rows * O.nt * 16;
    }
    // token chunks: about kContractTargetItems stage-2 workgroups in total
    const int64_t per_chunk = (int64_t)pend.size() * std::max(n, 1);
    const int64_t want_chunks = std::max<int64_t>(1, (kContractTargetItems + per_chunk - 1) / per_chunk);
    size_t spart_floats = 0;
    for (size_t i = 0; i < pend.size(); ++i) {
      ContractTask& C = P.ctasks[P.ctasks.size() - pend.size() + i];
      const SplitOp& A = P.sops[pend[i].a_op];
      const SplitOp& B = P.sops[pend[i].b_op];
      // slabs are summed into slab 0 before the contraction
      C.a_base = A.out_base; C.a_ld = A.nt * 16; C.a_slabs = 1;
      C.b_base = B.out_base; C.b_ld = B.nt * 16; C.b_slabs = 1;
      const int64_t tc = (C.T + want_chunks - 1) / want_chunks;
      C.tok_chunk = (int32_t)std::max<int64_t>(64, (tc + 31) / 32 * 32);
      C.n_tchunks = std::max(1, (C.T + C.tok_chunk - 1) / C.tok_chunk);
      P.split_max_tchunks = std::max(P.split_max_tchunks, C.n_tchunks);
      if (C.n_tchunks > 1) {
        const int ki16 = tiles16(C.k_in) * 16, ko16 = tiles16(C.k_out) * 16;
        C.partial_base = (int64_t)spart_floats;
        spart_floats += (size_t)n * C.n_tchunks * ki16 * ko16;
        ReduceTask R;
        std::memset(&R, 0, sizeof(R));
        R.partial_base = C.partial_base;
        R.phi_offset = C.phi_offset;
        R.n_parts = C.n_tchunks;
        R.k_in = C.k_in;
        R.k_out = C.k_out;
        R.ldp = ko16;
        R.part_floats = ki16 * ko16;
        R.ex_begin = 0;
        P.stasks.push_back(R);
        P.split_max_out = std::max(P.split_max_out, C.k_in * C.k_out);
      }
    }
    P.proj_bytes = proj_floats * 4;
    P.spart_bytes = spart_floats * 4;
    for (size_t o = op0; o < P.sops.size(); ++o) {
      const SplitOp& O = P.sops[o];
      if (O.n_slabs <= 1 || O.rows == 0) continue;
      SlabSumTask T;
      std::memset(&T, 0, sizeof(T));
      T.base = O.out_base;
      T.n4 = (int64_t)O.rows * O.nt * 4;
      T.stride4 = T.n4;
      T.n_slabs = O.n_slabs;
      P.slabsum.push_back(T);
      P.slabsum_max_n4 = std::max(P.slabsum_max_n4, T.n4);
    }
    // One launch per kernel instance (aligned, tiles).  Inside a launch, the
    // items of one op run on one XCD, so its projection map is fetched into
    // that XCD's L2 once and read there by all its row blocks: ops (units of
    // ops over the same block) are dealt, costliest first, to the
    // least-loaded of 8 per-XCD queues and the queues interleaved (workgroup i
    // runs on XCD i mod 8); short queues are padded with items that exit at
    // once.  Launches with fewer than 4 units per XCD keep the items in op
    // order over all XCDs (a few wide layers would otherwise leave XCDs idle).
    for (int al = 1; al >= 0; --al)
      for (int nt : {1, 2, 4, 8}) {
        std::vector<size_t> ops;
        for (size_t o = op0; o < P.sops.size(); ++o)
          if (P.sops[o].aligned == al && split_nt_instance(P.sops[o].nt) == nt) ops.push_back(o);
        if (ops.empty()) continue;
        // ops that stream the same block (the input of layers kept apart, e.g.
        // q/k/v) form a unit whose items are interleaved per (row block,
        // slab), so the side-by-side workgroups share its rows through L2
        std::vector<std::vector<size_t>> units;
        for (size_t o : ops) {
          const SplitOp& O = P.sops[o];
          size_t u = 0;
          for (; u < units.size(); ++u) {
            const SplitOp& H = P.sops[units[u][0]];
            if (H.X == O.X && H.rows == O.rows && H.ld == O.ld && H.n_slabs == O.n_slabs &&
                H.slab_cols == O.slab_cols)
              break;
          }
          if (u == units.size()) units.push_back({});
          units[u].push_back(o);
        }
        const int rows_wg = split_rows_of(nt);
        const int first = (int)P.sitems.size();
        if (units.size() < (size_t)4 * kXcds) {
          // too few units to keep every XCD busy with whole units: items in op
          // order, spread over all XCDs
          for (size_t o : ops) {
            const SplitOp& O = P.sops[o];
            const int rblocks = (O.rows + rows_wg - 1) / rows_wg;
            for (int rb = 0; rb < rblocks; ++rb)
              for (int sl = 0; sl < O.n_slabs; ++sl) P.sitems.push_back({(int)o, rb, sl, 0});
          }
          P.slaunches.push_back({elt, al, nt, first, (int)P.sitems.size() - first});
          continue;
        }
        auto cost = [&](const std::vector<size_t>& u) {  // every op's workgroups stream the block
          return (double)P.sops[u[0]].rows * P.sops[u[0]].ld * (double)u.size();
        };
        std::stable_sort(units.begin(), units.end(),
                         [&](const std::vector<size_t>& a, const std::vector<size_t>& b) { return cost(a) > cost(b); });
        std::vector<std::vector<SplitItem>> q(kXcds);
        double load[kXcds] = {0};
        for (const auto& u : units) {
          const SplitOp& O = P.sops[u[0]];
          const int x = (int)(std::min_element(load, load + kXcds) - load);
          const int rblocks = (O.rows + rows_wg - 1) / rows_wg;
          for (int rb = 0; rb < rblocks; ++rb)
            for (int sl = 0; sl < O.n_slabs; ++sl)
              for (size_t o : u) q[x].push_back({(int)o, rb, sl, 0});
          load[x] += cost(u);
        }
        size_t len = 0;
        for (const auto& v : q) len = std::max(len, v.size());
        for (size_t i = 0; i < len; ++i)
          for (int x = 0; x < kXcds; ++x)
            P.sitems.push_back(i < q[x].size() ? q[x][i] : SplitItem{-1, 0, 0, 0});
        const int count = (int)P.sitems.size() - first;
        if (count) P.slaunches.push_back({elt, al, nt, first, count});
      }
  }

  // ---- materialized layers: example chunks staged through G
  size_t g_floats = 0, mpart_floats = 0;
  for (size_t l = 0; l < ctx->layers.size(); ++l) {
    const Layer& L = ctx->layers[l];
    if (route[l] != DATTRI_ROUTE_MATERIALIZED) continue;
    if (fused_materialized(L, elt)) {  // one pass, G on chip: partial blocks per (row block, token chunk)
      const FusedShape fs = fused_shape(L, n, ctx->cost);
      const int n_ublocks = (L.d_out + kGFusedRows - 1) / kGFusedRows;
      const int ex_chunk = std::min(n, 65535);
      const int64_t part = (int64_t)tiles16(L.k_in) * 16 * tiles16(L.k_out) * 16;
      const int64_t parts = (int64_t)n_ublocks * fs.n_vsplit * fs.n_tchunks;
      mpart_floats = std::max(mpart_floats, (size_t)((int64_t)ex_chunk * parts * part));
      for (int e0 = 0; e0 < n; e0 += ex_chunk) {
        MatChunk mc{(int)l, e0, std::min(ex_chunk, n - e0), n_ublocks, 1, 0, (int)P.tasks.size()};
        mc.fused = 1;
        mc.n_tchunks = fs.n_tchunks;
        mc.tok_chunk = fs.tok_chunk;
        mc.n_vsplit = fs.n_vsplit;
        mc.vt_per_split = fs.vt_per_split;
        ReduceTask R;
        std::memset(&R, 0, sizeof(R));
        R.partial_base = 0;
        R.phi_offset = L.offset;
        R.n_parts = (int32_t)parts;
        R.k_in = L.k_in;
        R.k_out = L.k_out;
        R.ldp = tiles16(L.k_out) * 16;
        R.part_floats = (int32_t)part;
        R.ex_begin = e0;
        P.tasks.push_back(R);
        P.mat.push_back(mc);
      }
      continue;
    }
    const int64_t g_per_ex = (int64_t)L.d_out * L.d_in;
    if (4 * g_per_ex >= kMaxBlockBytes)
      return fail(DATTRI_E_UNSUPPORTED, "layer %zu: G = d_out x d_in float32 (%lld bytes) exceeds 4 GiB",
                  l, (long long)(4 * g_per_ex));
    const int ex_chunk = (int)materialized_chunk(L, n);
    const int n_ublocks = (L.d_out + kGProjRows - 1) / kGProjRows;
    // split d_in's k-blocks when row blocks x examples give too few workgroups
    const int nkb = (L.d_in + krows_of(elt) - 1) / krows_of(elt);
    const int64_t want = (kGProjTargetBlocks + (int64_t)n_ublocks * ex_chunk - 1) / ((int64_t)n_ublocks * ex_chunk);
    const int ks_req = (int)std::max<int64_t>(1, std::min<int64_t>(nkb, want));
    const int kbps = (nkb + ks_req - 1) / ks_req;
    const int n_ks = (nkb + kbps - 1) / kbps;
    const int64_t part = (int64_t)tiles16(L.k_in) * 16 * tiles16(L.k_out) * 16;
    g_floats = std::max(g_floats, (size_t)(ex_chunk * g_per_ex));
    mpart_floats = std::max(mpart_floats, (size_t)((int64_t)ex_chunk * n_ublocks * n_ks * part));
    for (int e0 = 0; e0 < n; e0 += ex_chunk) {
      MatChunk mc{(int)l, e0, std::min(ex_chunk, n - e0), n_ublocks, n_ks, kbps, (int)P.tasks.size()};
      ReduceTask R;
      std::memset(&R, 0, sizeof(R));
      R.partial_base = 0;
      R.phi_offset = L.offset;
      R.n_parts = n_ublocks * n_ks;
      R.k_in = L.k_in;
      R.k_out = L.k_out;
      R.ldp = tiles16(L.k_out) * 16;
      R.part_floats = (int32_t)part;
      R.ex_begin = e0;
      P.tasks.push_back(R);
      P.mat.push_back(mc);
    }
  }

  // ---- mask layers: (example, token chunk, entry group) work items
  {
    size_t mask_floats = 0;
    int64_t units = 0;  // example x entry-group pairs over all mask layers
    for (const Layer& L : ctx->layers)
      if (L.mask_size > 0) units += (int64_t)n * ((L.k_out + kMaskGroup - 1) / kMaskGroup);
    const int64_t want_chunks = units > 0 ? std::max<int64_t>(1, (2048 + units - 1) / units) : 1;
    for (size_t l = 0; l < ctx->layers.size(); ++l) {
      const Layer& L = ctx->layers[l];
      if (L.mask_size <= 0) continue;
      const int64_t row_bytes = (int64_t)(L.d_in + L.d_out) * elt;
      if (row_bytes + 2048 > 80 * 1024)
        return fail(DATTRI_E_UNSUPPORTED, "layer %zu: mask layers need (d_in + d_out) * %d <= 78 KiB", l, elt);
      MaskTask M;
      std::memset(&M, 0, sizeof(M));
      M.A = L.A; M.B = L.B; M.lengths = L.lengths;
      M.rows = (const int32_t*)L.P_in;
      M.cols = (const int32_t*)L.P_in + L.k_out;
      M.pos = (const int32_t*)L.P_in + 2 * (int64_t)L.k_out;
      M.slices = (const int32_t*)L.P_in + 3 * (int64_t)L.k_out;
      M.d_in = L.d_in; M.d_out = L.d_out; M.T = L.T; M.m = L.k_out;
      M.stage_tokens = (int)std::max<int64_t>(1, std::min<int64_t>(16, kMaskStageBudget / row_bytes));
      const int64_t tc = (L.T + want_chunks - 1) / want_chunks;
      M.chunk_tokens = (int)std::max<int64_t>(M.stage_tokens, (tc + M.stage_tokens - 1) / M.stage_tokens * M.stage_tokens);
      M.n_chunks = std::max(1, (L.T + M.chunk_tokens - 1) / M.chunk_tokens);
      M.aligned = ((uintptr_t)L.A % 16 == 0) && ((uintptr_t)L.B % 16 == 0) && (L.d_in * elt) % 16 == 0 &&
                  (L.d_out * elt) % 16 == 0;
      // whole groups take the fixed-slot gather when every one's slices fit a slot
      // (and each example's factor blocks below 2 GiB: its chunk offsets past a
      // slice start at 2^31)
      M.fixed = M.aligned && L.mask_slices.size() >= (size_t)4 * (L.k_out / kMaskGroup) &&  // bound
                (int64_t)L.T * std::max(L.d_in, L.d_out) * elt < ((int64_t)1 << 31) &&
                mask_fixed_layout(elt, L.d_in, L.d_out, L.k_out, L.mask_slices.data());
      M.partial_base = (int64_t)mask_floats;
      mask_floats += (size_t)n * M.n_chunks * M.m;
      // aligned: two buffers of [A part | B part], parts rounded up to 1 KiB; else one buffer
      const int64_t a_part = ((int64_t)M.stage_tokens * L.d_in * elt + 1023) & ~(int64_t)1023;
      const int64_t b_part = ((int64_t)M.stage_tokens * L.d_out * elt + 1023) & ~(int64_t)1023;
      const size_t lds = (size_t)(M.aligned ? 2 * (a_part + b_part) : a_part + b_part);
      P.mask_lds = std::max(P.mask_lds, lds);
      P.mask_b16 = P.mask_b16 && elt == 2 && L.d_in <= 32768 && L.d_out <= 32768;
      ReduceTask R;
      std::memset(&R, 0, sizeof(R));
      R.partial_base = M.partial_base;
      R.phi_offset = L.offset;
      R.n_parts = M.n_chunks;
      R.k_in = 1;
      R.k_out = M.m;
      R.ldp = M.m;
      R.part_floats = M.m;
      P.mreduce.push_back(R);
      P.mask_max_out = std::max(P.mask_max_out, M.m);
      P.mtasks.push_back(M);
    }
    // Every entry group of one (layer, example, token chunk) stages the same
    // token rows: the groups of a chunk go to one XCD, back to back, so they
    // run together and share the rows through that XCD's L2.  Chunks are dealt
    // to the least-loaded of 8 per-XCD queues and the queues interleaved
    // (workgroup i runs on XCD i mod 8); short queues are padded.
    // One launch per (alignment, whole groups or not, fixed slots or not): a
    // whole group of kMaskGroup entries takes the gather without slot bounds,
    // and the fixed-slot one when its task allows.
    for (int al = 1; al >= 0; --al)
      for (int full = 1; full >= 0; --full)
        for (int fx = full && al ? 1 : 0; fx >= 0; --fx) {
          std::vector<std::vector<MaskItem>> q(kXcds);
          int64_t load[kXcds] = {0};
          for (size_t t = 0; t < P.mtasks.size(); ++t) {
            const MaskTask& M = P.mtasks[t];
            if (M.aligned != al || (full && M.fixed != fx)) continue;
            const int whole = M.m / kMaskGroup, groups = (M.m + kMaskGroup - 1) / kMaskGroup;
            const int g0 = full ? 0 : whole, g1 = full ? whole : groups;
            if (g1 <= g0) continue;
            for (int e = 0; e < n; ++e)
              for (int c = 0; c < M.n_chunks; ++c) {
                const int x = (int)(std::min_element(load, load + kXcds) - load);
                for (int g = g0; g < g1; ++g) q[x].push_back({(int)t, e, c, g});
                load[x] += g1 - g0;
              }
          }
          size_t len = 0;
          for (const auto& v : q) len = std::max(len, v.size());
          const int first = (int)P.mitems.size();
          for (size_t i = 0; i < len; ++i)
            for (int x = 0; x < kXcds; ++x)
              P.mitems.push_back(i < q[x].size() ? q[x][i] : MaskItem{-1, 0, 0, 0});
          const int count = (int)P.mitems.size() - first;
          if (count) P.mlaunches.push_back({al, full, fx, first, count});
        }
    P.maskpart_bytes = mask_floats * 4;
  }

  // ---- workspace layout
  size_t off = 0;
  P.off_items = off;   off = align_up(off + P.items.size() * sizeof(FactItem));
  P.off_groups = off;  off = align_up(off + P.groups.size() * sizeof(FactGroup));
  P.off_members = off; off = align_up(off + P.members.size() * sizeof(FactMember));
  P.off_tasks = off;   off = align_up(off + P.tasks.size() * sizeof(ReduceTask));
  P.off_sops = off;    off = align_up(off + P.sops.size() * sizeof(SplitOp));
  P.off_sitems = off;  off = align_up(off + P.sitems.size() * sizeof(SplitItem));
  P.off_ctasks = off;  off = align_up(off + P.ctasks.size() * sizeof(ContractTask));
  P.off_stasks = off;  off = align_up(off + P.stasks.size() * sizeof(ReduceTask));
  P.off_slabsum = off; off = align_up(off + P.slabsum.size() * sizeof(SlabSumTask));
  P.off_mtasks = off;  off = align_up(off + P.mtasks.size() * sizeof(MaskTask));
  P.off_mitems = off;  off = align_up(off + P.mitems.size() * sizeof(MaskItem));
  P.off_mreduce = off; off = align_up(off + P.mreduce.size() * sizeof(ReduceTask));
  P.blob_bytes = off;
  P.off_fpart = off;   P.fpart_bytes = fpart_floats * 4; off = align_up(off + P.fpart_bytes);
  P.off_g = off;       P.g_bytes = g_floats * 4;         off = align_up(off + P.g_bytes);
  P.off_mpart = off;   P.mpart_bytes = mpart_floats * 4; off = align_up(off + P.mpart_bytes);
  P.off_proj = off;    off = align_up(off + P.proj_bytes);
  P.off_spart = off;   off = align_up(off + P.spart_bytes);
  P.off_maskpart = off; off = align_up(off + P.maskpart_bytes);
  // projected token rows of the fused members, and where every factored
  // layer side's rows sit (split form: slab 0 of its stage-1 op)
  P.rows = rows;
  if (rows) {
    P.off_rows = off;
    size_t r = 0;
    P.member_rows.assign(2 * P.members.size(), 0);
    for (const FactGroup& G : P.groups)
      for (int m = 0; m < G.n_members; ++m) {
        const int mi = G.member0 + m;
        const FactMember& M = P.members[mi];
        const size_t a = align_up(r + (size_t)n * G.T * M.k_in * 4);
        P.member_rows[2 * mi] = P.off_rows + r;
        P.member_rows[2 * mi + 1] = P.off_rows + a;
        r = align_up(a + (size_t)n * G.T * M.k_out * 4);
        P.row_srcs.push_back({member_layer[mi], 0, P.member_rows[2 * mi], M.k_in, 0});
        P.row_srcs.push_back({member_layer[mi], 1, P.member_rows[2 * mi + 1], M.k_out, 0});
      }
    P.rows_bytes = r;
    off = align_up(off + r);
    for (const SplitRows& R : split_rows) {
      const SplitOp& A = P.sops[R.a_op];
      const SplitOp& B = P.sops[R.b_op];
      P.row_srcs.push_back({R.layer, 0, P.off_proj + (size_t)A.out_base * 4, A.nt * 16, R.a_col0});
      P.row_srcs.push_back({R.layer, 1, P.off_proj + (size_t)B.out_base * 4, B.nt * 16, 0});
    }
    for (size_t l = 0; l < ctx->layers.size(); ++l)
      if (route[l] == DATTRI_ROUTE_MATERIALIZED) P.mat_layers.push_back((int)l);
  }
  P.total = std::max<size_t>(off, kAlign);
  return DATTRI_OK;
}

namespace {

// Everything build_plan reads from the context, as one flat key: a plan built
// from an equal key is the same plan.
std::vector<uint64_t> plan_key(const dattri_ctx* ctx, dattri_route forced, bool rows) {
  std::vector<uint64_t> k;
  k.reserve(16 + 10 * ctx->layers.size());
  auto pack = [](int64_t hi, int64_t lo) { return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo; };
  auto ptr = [](const void* p) { return (uint64_t)(uintptr_t)p; };
  k.push_back(pack(forced, rows));
  k.push_back(pack(ctx->form, ctx->elt));
  uint64_t words[sizeof(dattri_cost_model) / 8];
  static_assert(sizeof(dattri_cost_model) % 8 == 0, "cost model is a plain array of doubles");
  std::memcpy(words, &ctx->cost, sizeof(words));
  k.insert(k.end(), words, words + sizeof(words) / 8);
  for (const Layer& L : ctx->layers) {
    k.push_back(pack(L.d_in, L.d_out));
    k.push_back(pack(L.k_in, L.k_out));
    k.push_back(pack(L.mask_size, L.mask_id));
    k.push_back(pack(L.mask_count, L.n));
    k.push_back(pack(L.T, (L.captured ? 2 : 0) | (L.bound ? 1 : 0)));
    k.push_back(ptr(L.A));
    k.push_back(ptr(L.B));
    k.push_back(ptr(L.lengths));
    k.push_back(ptr(L.P_in));
    k.push_back(ptr(L.P_out));
  }
  return k;
}

constexpr size_t kPlansKept = 4;  // recent plans remembered per context

}  // namespace

dattri_status dattri::get_plan(const dattri_ctx* ctx, dattri_route forced, bool rows,
                               std::shared_ptr<const Plan>* out) {
  std::vector<uint64_t> key = plan_key(ctx, forced, rows);
  auto& kept = ctx->plans;
  for (size_t i = 0; i < kept.size(); ++i)
    if (kept[i].first == key) {
      std::rotate(kept.begin(), kept.begin() + i, kept.begin() + i + 1);  // most recent first
      *out = kept.front().second;
      return DATTRI_OK;
    }
  auto P = std::make_shared<Plan>();
  const dattri_status st = build_plan(ctx, forced, *P, rows);
  if (st != DATTRI_OK) return st;
  kept.insert(kept.begin(), {std::move(key), P});
  if (kept.size() > kPlansKept) kept.pop_back();
  *out = P;
  return DATTRI_OK;
}

hipError_t dattri::place_table(const dattri_ctx* ctx, TableKind kind, const std::vector<uint8_t>& blob,
                               uint8_t* fallback, hipStream_t s, uint8_t** dev) {
  *dev = fallback;
  if (blob.empty()) return hipSuccess;
  const size_t need = align_up(blob.size());
  if (!ctx->plan_buf || need > ctx->plan_cap) {
    ctx->blob = blob;
    return hipMemcpyAsync(fallback, ctx->blob.data(), blob.size(), hipMemcpyHostToDevice, s);
  }
  TableSlot* slot = nullptr;
  for (TableSlot& t : ctx->slots)
    if (t.kind == kind) slot = &t;
  if (slot && slot->bytes == blob) {  // already resident: no copy
    *dev = ctx->plan_buf + slot->off;
    return hipSuccess;
  }
  if (!slot || slot->cap < need) {
    // a new slot at the end of the buffer; when the buffer is full, every
    // table is dropped and placement starts again at its head
    if (slot) slot->kind = -1;
    if (ctx->slots_used + need > ctx->plan_cap) {
      ctx->slots.clear();
      ctx->slots_used = 0;
    }
    ctx->slots.emplace_back();
    slot = &ctx->slots.back();
    slot->kind = kind;
    slot->off = ctx->slots_used;
    slot->cap = need;
    ctx->slots_used += need;
  }
  slot->bytes = blob;
  *dev = ctx->plan_buf + slot->off;
  const hipError_t e = hipMemcpyAsync(*dev, slot->bytes.data(), blob.size(), hipMemcpyHostToDevice, s);
  if (e != hipSuccess) slot->bytes.clear();  // contents unknown: never matched
  return e;
}

// Whether a mask layer's whole groups take the fixed-slot gather (bf16 rows
// of whole 16-byte chunks, every whole group's A and B slices at most
// kMaskSlot bytes); slices as in the layer's entry table.  The planner adds
// the captures' alignment.
bool dattri::mask_fixed_layout(int elt, int d_in, int d_out, int m, const int32_t* slices) {
  if (elt != 2 || (d_in * elt) % 16 || (d_out * elt) % 16 || m < kMaskGroup) return false;
  for (int g = 0; g < m / kMaskGroup; ++g)
    if (slices[4 * g + 1] > kMaskSlot || slices[4 * g + 3] > kMaskSlot) return false;
  return true;
}

namespace {

dattri_status check_layer(const dattri_ctx* ctx, int32_t layer) {
  if (!ctx) return fail(DATTRI_E_INVALID_ARG, "ctx is NULL");
  if (layer < 0 || layer >= (int32_t)ctx->layers.size())
    return fail(DATTRI_E_INVALID_ARG, "layer %d out of range [0, %zu)", layer, ctx->layers.size());
  return DATTRI_OK;
}

// Device entry table of a mask layer: [rows | cols | pos], int32, m each,
// then 4 int32 per entry group: the byte slice of each A token row (first
// byte, length) and of each B token row covering the group's columns and rows,
// both ends on 16-byte boundaries (the row's end for rows that are not a
// multiple of 16 bytes).
// Entries are placed into the gather kernel's slots group by group (groups of
// kMaskGroup entries; slot e of a group is read by thread e % W at step
// e / W for W = 256 or 512 threads, so slots 32h .. 32h + 31 form the
// half-wave h of one LDS read).
// A layer with more than one group deals its entries to the groups in order
// of their index on the wider side of DW (rows when d_out >= d_in, else
// columns; equal indices in mask order): each group's entries then span about
// 1/groups of that side, and the kernel stages only that slice of each token
// row instead of the whole row.  Inside a group, each entry goes to the first
// half-wave where neither its A word nor its B word meets another word in the
// same bank (32 banks of 4 bytes; a word already there is read once for all
// its lanes), else one where one of the two does not, else any with room; so
// most gathers are free of bank conflicts.  The words are those the group's
// kernel reads: a 4-byte token pair per feature for the fixed-slot gather
// (mask_fixed_layout), the element's own word otherwise.  pos[slot] is the
// entry's index in mask order, where the kernel writes its sum.
void mask_slot_table(const std::vector<int32_t>& rows, const std::vector<int32_t>& cols, int d_in, int d_out,
                     int elt, std::vector<int32_t>& table) {
  const int m = (int)rows.size(), n_groups = (m + kMaskGroup - 1) / kMaskGroup;
  table.assign((size_t)3 * m + 4 * (size_t)n_groups, 0);
  int32_t* t_rows = table.data();
  int32_t* t_cols = table.data() + m;
  int32_t* t_pos = table.data() + 2 * (size_t)m;
  std::vector<int32_t> order((size_t)m);
  for (int i = 0; i < m; ++i) order[i] = i;
  if (m > kMaskGroup) {
    const std::vector<int32_t>& key = d_out >= d_in ? rows : cols;
    std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return key[a] < key[b]; });
  }
  int32_t* slices = table.data() + 3 * (size_t)m;
  for (int g = 0; g < n_groups; ++g) {
    const int e0 = g * kMaskGroup, N = std::min(kMaskGroup, m - e0);
    int32_t lo_r = d_out, hi_r = -1, lo_c = d_in, hi_c = -1;
    for (int i = 0; i < N; ++i) {
      const int32_t e = order[e0 + i];
      lo_r = std::min(lo_r, rows[e]); hi_r = std::max(hi_r, rows[e]);
      lo_c = std::min(lo_c, cols[e]); hi_c = std::max(hi_c, cols[e]);
    }
    auto slice = [&](int32_t lo, int32_t hi, int d, int32_t* out) {
      const int64_t b0 = ((int64_t)lo * elt) & ~(int64_t)15;
      const int64_t b1 = std::min(((int64_t)(hi + 1) * elt + 15) & ~(int64_t)15, (int64_t)d * elt);
      out[0] = (int32_t)b0;
      out[1] = (int32_t)(b1 - b0);
    };
    slice(lo_c, hi_c, d_in, slices + 4 * g);
    slice(lo_r, hi_r, d_out, slices + 4 * g + 2);
  }
  const bool pairs = mask_fixed_layout(elt, d_in, d_out, m, slices);
  constexpr int kHalf = 32, kMaxHalves = kMaskGroup / kHalf, kW = kMaxHalves / 64;
  struct Bits {
    uint64_t w[kW];
  };
  auto first = [](const Bits& x) {
    for (int i = 0; i < kW; ++i)
      if (x.w[i]) return i * 64 + __builtin_ctzll(x.w[i]);
    return -1;
  };
  // per factor side: word -> index into `holders` (the half-waves holding that word)
  std::vector<int32_t> slot_of[2] = {std::vector<int32_t>((size_t)d_in, -1), std::vector<int32_t>((size_t)d_out, -1)};
  std::vector<Bits> holders[2];
  std::vector<int32_t> touched[2];
  for (int e0 = 0; e0 < m; e0 += kMaskGroup) {
    const int N = std::min(kMaskGroup, m - e0), H = (N + kHalf - 1) / kHalf;
    // fixed-slot groups read one word per feature (a token pair, placed by
    // mask_pair_offset), others the word holding the element
    const bool pw = pairs && N == kMaskGroup;
    Bits all{};
    for (int h = 0; h < H; ++h) all.w[h >> 6] |= 1ull << (h & 63);
    Bits free_bank[2][kHalf], room = all;
    for (int side = 0; side < 2; ++side)
      for (int b = 0; b < kHalf; ++b) free_bank[side][b] = all;
    int fill[kMaxHalves] = {0};
    for (int i = 0; i < N; ++i) {
      const int32_t e = order[e0 + i];
      const int32_t word[2] = {pw ? cols[e] : (int32_t)(((int64_t)cols[e] * elt) >> 2),
                               pw ? rows[e] : (int32_t)(((int64_t)rows[e] * elt) >> 2)};
      // a slice starts on 16 bytes (8 features), so the banks of a group's
      // pair words are those of the absolute feature index, rotated alike
      int bank[2];
      for (int side = 0; side < 2; ++side)
        bank[side] = pw ? (int)(mask_pair_offset((uint32_t)word[side]) >> 2) % kHalf : word[side] % kHalf;
      Bits ok[2];
      for (int side = 0; side < 2; ++side) {
        ok[side] = free_bank[side][bank[side]];
        const int32_t hs = slot_of[side][word[side]];
        if (hs >= 0)
          for (int k = 0; k < kW; ++k) ok[side].w[k] |= holders[side][hs].w[k];
      }
      Bits both, one;
      for (int k = 0; k < kW; ++k) {
        both.w[k] = ok[0].w[k] & ok[1].w[k] & room.w[k];
        one.w[k] = (ok[0].w[k] | ok[1].w[k]) & room.w[k];
      }
      int h = first(both);
      if (h < 0) h = first(one);
      if (h < 0) h = first(room);
      const uint64_t bit = 1ull << (h & 63);
      const int slot = h * kHalf + fill[h]++;
      if (fill[h] == std::min(kHalf, N - h * kHalf)) room.w[h >> 6] &= ~bit;
      for (int side = 0; side < 2; ++side) {
        Bits& fb = free_bank[side][bank[side]];
        if (fb.w[h >> 6] & bit) {  // the bank was empty: this word now holds it
          fb.w[h >> 6] &= ~bit;
          int32_t& hs = slot_of[side][word[side]];
          if (hs < 0) {
            hs = (int32_t)holders[side].size();
            holders[side].push_back(Bits{});
            touched[side].push_back(word[side]);
          }
          holders[side][hs].w[h >> 6] |= bit;
        }
      }
      t_rows[e0 + slot] = rows[e];
      t_cols[e0 + slot] = cols[e];
      t_pos[e0 + slot] = e;
    }
    for (int side = 0; side < 2; ++side) {  // reset the word index for the next group
      for (int32_t w : touched[side]) slot_of[side][w] = -1;
      touched[side].clear();
      holders[side].clear();
    }
  }
}

void logical_map(const dattri_ctx* ctx, int layer, int side, std::vector<float>& out) {
  const Layer& L = ctx->layers[layer];
  const int d = side ? L.d_out : L.d_in, k = side ? L.k_out : L.k_in;
  const std::vector<float>& ov = side ? L.override_out : L.override_in;
  if (!ov.empty()) { out = ov; return; }
  out.resize((size_t)d * k);
  seeded_map(derive_side_seed(ctx->seed, layer, side), d, k, ctx->elt, L.map_kind, out.data());
}

}  // namespace

// =================================================================== C ABI
dattri_status dattri::run_plan(dattri_ctx* ctx, const Plan& P, void* phi, dattri_dtype phi_dtype,
                               int64_t ld_phi, void* workspace, size_t ws_bytes, hipStream_t s) {
  const int32_t n = ctx->layers[0].n;
  if (ld_phi < ctx->F) return fail(DATTRI_E_SHAPE, "ld_phi=%lld < F=%lld", (long long)ld_phi, (long long)ctx->F);
  if (n == 0) return DATTRI_OK;
  if (!phi) return fail(DATTRI_E_INVALID_ARG, "phi is NULL");
  if (!workspace) return fail(DATTRI_E_WORKSPACE, "workspace is NULL (needs %zu bytes)", P.total);
  if ((uintptr_t)workspace % kAlign) return fail(DATTRI_E_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < P.total)
    return fail(DATTRI_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, P.total);

  // The launch plan's tables: into the bound plan buffer, else the head of
  // the workspace.
  std::vector<uint8_t> blob(P.blob_bytes, 0);
  auto put = [&](size_t off, const void* src, size_t bytes) {
    if (bytes) std::memcpy(blob.data() + off, src, bytes);
  };
  put(P.off_items, P.items.data(), P.items.size() * sizeof(FactItem));
  put(P.off_groups, P.groups.data(), P.groups.size() * sizeof(FactGroup));
  if (P.rows) {  // members keep their projected token rows in the workspace
    std::vector<FactMember> mem = P.members;
    for (size_t m = 0; m < mem.size(); ++m) {
      mem[m].rows_a = (float*)((uint8_t*)workspace + P.member_rows[2 * m]);
      mem[m].rows_b = (float*)((uint8_t*)workspace + P.member_rows[2 * m + 1]);
    }
    put(P.off_members, mem.data(), mem.size() * sizeof(FactMember));
  } else {
    put(P.off_members, P.members.data(), P.members.size() * sizeof(FactMember));
  }
  put(P.off_tasks, P.tasks.data(), P.tasks.size() * sizeof(ReduceTask));
  put(P.off_sops, P.sops.data(), P.sops.size() * sizeof(SplitOp));
  put(P.off_sitems, P.sitems.data(), P.sitems.size() * sizeof(SplitItem));
  put(P.off_ctasks, P.ctasks.data(), P.ctasks.size() * sizeof(ContractTask));
  put(P.off_stasks, P.stasks.data(), P.stasks.size() * sizeof(ReduceTask));
  put(P.off_slabsum, P.slabsum.data(), P.slabsum.size() * sizeof(SlabSumTask));
  put(P.off_mtasks, P.mtasks.data(), P.mtasks.size() * sizeof(MaskTask));
  put(P.off_mitems, P.mitems.data(), P.mitems.size() * sizeof(MaskItem));
  put(P.off_mreduce, P.mreduce.data(), P.mreduce.size() * sizeof(ReduceTask));
  uint8_t* ws = (uint8_t*)workspace;
  uint8_t* tab = nullptr;
  HIP_TRY(place_table(ctx, kTabProj, blob, ws, s, &tab));

  const FactItem* d_items = (const FactItem*)(tab + P.off_items);
  const FactGroup* d_groups = (const FactGroup*)(tab + P.off_groups);
  const FactMember* d_members = (const FactMember*)(tab + P.off_members);
  const ReduceTask* d_tasks = (const ReduceTask*)(tab + P.off_tasks);
  float* fpart = (float*)(ws + P.off_fpart);
  const int phi_bf16 = phi_dtype == DATTRI_BF16;
  for (const Plan::Launch& L : P.launches)
    HIP_TRY(launch_factored(L.elt, L.na, L.nb, L.aligned, d_items + L.first, L.count, d_groups,
                            d_members, fpart, s));
  if (P.n_fact_tasks)
    HIP_TRY(launch_reduce(d_tasks, P.n_fact_tasks, n, P.fact_max_out, fpart, phi, phi_bf16, ld_phi, s));

  const SplitOp* d_sops = (const SplitOp*)(tab + P.off_sops);
  const SplitItem* d_sitems = (const SplitItem*)(tab + P.off_sitems);
  const ContractTask* d_ctasks = (const ContractTask*)(tab + P.off_ctasks);
  float* proj = (float*)(ws + P.off_proj);
  for (const Plan::SplitLaunch& L : P.slaunches)
    HIP_TRY(launch_split_project(L.elt, L.aligned, L.nt, d_sitems + L.first, L.count, d_sops, proj, s));
  if (!P.slabsum.empty())
    HIP_TRY(launch_slab_sum((const SlabSumTask*)(tab + P.off_slabsum), (int)P.slabsum.size(),
                            P.slabsum_max_n4, proj, s));
  float* spart = (float*)(ws + P.off_spart);
  if (!P.ctasks.empty())
    HIP_TRY(launch_split_contract(d_ctasks, (int)P.ctasks.size(), n, P.split_max_tchunks, proj, spart,
                                  phi, phi_bf16, ld_phi, s));
  if (!P.stasks.empty())
    HIP_TRY(launch_reduce((const ReduceTask*)(tab + P.off_stasks), (int)P.stasks.size(), n,
                          P.split_max_out, spart, phi, phi_bf16, ld_phi, s));

  if (!P.mtasks.empty()) {
    float* kpart = (float*)(ws + P.off_maskpart);
    for (const Plan::MaskLaunch& L : P.mlaunches) {
      const MaskItem* items = (const MaskItem*)(tab + P.off_mitems) + L.first;
      const MaskTask* tasks = (const MaskTask*)(tab + P.off_mtasks);
      if (L.fixed)
        HIP_TRY(launch_mask_fixed(items, L.count, tasks, kpart, s));
      else
        HIP_TRY(launch_mask(ctx->elt, L.aligned, L.full, P.mask_b16 ? 1 : 0, items, L.count, tasks, P.mask_lds,
                            kpart, s));
    }
    HIP_TRY(launch_reduce((const ReduceTask*)(tab + P.off_mreduce), (int)P.mreduce.size(), n, P.mask_max_out,
                          kpart, phi, phi_bf16, ld_phi, s));
  }

  float* gbuf = (float*)(ws + P.off_g);
  float* mpart = (float*)(ws + P.off_mpart);
  for (const MatChunk& mc : P.mat) {
    const Layer& L = ctx->layers[mc.layer];
    if (mc.fused) {
      GFusedArgs fa;
      fa.A = L.A; fa.B = L.B; fa.lengths = L.lengths; fa.P_in = L.P_in; fa.P_out = L.P_out;
      fa.d_in = L.d_in; fa.d_out = L.d_out; fa.T = L.T; fa.k_in = L.k_in; fa.k_out = L.k_out;
      fa.ex_begin = mc.ex_begin; fa.ex_count = mc.ex_count; fa.n_ublocks = mc.n_ublocks;
      fa.n_tchunks = mc.n_tchunks; fa.tok_chunk = mc.tok_chunk; fa.partials = mpart;
      fa.n_vsplit = mc.n_vsplit; fa.vt_per_split = mc.vt_per_split;
      HIP_TRY(launch_gfused(fa, s));
      HIP_TRY(launch_reduce(d_tasks + mc.task, 1, mc.ex_count, L.k_in * L.k_out, mpart, phi, phi_bf16,
                            ld_phi, s));
      continue;
    }
    GradArgs ga;
    ga.A = L.A; ga.B = L.B; ga.lengths = L.lengths;
    ga.d_in = L.d_in; ga.d_out = L.d_out; ga.T = L.T;
    ga.ex_begin = mc.ex_begin; ga.ex_count = mc.ex_count;
    ga.aligned = ((uintptr_t)L.A % 16 == 0) && ((uintptr_t)L.B % 16 == 0) &&
                 (L.d_in * ctx->elt) % 16 == 0 && (L.d_out * ctx->elt) % 16 == 0;
    ga.G = gbuf;
    HIP_TRY(launch_gradient(ctx->elt, ga, s));
    GProjArgs pa;
    pa.G = gbuf; pa.P_in = L.P_in; pa.P_out = L.P_out;
    pa.d_in = L.d_in; pa.d_out = L.d_out; pa.k_in = L.k_in; pa.k_out = L.k_out;
    pa.ex_count = mc.ex_count; pa.n_ublocks = mc.n_ublocks; pa.partials = mpart;
    pa.n_ksplit = mc.n_ksplit; pa.kb_per_split = mc.kb_per_split;
    HIP_TRY(launch_gproject(ctx->elt, pa, s));
    HIP_TRY(launch_reduce(d_tasks + mc.task, 1, mc.ex_count, L.k_in * L.k_out, mpart, phi, phi_bf16,
                          ld_phi, s));
  }
  return DATTRI_OK;
}


extern "C" {

const char* dattri_last_error(void) { return last_error_message(); }

dattri_status dattri_create(dattri_ctx** out, dattri_dtype compute, uint64_t seed) {
  reset_error();
  if (!out) return fail(DATTRI_E_INVALID_ARG, "out is NULL");
  if (compute != DATTRI_F32 && compute != DATTRI_BF16)
    return fail(DATTRI_E_DTYPE, "compute dtype %d is neither F32 nor BF16", (int)compute);
  dattri_ctx* c = new (std::nothrow) dattri_ctx();
  if (!c) return fail(DATTRI_E_INVALID_ARG, "out of host memory");
  c->dtype = compute;
  c->elt = compute == DATTRI_BF16 ? 2 : 4;
  c->seed = seed;
  c->cost = default_cost_model();
  c->xcost = default_crossgram_cost_model();
  *out = c;
  return DATTRI_OK;
}

void dattri_destroy(dattri_ctx* ctx) { delete ctx; }

dattri_status dattri_register_layer(dattri_ctx* ctx, int32_t d_in, int32_t d_out, int32_t k_in,
                                    int32_t k_out, int32_t* layer_id) {
  reset_error();
  if (!ctx || !layer_id) return fail(DATTRI_E_INVALID_ARG, "ctx or layer_id is NULL");
  if (d_in < 1 || d_out < 1 || k_in < 1 || k_out < 1 || d_in > kMaxDim || d_out > kMaxDim ||
      k_in > kMaxDim || k_out > kMaxDim)
    return fail(DATTRI_E_INVALID_ARG, "sizes must lie in [1, 2^20]: d_in=%d d_out=%d k_in=%d k_out=%d",
                d_in, d_out, k_in, k_out);
  Layer L;
  L.d_in = d_in; L.d_out = d_out; L.k_in = k_in; L.k_out = k_out;
  L.offset = ctx->F;
  ctx->F += (int64_t)k_in * k_out;
  ctx->layers.push_back(std::move(L));
  *layer_id = (int32_t)ctx->layers.size() - 1;
  return DATTRI_OK;
}

dattri_status dattri_register_mask_layer(dattri_ctx* ctx, int32_t d_in, int32_t d_out, int32_t mask_size,
                                         int32_t mask_id, int32_t mask_count, int32_t* layer_id) {
  reset_error();
  if (!ctx || !layer_id) return fail(DATTRI_E_INVALID_ARG, "ctx or layer_id is NULL");
  if (d_in < 1 || d_out < 1 || d_in > kMaxDim || d_out > kMaxDim)
    return fail(DATTRI_E_INVALID_ARG, "sizes must lie in [1, 2^20]: d_in=%d d_out=%d", d_in, d_out);
  if (mask_size < 1 || mask_id < 0 || mask_count < 1 || (int64_t)mask_size * mask_count > (1 << 24))
    return fail(DATTRI_E_INVALID_ARG, "mask_size=%d, mask_count=%d must be >= 1 with at most 2^24 entries in all, "
                "mask_id=%d >= 0", mask_size, mask_count, mask_id);
  const int64_t last = ((int64_t)mask_id + mask_count) * mask_size;
  if (2 * last > (int64_t)d_in * d_out)
    return fail(DATTRI_E_INVALID_ARG, "(mask_id + mask_count) * mask_size = %lld exceeds half of the %lld entries",
                (long long)last, (long long)((int64_t)d_in * d_out));
  Layer L;
  L.d_in = d_in; L.d_out = d_out; L.k_in = 1; L.k_out = mask_size * mask_count;
  L.mask_size = mask_size;
  L.mask_id = mask_id;
  L.mask_count = mask_count;
  L.offset = ctx->F;
  ctx->F += (int64_t)mask_size * mask_count;
  ctx->layers.push_back(std::move(L));
  *layer_id = (int32_t)ctx->layers.size() - 1;
  return DATTRI_OK;
}

dattri_status dattri_get_mask(const dattri_ctx* ctx, int32_t layer, int32_t* rows, int32_t* cols) {
  reset_error();
  dattri_status st = check_layer(ctx, layer);
  if (st != DATTRI_OK) return st;
  const Layer& L = ctx->layers[layer];
  if (L.mask_size <= 0) return fail(DATTRI_E_INVALID_ARG, "layer %d is not a mask layer", layer);
  std::vector<int32_t> r, c;
  mask_entries(derive_mask_seed(ctx->seed, layer), L.d_in, L.d_out, L.mask_size, L.mask_id, L.mask_count, r, c);
  if (rows) std::memcpy(rows, r.data(), r.size() * 4);
  if (cols) std::memcpy(cols, c.data(), c.size() * 4);
  return DATTRI_OK;
}

dattri_status dattri_num_layers(const dattri_ctx* ctx, int32_t* n) {
  reset_error();
  if (!ctx || !n) return fail(DATTRI_E_INVALID_ARG, "ctx or n is NULL");
  *n = (int32_t)ctx->layers.size();
  return DATTRI_OK;
}

dattri_status dattri_layer_dims(const dattri_ctx* ctx, int32_t layer, int32_t* d_in, int32_t* d_out,
                                int32_t* k_in, int32_t* k_out) {
  reset_error();
  dattri_status st = check_layer(ctx, layer);
  if (st != DATTRI_OK) return st;
  const Layer& L = ctx->layers[layer];
  if (d_in) *d_in = L.d_in;
  if (d_out) *d_out = L.d_out;
  if (k_in) *k_in = L.k_in;
  if (k_out) *k_out = L.k_out;
  return DATTRI_OK;
}

dattri_status dattri_feature_dim(const dattri_ctx* ctx, int64_t* F) {
  reset_error();
  if (!ctx || !F) return fail(DATTRI_E_INVALID_ARG, "ctx or F is NULL");
  *F = ctx->F;
  return DATTRI_OK;
}

dattri_status dattri_layer_offset(const dattri_ctx* ctx, int32_t layer, int64_t* offset) {
  reset_error();
  dattri_status st = check_layer(ctx, layer);
  if (st != DATTRI_OK) return st;
  if (!offset) return fail(DATTRI_E_INVALID_ARG, "offset is NULL");
  *offset = ctx->layers[layer].offset;
  return DATTRI_OK;
}

dattri_status dattri_projection_bytes(const dattri_ctx* ctx, int32_t layer, size_t* bytes_in,
                                      size_t* bytes_out) {
  reset_error();
  dattri_status st = check_layer(ctx, layer);
  if (st != DATTRI_OK) return st;
  const Layer& L = ctx->layers[layer];
  if (L.mask_size > 0) {  // the mask's entry table: rows, cols, output positions; group slices
    if (bytes_in) *bytes_in = (size_t)12 * L.k_out + (size_t)16 * ((L.k_out + kMaskGroup - 1) / kMaskGroup);
    if (bytes_out) *bytes_out = 0;
    return DATTRI_OK;
  }
  if (bytes_in) *bytes_in = (size_t)packed_bytes(L.d_in, L.k_in, ctx->elt);
  if (bytes_out) *bytes_out = (size_t)packed_bytes(L.d_out, L.k_out, ctx->elt);
  return DATTRI_OK;
}

dattri_status dattri_bind_projection(dattri_ctx* ctx, int32_t layer, void* dev_P_in, void* dev_P_out,
                                     const float* host_P_in_override,
                                     const float* host_P_out_override, void* stream) {
  reset_error();
  dattri_status st = check_layer(ctx, layer);
  if (st != DATTRI_OK) return st;
  Layer& L = ctx->layers[layer];
  if (L.mask_size > 0) {  // upload the mask's entry table into dev_P_in
    if (!dev_P_in) return fail(DATTRI_E_INVALID_ARG, "device table pointer is NULL");
    if ((uintptr_t)dev_P_in % 16) return fail(DATTRI_E_INVALID_ARG, "device table pointer must be 16-byte aligned");
    if (host_P_in_override || host_P_out_override)
      return fail(DATTRI_E_INVALID_ARG, "mask layers take no map overrides");
    std::vector<int32_t> r, c, table;
    mask_entries(derive_mask_seed(ctx->seed, layer), L.d_in, L.d_out, L.mask_size, L.mask_id, L.mask_count, r, c);
    mask_slot_table(r, c, L.d_in, L.d_out, ctx->elt, table);
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(hipMemcpyAsync(dev_P_in, table.data(), table.size() * 4, hipMemcpyHostToDevice, s));
    HIP_TRY(hipStreamSynchronize(s));
    L.mask_slices.assign(table.begin() + 3 * (size_t)L.k_out, table.end());
    L.P_in = dev_P_in;
    L.P_out = nullptr;
    L.bound = true;
    return DATTRI_OK;
  }
  if (!dev_P_in || !dev_P_out) return fail(DATTRI_E_INVALID_ARG, "device map pointer is NULL");
  if ((uintptr_t)dev_P_in % 16 || (uintptr_t)dev_P_out % 16)
    return fail(DATTRI_E_INVALID_ARG, "device map pointers must be 16-byte aligned");
  for (int side = 0; side < 2; ++side) {
    const int d = side ? L.d_out : L.d_in, k = side ? L.k_out : L.k_in;
    const float* ov = side ? host_P_out_override : host_P_in_override;
    std::vector<float>& keep = side ? L.override_out : L.override_in;
    keep.clear();
    if (ov) {
      keep.resize((size_t)d * k);
      for (size_t i = 0; i < keep.size(); ++i) keep[i] = round_to_compute((double)ov[i], ctx->elt);
    }
  }
  hipStream_t s = (hipStream_t)stream;
  for (int side = 0; side < 2; ++side) {
    const int d = side ? L.d_out : L.d_in, k = side ? L.k_out : L.k_in;
    std::vector<float> logical;
    logical_map(ctx, layer, side, logical);
    std::vector<uint8_t> packed;
    pack_map(logical.data(), d, k, ctx->elt, packed);
    HIP_TRY(hipMemcpyAsync(side ? dev_P_out : dev_P_in, packed.data(), packed.size(),
                           hipMemcpyHostToDevice, s));
    HIP_TRY(hipStreamSynchronize(s));
  }
  L.P_in = dev_P_in;
  L.P_out = dev_P_out;
  L.bound = true;
  return DATTRI_OK;
}

dattri_status dattri_set_map_kind(dattri_ctx* ctx, int32_t layer, dattri_map_kind kind) {
  reset_error();
  dattri_status st = check_layer(ctx, layer);
  if (st != DATTRI_OK) return st;
  if (kind != DATTRI_MAP_GAUSSIAN && kind != DATTRI_MAP_RADEMACHER)
    return fail(DATTRI_E_INVALID_ARG, "map kind %d unknown", (int)kind);
  Layer& L = ctx->layers[layer];
  if (L.mask_size > 0) return fail(DATTRI_E_INVALID_ARG, "layer %d is a mask layer", layer);
  if (L.map_kind != kind) {
    L.map_kind = kind;
    L.bound = false;  // the bound maps are of the other kind: bind again
  }
  return DATTRI_OK;
}

dattri_status dattri_get_map_kind(const dattri_ctx* ctx, int32_t layer, dattri_map_kind* kind) {
  reset_error();
  dattri_status st = check_layer(ctx, layer);
  if (st != DATTRI_OK) return st;
  if (!kind) return fail(DATTRI_E_INVALID_ARG, "kind is NULL");
  *kind = (dattri_map_kind)ctx->layers[layer].map_kind;
  return DATTRI_OK;
}

dattri_status dattri_get_projection(const dattri_ctx* ctx, int32_t layer, float* host_P_in,
                                    float* host_P_out) {
  reset_error();
  dattri_status st = check_layer(ctx, layer);
  if (st != DATTRI_OK) return st;
  if (ctx->layers[layer].mask_size > 0)
    return fail(DATTRI_E_INVALID_ARG, "layer %d is a mask layer (see dattri_get_mask)", layer);
  std::vector<float> v;
  if (host_P_in) {
    logical_map(ctx, layer, 0, v);
    std::memcpy(host_P_in, v.data(), v.size() * 4);
  }
  if (host_P_out) {
    logical_map(ctx, layer, 1, v);
    std::memcpy(host_P_out, v.data(), v.size() * 4);
  }
  return DATTRI_OK;
}

dattri_status dattri_capture_layer(dattri_ctx* ctx, int32_t layer, const void* A, const void* B,
                                   int32_t n, int32_t T, const int32_t* dev_lengths) {
  reset_error();
  dattri_status st = check_layer(ctx, layer);
  if (st != DATTRI_OK) return st;
  if (n < 0 || T < 0) return fail(DATTRI_E_INVALID_ARG, "n=%d and T=%d must be >= 0", n, T);
  if ((int64_t)n * T > 0 && (!A || !B))
    return fail(DATTRI_E_INVALID_ARG, "A or B is NULL for a non-empty capture");
  Layer& L = ctx->layers[layer];
  if ((int64_t)T * std::max(L.d_in, L.d_out) * ctx->elt >= kMaxBlockBytes)
    return fail(DATTRI_E_SHAPE, "layer %d: one example's factor block (T*d = %lld elements) exceeds 4 GiB",
                layer, (long long)T * std::max(L.d_in, L.d_out));
  L.A = A;
  L.B = B;
  L.n = n;
  L.T = T;
  L.lengths = dev_lengths;
  L.captured = true;
  return DATTRI_OK;
}

dattri_status dattri_clear_captures(dattri_ctx* ctx) {
  reset_error();
  if (!ctx) return fail(DATTRI_E_INVALID_ARG, "ctx is NULL");
  for (Layer& L : ctx->layers) {
    L.A = L.B = nullptr;
    L.lengths = nullptr;
    L.n = L.T = 0;
    L.captured = false;
  }
  return DATTRI_OK;
}

dattri_status dattri_workspace_bytes(const dattri_ctx* ctx, dattri_route route, size_t* bytes) {
  reset_error();
  if (!ctx || !bytes) return fail(DATTRI_E_INVALID_ARG, "ctx or bytes is NULL");
  if (route < DATTRI_ROUTE_AUTO || route > DATTRI_ROUTE_MATERIALIZED)
    return fail(DATTRI_E_INVALID_ARG, "route %d unknown", (int)route);
  std::shared_ptr<const Plan> P;
  dattri_status st = get_plan(ctx, route, false, &P);
  if (st != DATTRI_OK) return st;
  *bytes = P->total;
  return DATTRI_OK;
}

dattri_status dattri_set_factored_form(dattri_ctx* ctx, dattri_factored_form form) {
  reset_error();
  if (!ctx) return fail(DATTRI_E_INVALID_ARG, "ctx is NULL");
  if (form < DATTRI_FORM_AUTO || form > DATTRI_FORM_SPLIT)
    return fail(DATTRI_E_INVALID_ARG, "factored form %d unknown", (int)form);
  ctx->form = form;
  return DATTRI_OK;
}

dattri_status dattri_get_factored_form(const dattri_ctx* ctx, dattri_factored_form* form) {
  reset_error();
  if (!ctx || !form) return fail(DATTRI_E_INVALID_ARG, "ctx or form is NULL");
  *form = ctx->form;
  return DATTRI_OK;
}

dattri_status dattri_project_per_example(dattri_ctx* ctx, void* phi, dattri_dtype phi_dtype,
                                         int64_t ld_phi, void* workspace, size_t ws_bytes,
                                         dattri_route route, void* stream) {
  reset_error();
  if (!ctx) return fail(DATTRI_E_INVALID_ARG, "ctx is NULL");
  if (phi_dtype != DATTRI_F32 && phi_dtype != DATTRI_BF16)
    return fail(DATTRI_E_DTYPE, "phi dtype %d is neither F32 nor BF16", (int)phi_dtype);
  if (route < DATTRI_ROUTE_AUTO || route > DATTRI_ROUTE_MATERIALIZED)
    return fail(DATTRI_E_INVALID_ARG, "route %d unknown", (int)route);
  for (size_t l = 0; l < ctx->layers.size(); ++l)
    if (!ctx->layers[l].bound)
      return fail(DATTRI_E_STATE, "layer %zu: projection maps not bound", l);
  std::shared_ptr<const Plan> P;
  dattri_status st = get_plan(ctx, route, false, &P);
  if (st != DATTRI_OK) return st;
  return run_plan(ctx, *P, phi, phi_dtype, ld_phi, workspace, ws_bytes, (hipStream_t)stream);
}

dattri_status dattri_plan_bytes(const dattri_ctx* ctx, dattri_route route, size_t* bytes) {
  reset_error();
  if (!ctx || !bytes) return fail(DATTRI_E_INVALID_ARG, "ctx or bytes is NULL");
  if (route < DATTRI_ROUTE_AUTO || route > DATTRI_ROUTE_MATERIALIZED)
    return fail(DATTRI_E_INVALID_ARG, "route %d unknown", (int)route);
  std::shared_ptr<const Plan> P;
  dattri_status st = get_plan(ctx, route, false, &P);
  if (st != DATTRI_OK) return st;
  *bytes = align_up(P->blob_bytes);
  return DATTRI_OK;
}

dattri_status dattri_bind_plan_buffer(dattri_ctx* ctx, void* dev_plan, size_t bytes) {
  reset_error();
  if (!ctx) return fail(DATTRI_E_INVALID_ARG, "ctx is NULL");
  if (dev_plan && (uintptr_t)dev_plan % kAlign)
    return fail(DATTRI_E_INVALID_ARG, "plan buffer must be 256-byte aligned");
  ctx->plan_buf = dev_plan ? (uint8_t*)dev_plan : nullptr;
  ctx->plan_cap = dev_plan ? bytes / kAlign * kAlign : 0;
  ctx->slots.clear();
  ctx->slots_used = 0;
  return DATTRI_OK;
}

dattri_status dattri_materialize_gradient(dattri_ctx* ctx, int32_t layer, int32_t ex_begin,
                                          int32_t ex_count, float* G_out, void* stream) {
  reset_error();
  dattri_status st = check_layer(ctx, layer);
  if (st != DATTRI_OK) return st;
  const Layer& L = ctx->layers[layer];
  if (!L.captured) return fail(DATTRI_E_STATE, "layer %d has no capture", layer);
  if (ex_begin < 0 || ex_count < 0 || (int64_t)ex_begin + ex_count > L.n)
    return fail(DATTRI_E_INVALID_ARG, "examples [%d, %d+%d) outside [0, %d)", ex_begin, ex_begin,
                ex_count, L.n);
  if (ex_count == 0) return DATTRI_OK;
  if (!G_out) return fail(DATTRI_E_INVALID_ARG, "G_out is NULL");
  GradArgs ga;
  ga.A = L.A; ga.B = L.B; ga.lengths = L.lengths;
  ga.d_in = L.d_in; ga.d_out = L.d_out; ga.T = L.T;
  ga.ex_begin = ex_begin; ga.ex_count = ex_count;
  ga.aligned = ((uintptr_t)L.A % 16 == 0) && ((uintptr_t)L.B % 16 == 0) &&
               (L.d_in * ctx->elt) % 16 == 0 && (L.d_out * ctx->elt) % 16 == 0;
  ga.G = G_out;
  HIP_TRY(launch_gradient(ctx->elt, ga, (hipStream_t)stream));
  return DATTRI_OK;
}

dattri_status dattri_set_cost_model(dattri_ctx* ctx, const dattri_cost_model* m) {
  reset_error();
  if (!ctx || !m) return fail(DATTRI_E_INVALID_ARG, "ctx or model is NULL");
  const dattri_status st = check_cost_model(*m);
  if (st != DATTRI_OK) return st;
  ctx->cost = *m;
  return DATTRI_OK;
}

dattri_status dattri_set_cost_calibration(dattri_ctx* ctx, const char* json_path) {
  reset_error();
  if (!ctx || !json_path) return fail(DATTRI_E_INVALID_ARG, "ctx or json_path is NULL");
  dattri_cost_model m;
  dattri_status st = read_cost_calibration(json_path, &m);
  if (st != DATTRI_OK) return st;
  if ((st = check_cost_model(m)) != DATTRI_OK) return st;
  ctx->cost = m;
  return DATTRI_OK;
}

dattri_status dattri_get_cost_model(const dattri_ctx* ctx, dattri_cost_model* m) {
  reset_error();
  if (!ctx || !m) return fail(DATTRI_E_INVALID_ARG, "ctx or model is NULL");
  *m = ctx->cost;
  return DATTRI_OK;
}

dattri_status dattri_layer_costs(const dattri_ctx* ctx, int32_t layer, int32_t T,
                                 int64_t* factored_flops, int64_t* materialized_flops,
                                 int64_t* factored_bytes, int64_t* materialized_bytes) {
  reset_error();
  dattri_status st = check_layer(ctx, layer);
  if (st != DATTRI_OK) return st;
  if (T < 0) return fail(DATTRI_E_INVALID_ARG, "T=%d < 0", T);
  const Layer& ML = ctx->layers[layer];
  if (ML.mask_size > 0) {  // the gather: one product per entry and token, both factor rows read
    if (factored_flops) *factored_flops = 2 * (int64_t)T * ML.k_out;
    if (factored_bytes) *factored_bytes = (int64_t)T * (ML.d_in + ML.d_out) * ctx->elt;
    if (materialized_flops) *materialized_flops = 0;
    if (materialized_bytes) *materialized_bytes = 0;
    return DATTRI_OK;
  }
  const Counts c = layer_counts(ctx->layers[layer], T, ctx->elt);
  if (factored_flops) *factored_flops = c.f_flops;
  if (materialized_flops) *materialized_flops = c.m_flops;
  if (factored_bytes) *factored_bytes = c.f_bytes;
  if (materialized_bytes) *materialized_bytes = c.m_bytes;
  return DATTRI_OK;
}

dattri_status dattri_layer_route(const dattri_ctx* ctx, int32_t layer, dattri_route* chosen,
                                 double* pred_factored_us, double* pred_materialized_us) {
  reset_error();
  dattri_status st = check_layer(ctx, layer);
  if (st != DATTRI_OK) return st;
  const Layer& L = ctx->layers[layer];
  if (!L.captured) return fail(DATTRI_E_STATE, "layer %d has no capture", layer);
  if (L.mask_size > 0) {
    if (chosen) *chosen = DATTRI_ROUTE_MASK;
    if (pred_factored_us) *pred_factored_us = INFINITY;
    if (pred_materialized_us) *pred_materialized_us = INFINITY;
    return DATTRI_OK;
  }
  double f, m;
  predict(ctx, L, &f, &m);
  if (chosen) *chosen = call_routes(ctx, DATTRI_ROUTE_AUTO)[layer];
  if (pred_factored_us) *pred_factored_us = factored_supported(L) ? f : INFINITY;
  if (pred_materialized_us) *pred_materialized_us = m;
  return DATTRI_OK;
}

}  // extern "C"
