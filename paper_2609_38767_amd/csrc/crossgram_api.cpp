// C ABI of cross-Gram matrices and squared norms of unprojected per-example
// weight gradients (Sec. 3.2 "Factorized inner product", Eq. (4), and
// "FLOP-aware routing"; App. A.4 routing table and "Routing"): validation,
// exact operation counts, the MI355X time model that routes each layer, launch
// planning and execution.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <utility>
#include <vector>

#include "api_common.h"
#include "context.h"
#include "dattri.h"
#include "internal.h"
#include "plan.h"

using namespace dattri;

namespace dattri {

dattri_crossgram_cost_model default_crossgram_cost_model() {
  // Effective rates measured on MI355X (bf16 factor blocks): the factorized
  // route, both forms of the materialized one and the gradient build timed on
  // 28 shapes (1024..4096-wide and 128-wide layers, T = 16..2048, 8 x 1,
  // 16 x 16 and 8 x 8 batches), each a stack of 24 layers so the factorized
  // and one-pass routes run as one grouped launch each, and fitted by least
  // squares on log time.  The two bandwidths come out far above HBM's: on
  // this sweep the factor reads never bound those kernels.
  dattri_crossgram_cost_model m;
  m.ghost_tflops = 658.3;  // on whole padded tiles
  m.ghost_gbs = 6.56e6;
  m.ghost_layer_us = 2.12;
  m.build_tflops = 638.0;  // on the tile builds of the build kernel's rounds
  m.build_gbs = 1.17e8;
  m.dot_gbs = 1180.0;
  m.launch_us = 4.81;
  m.onepass_tflops = 1174.7;  // on the tile builds the one-pass kernel issues
  return m;
}

}  // namespace dattri

namespace {

constexpr int64_t kGhostPartsBudget = (int64_t)256 << 20;  // block sums per factorized group
constexpr int64_t kGhostTilesMax = (int64_t)1 << 22;      // tiles per factorized group
constexpr int64_t kXgGBudget = (int64_t)2 << 30;          // staged float32 DW per chunk
constexpr int64_t kDotChunk = 16384;                      // floats per Frobenius-product chunk
constexpr int64_t kOOBLimit = 0xFFFFFFF0LL;                // first byte offset a descriptor never covers
constexpr int64_t kXOnePartsBudget = (int64_t)64 << 20;     // one-pass tile sums per launch (bytes)
constexpr int64_t kXOneSlots = 2 * 256;                    // resident one-pass workgroups (2 per CU)
constexpr int64_t kXOneMaxRun = 4;  // examples of batch a per one-pass workgroup, at most (measured:
                                    // runs of 8 took 16.1 ms against 14.6-14.9 for 3-4 on the
                                    // 96-layer T = 2048 sweep, though they issue 10% less work)

inline int64_t r16(int64_t T) { return (T + 15) / 16 * 16; }
inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct XCounts {
  int64_t f_flops, m_flops, f_bytes, m_bytes, build_flops, build_bytes, dot_bytes;
};

XCounts xcounts(int64_t na, int64_t nb, int64_t Ta, int64_t Tb, int64_t di, int64_t dq, int64_t elt) {
  XCounts c;
  c.f_flops = 2 * na * nb * Ta * Tb * (di + dq + 1);
  c.build_flops = 2 * (na * Ta + nb * Tb) * di * dq;
  c.m_flops = c.build_flops + 2 * na * nb * di * dq;
  c.f_bytes = (na * Ta + nb * Tb) * (di + dq) * elt;
  c.build_bytes = c.f_bytes + 4 * (na + nb) * di * dq;
  c.dot_bytes = 4 * (na + nb) * di * dq;
  c.m_bytes = c.build_bytes + c.dot_bytes;
  return c;
}

// One-pass materialized launch over ci examples of batch a against cj of
// batch b (diag: the ci examples against themselves): a workgroup forms one
// 128 x 128 tile of DW_b[j] once, then the same tile of DW_a[i] for each of
// its ipw <= kXOneMaxRun examples.  nz = runs of batch a per (tile, j) is
// chosen to minimise the predicted time: rounds of kXOneSlots workgroups, each
// round as long as one workgroup's builds (ipw, plus the reference build
// unless diag).
struct XOneShape {
  int nz = 1, ipw = 1;
  double us = 0.0;
};

inline int64_t r32(int64_t T) { return (T + 31) / 32 * 32; }

XOneShape xone_shape(const dattri_crossgram_cost_model& m, int64_t tiles, int64_t ci, int64_t cj, int64_t Ta,
                     int64_t Tb, bool diag) {
  XOneShape best;
  best.us = INFINITY;
  if (tiles <= 0 || ci <= 0) {
    best.us = 0.0;
    return best;
  }
  const double per_token = 2.0 * kXOneTile * kXOneTile / (m.onepass_tflops * 1e6 / kXOneSlots);
  const double ta = per_token * (double)r32(Ta), tb = diag ? 0.0 : per_token * (double)r32(Tb);
  const int64_t ys = diag ? 1 : cj;
  const int64_t nz_max = std::min<int64_t>(ci, 65535);
  for (int64_t nz = cdiv(ci, kXOneMaxRun); nz <= nz_max; ++nz) {
    const int64_t ipw = cdiv(ci, nz);
    if (cdiv(ci, ipw) != nz) continue;  // same runs as a smaller nz
    const int64_t rounds = cdiv(tiles * ys * nz, kXOneSlots);
    const double us = (double)rounds * ((double)ipw * ta + tb);
    if (us < best.us) best = XOneShape{(int)nz, (int)ipw, us};
  }
  return best;
}

// Whether a layer can take the one-pass materialized kernel: bf16 blocks with
// 16-byte aligned rows, and one example's block within a 32-bit byte range.
bool xone_ok(const Layer& La, const Layer& Lb, int elt);

// Predicted microseconds of one layer's two routes, as this build runs them:
// the factorized kernel computes whole 128 x 128 tiles of the padded token
// Gram and reads 128 rows of each side per tile (diag: each example's own
// Gram); the materialized route is the faster of its two forms: DW staged in
// HBM (build both batches, in rounds of tile builds as the one-pass form, or
// by the bytes written; then the products: four launches) and, where `one`
// allows it, the one-pass kernel (xone_shape, plus the tile-sum launch).
void xpredict(const dattri_crossgram_cost_model& m, int64_t na, int64_t nb, int64_t Ta, int64_t Tb,
              int64_t di, int64_t dq, int elt, bool diag, bool one, double* f_us, double* m_us) {
  if (diag) nb = na;
  const XCounts c = diag ? xcounts(na, 0, Ta, 0, di, dq, elt) : xcounts(na, nb, Ta, Tb, di, dq, elt);
  const int64_t tiles = diag ? na * cdiv(r16(Ta), kGhostTile) * cdiv(r16(Ta), kGhostTile)
                             : cdiv(na * r16(Ta), kGhostTile) * cdiv(nb * r16(Tb), kGhostTile);
  const double tflops = (double)tiles * 2.0 * kGhostTile * kGhostTile * (double)(di + dq + 1);
  const double tbytes = (double)tiles * 2.0 * kGhostTile * (double)(di + dq) * elt;
  *f_us = (tiles == 0) ? 0.0
                       : std::max(tflops / (m.ghost_tflops * 1e6), tbytes / (m.ghost_gbs * 1e3)) +
                             m.ghost_layer_us;
  // the build kernel runs one workgroup per 128 x 128 tile of DW and example:
  // rounds of kXOneSlots workgroups per batch, each as long as one tile build
  const int64_t dtiles = cdiv(dq, kXOneTile) * cdiv(di, kXOneTile);
  const double per_token = 2.0 * kXOneTile * kXOneTile / (m.build_tflops * 1e6 / kXOneSlots);
  const double rounds = (double)cdiv(dtiles * na, kXOneSlots) * per_token * (double)r32(Ta) +
                        (diag ? 0.0 : (double)cdiv(dtiles * nb, kXOneSlots) * per_token * (double)r32(Tb));
  const double build = std::max(rounds, (double)c.build_bytes / (m.build_gbs * 1e3));
  const double dot_bytes = diag ? 4.0 * na * di * dq : (double)c.dot_bytes;
  *m_us = build + dot_bytes / (m.dot_gbs * 1e3) + (diag ? 3.0 : 4.0) * m.launch_us;
  if (one) {
    const double o = xone_shape(m, dtiles, na, nb, Ta, Tb, diag).us + 2.0 * m.launch_us;
    *m_us = std::min(*m_us, o);
  }
}

dattri_status check_pair(const dattri_ctx* a, const dattri_ctx* b) {
  if (!a || !b) return fail(DATTRI_E_INVALID_ARG, "context is NULL");
  if (a->dtype != b->dtype) return fail(DATTRI_E_SHAPE, "the two contexts have different compute types");
  if (a->layers.empty()) return fail(DATTRI_E_STATE, "no layers registered");
  if (a->layers.size() != b->layers.size())
    return fail(DATTRI_E_SHAPE, "layer counts differ (%zu vs %zu)", a->layers.size(), b->layers.size());
  for (size_t l = 0; l < a->layers.size(); ++l) {
    const Layer &La = a->layers[l], &Lb = b->layers[l];
    if (La.d_in != Lb.d_in || La.d_out != Lb.d_out)
      return fail(DATTRI_E_SHAPE, "layer %zu: (d_in, d_out) = (%d, %d) vs (%d, %d)", l, La.d_in, La.d_out,
                  Lb.d_in, Lb.d_out);
    if (!La.captured || !Lb.captured) return fail(DATTRI_E_STATE, "layer %zu is not captured in both", l);
    if (La.n != a->layers[0].n || Lb.n != b->layers[0].n)
      return fail(DATTRI_E_STATE, "captures disagree on the number of examples");
  }
  return DATTRI_OK;
}

// Whether the factorized kernel can stream an entry's token rows by direct
// loads: bf16, 16-byte aligned rows, and the rows one tile touches (at most
// 128 + 2 T from the tile's first example) within 32-bit byte offsets.
bool ghost_dma_ok(const GhostEntry& E, int elt) {
  const int64_t d = std::max(E.d_in, E.d_out), lim = (int64_t)kOOBLimit;
  return elt == 2 && E.aligned && (128 + 2 * (int64_t)E.T1) * d * elt < lim &&
         (128 + 2 * (int64_t)E.T2) * d * elt < lim;
}

bool layer_aligned(const Layer& L, int elt) {
  return ((uintptr_t)L.A % 16 == 0) && ((uintptr_t)L.B % 16 == 0) && (L.d_in * elt) % 16 == 0 &&
         (L.d_out * elt) % 16 == 0;
}

bool xone_ok(const Layer& La, const Layer& Lb, int elt) {
  const int64_t lim = (int64_t)1 << 32;
  return elt == 2 && layer_aligned(La, elt) && layer_aligned(Lb, elt) &&
         (int64_t)La.T * std::max(La.d_in, La.d_out) * elt < lim &&
         (int64_t)Lb.T * std::max(Lb.d_in, Lb.d_out) * elt < lim;
}

// The one-pass form is taken when it is allowed and predicted faster than
// staging DW.
bool xone_pick(const dattri_crossgram_cost_model& m, const Layer& La, const Layer& Lb, int elt, bool diag) {
  if (!xone_ok(La, Lb, elt)) return false;
  double f, staged, best;
  xpredict(m, La.n, Lb.n, La.T, Lb.T, La.d_in, La.d_out, elt, diag, false, &f, &staged);
  xpredict(m, La.n, Lb.n, La.T, Lb.T, La.d_in, La.d_out, elt, diag, true, &f, &best);
  return best < staged;
}

struct XGroup { int e0, e1, t0, t1; int64_t parts_floats; };

struct XPlan {
  std::vector<int> fact, mat;  // layer ids by route
  std::vector<char> one;       // per entry of mat: the one-pass form
  std::vector<XOneEntry> xents;  // one-pass layers, all in one launch
  std::vector<int32_t> xslot;    // entry of every one-pass workgroup slot
  int xT1 = 0, xT2 = 0;        // longest sequences among them (run-length choice)
  int oa = 0, ob = 0;          // examples per one-pass launch (batch a, batch b)
  int64_t oparts = 0;          // floats of one-pass tile sums
  std::vector<GhostEntry> entries;
  std::vector<GhostTile> tiles;
  std::vector<XGroup> groups;
  int64_t max_parts = 0;
  int64_t D_max = 0, nchunks_max = 0;
  int ca = 0, cb = 0;          // examples of DW staged per chunk (batch a, batch b)
  bool reuse_g = false;        // a == b and both fit: DW built once
  size_t off_entries = 0, off_tiles = 0, off_xents = 0, off_xslots = 0, off_parts = 0, off_g1 = 0, off_g2 = 0,
         off_dparts = 0, off_oparts = 0;
  size_t total = 0;
  size_t blob_entries = 0, blob_bytes = 0;
};

// Adds entry E (with its tiles) to the current group, opening a new group when
// the block sums or tiles would exceed the group budget.
void add_entry(XPlan& P, GhostEntry E, int64_t n_rt, int64_t n_ct) {
  const int64_t pf = (int64_t)E.nbr * E.nbc;
  const int64_t nt = n_rt * n_ct;
  if (P.groups.empty() ||
      (P.groups.back().e1 > P.groups.back().e0 &&
       (P.groups.back().parts_floats + pf > kGhostPartsBudget / 4 ||
        (int64_t)(P.tiles.size() - P.groups.back().t0) + nt > kGhostTilesMax))) {
    P.groups.push_back({(int)P.entries.size(), (int)P.entries.size(), (int)P.tiles.size(),
                        (int)P.tiles.size(), 0});
  }
  XGroup& G = P.groups.back();
  E.part_off = G.parts_floats;
  const int idx = (int)P.entries.size() - G.e0;  // entry index within the group
  P.entries.push_back(E);
  for (int64_t rt = 0; rt < n_rt; ++rt)
    for (int64_t ct = 0; ct < n_ct; ++ct) P.tiles.push_back({idx, (int)rt, (int)ct, 0});
  G.e1 = (int)P.entries.size();
  G.t1 = (int)P.tiles.size();
  G.parts_floats += pf;
  P.max_parts = std::max(P.max_parts, G.parts_floats);
}

dattri_route layer_route(const dattri_ctx* a, const dattri_ctx* b, int l, dattri_route forced, bool diag) {
  if (forced != DATTRI_ROUTE_AUTO) return forced;
  const Layer &La = a->layers[l], &Lb = b->layers[l];
  double f, m;
  xpredict(a->xcost, La.n, Lb.n, La.T, Lb.T, La.d_in, La.d_out, a->elt, diag, xone_ok(La, Lb, a->elt), &f, &m);
  return f <= m ? DATTRI_ROUTE_FACTORED : DATTRI_ROUTE_MATERIALIZED;
}

// diag: the squared norms of a's examples (b == a).
dattri_status build_xplan(const dattri_ctx* a, const dattri_ctx* b, dattri_route route, bool diag,
                          XPlan& P) {
  if (route < DATTRI_ROUTE_AUTO || route > DATTRI_ROUTE_MATERIALIZED)
    return fail(DATTRI_E_INVALID_ARG, "route %d unknown", (int)route);
  const int elt = a->elt;
  const int na = a->layers[0].n, nb = b->layers[0].n;
  for (int l = 0; l < (int)a->layers.size(); ++l)
    (layer_route(a, b, l, route, diag) == DATTRI_ROUTE_FACTORED ? P.fact : P.mat).push_back(l);

  for (int l : P.fact) {
    const Layer &La = a->layers[l], &Lb = b->layers[l];
    GhostEntry E;
    std::memset(&E, 0, sizeof(E));
    E.d_in = La.d_in;
    E.d_out = La.d_out;
    E.aligned = layer_aligned(La, elt) && layer_aligned(Lb, elt);
    if (!diag) {
      if ((int64_t)na * La.T == 0 || (int64_t)nb * Lb.T == 0) continue;
      E.A1 = La.A; E.B1 = La.B; E.len1 = La.lengths;
      E.A2 = Lb.A; E.B2 = Lb.B; E.len2 = Lb.lengths;
      E.n1 = na; E.n2 = nb; E.T1 = La.T; E.T2 = Lb.T;
      E.Tp1 = (int)r16(La.T); E.Tp2 = (int)r16(Lb.T);
      if ((int64_t)na * E.Tp1 > INT32_MAX / 2 || (int64_t)nb * E.Tp2 > INT32_MAX / 2)
        return fail(DATTRI_E_UNSUPPORTED, "layer %d: n*T too large for the factorized route", l);
      E.nbr = na * E.Tp1 / 16;
      E.nbc = nb * E.Tp2 / 16;
      E.out0 = 0;
      E.dma = ghost_dma_ok(E, elt) ? 1 : 0;
      add_entry(P, E, cdiv((int64_t)na * E.Tp1, kGhostTile), cdiv((int64_t)nb * E.Tp2, kGhostTile));
    } else {
      if (La.T == 0) continue;
      for (int i = 0; i < na; ++i) {  // each example against itself
        const int64_t off_a = (int64_t)i * La.T * La.d_in * elt, off_b = (int64_t)i * La.T * La.d_out * elt;
        E.A1 = E.A2 = (const uint8_t*)La.A + off_a;
        E.B1 = E.B2 = (const uint8_t*)La.B + off_b;
        E.len1 = E.len2 = La.lengths ? La.lengths + i : nullptr;
        E.aligned = layer_aligned(La, elt) && ((uintptr_t)E.A1 % 16 == 0) && ((uintptr_t)E.B1 % 16 == 0);
        E.n1 = E.n2 = 1;
        E.T1 = E.T2 = La.T;
        E.Tp1 = E.Tp2 = (int)r16(La.T);
        E.nbr = E.nbc = E.Tp1 / 16;
        E.out0 = i;
        E.dma = ghost_dma_ok(E, elt) ? 1 : 0;
        add_entry(P, E, cdiv(E.Tp1, kGhostTile), cdiv(E.Tp2, kGhostTile));
      }
    }
  }

  // materialized layers: one-pass where picked (all in one launch: each layer
  // owns its tiles' workgroup slots, rounded up to a multiple of 8 so every
  // layer starts on XCD 0), else DW staged in HBM
  for (int l : P.mat) {
    const Layer &La = a->layers[l], &Lb = b->layers[l];
    const bool one = xone_pick(a->xcost, La, Lb, elt, diag) && (int64_t)La.d_in * La.d_out > 0;
    P.one.push_back(one ? 1 : 0);
    if (!one) {
      P.D_max = std::max<int64_t>(P.D_max, (int64_t)La.d_in * La.d_out);
      continue;
    }
    XOneEntry E;
    std::memset(&E, 0, sizeof(E));
    E.A1 = La.A; E.B1 = La.B; E.len1 = La.lengths;
    E.A2 = Lb.A; E.B2 = Lb.B; E.len2 = Lb.lengths;
    E.d_in = La.d_in; E.d_out = La.d_out; E.T1 = La.T; E.T2 = Lb.T;
    E.n_ub = (int)cdiv(La.d_out, kXOneTile);
    E.n_vt = (int)cdiv(La.d_in, kXOneTile);
    const int64_t slots = cdiv((int64_t)E.n_ub * E.n_vt, 8) * 8;
    if ((int64_t)P.xslot.size() + slots > INT32_MAX)
      return fail(DATTRI_E_UNSUPPORTED, "layer %d: too many one-pass workgroups in one call", l);
    E.slot0 = (int)P.xslot.size();
    E.nslots = (int)slots;
    P.xslot.insert(P.xslot.end(), (size_t)slots, (int32_t)P.xents.size());
    P.xents.push_back(E);
    P.xT1 = std::max(P.xT1, La.T);
    P.xT2 = std::max(P.xT2, Lb.T);
  }
  if (!P.xslot.empty()) {
    const int64_t n_slots = (int64_t)P.xslot.size();
    const int64_t cap = std::max<int64_t>(1, kXOnePartsBudget / 4 / n_slots);  // (i, j) cells per launch
    P.ob = diag ? 0 : (int)std::min<int64_t>({(int64_t)nb, 65535, cap});
    P.oa = (int)std::max<int64_t>(1, std::min<int64_t>({(int64_t)na, cap / std::max(1, P.ob),
                                                         65535 * kXOneMaxRun}));  // grid z <= 65535 runs
    P.oparts = n_slots * P.oa * std::max(1, P.ob);
  }
  if (P.D_max > 0) {
    const int64_t per = P.D_max * 4;
    if (diag) {
      P.ca = (int)std::max<int64_t>(1, std::min<int64_t>(na, kXgGBudget / per));
      P.cb = 0;
      P.reuse_g = true;
    } else if ((int64_t)(na + nb) * per <= kXgGBudget) {
      P.ca = na;
      P.cb = nb;
      P.reuse_g = (a == b);
    } else {
      P.cb = (int)std::max<int64_t>(1, std::min<int64_t>(nb, kXgGBudget / 2 / per));
      P.ca = (int)std::max<int64_t>(1, std::min<int64_t>(na, (kXgGBudget - (int64_t)P.cb * per) / per));
    }
    P.nchunks_max = cdiv(P.D_max, kDotChunk);
  }

  size_t off = 0;
  P.off_entries = off;
  off = align_up(off + P.entries.size() * sizeof(GhostEntry));
  P.off_tiles = off;
  off = align_up(off + P.tiles.size() * sizeof(GhostTile));
  P.off_xents = off;
  off = align_up(off + P.xents.size() * sizeof(XOneEntry));
  P.off_xslots = off;
  off = align_up(off + P.xslot.size() * sizeof(int32_t));
  P.blob_entries = P.off_tiles;
  P.blob_bytes = off;
  P.off_parts = off;
  off = align_up(off + (size_t)P.max_parts * 4);
  P.off_g1 = off;
  off = align_up(off + (size_t)P.ca * P.D_max * 4);
  P.off_g2 = off;
  if (!P.reuse_g) off = align_up(off + (size_t)P.cb * P.D_max * 4);
  P.off_dparts = off;
  const int64_t dp = diag ? (int64_t)P.nchunks_max * P.ca : (int64_t)P.nchunks_max * P.ca * P.cb;
  off = align_up(off + (size_t)dp * 4);
  P.off_oparts = off;
  off = align_up(off + (size_t)P.oparts * 4);
  P.total = std::max<size_t>(off, kAlign);
  return DATTRI_OK;
}

dattri_status check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (!ws) return fail(DATTRI_E_WORKSPACE, "workspace is NULL (needs %zu bytes)", need);
  if ((uintptr_t)ws % kAlign) return fail(DATTRI_E_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < need) return fail(DATTRI_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  return DATTRI_OK;
}

GradArgs grad_args(const Layer& L, int elt, int ex_begin, int ex_count, float* G) {
  GradArgs ga;
  ga.A = L.A; ga.B = L.B; ga.lengths = L.lengths;
  ga.d_in = L.d_in; ga.d_out = L.d_out; ga.T = L.T;
  ga.ex_begin = ex_begin; ga.ex_count = ex_count;
  ga.aligned = layer_aligned(L, elt);
  ga.G = G;
  return ga;
}

// Runs the plan: factorized groups (the first writes K, later ones add), then
// the materialized layers add their products.
dattri_status run_xplan(dattri_ctx* a, dattri_ctx* b, const XPlan& P, bool diag, float* K, int64_t ld,
                        uint8_t* ws, hipStream_t s) {
  const int elt = a->elt;
  const int na = a->layers[0].n, nb = b->layers[0].n;
  const int rows = na, cols = diag ? 1 : nb;
  bool wrote = false;
  uint8_t* tab = nullptr;
  if (!P.entries.empty() || !P.xents.empty()) {
    std::vector<uint8_t> blob(P.blob_bytes, 0);
    std::memcpy(blob.data() + P.off_entries, P.entries.data(), P.entries.size() * sizeof(GhostEntry));
    std::memcpy(blob.data() + P.off_tiles, P.tiles.data(), P.tiles.size() * sizeof(GhostTile));
    std::memcpy(blob.data() + P.off_xents, P.xents.data(), P.xents.size() * sizeof(XOneEntry));
    std::memcpy(blob.data() + P.off_xslots, P.xslot.data(), P.xslot.size() * sizeof(int32_t));
    HIP_TRY(place_table(a, kTabCross, blob, ws, s, &tab));
  }
  if (!P.entries.empty()) {
    const GhostEntry* d_entries = (const GhostEntry*)(tab + P.off_entries);
    const GhostTile* d_tiles = (const GhostTile*)(tab + P.off_tiles);
    float* parts = (float*)(ws + P.off_parts);
    for (const XGroup& G : P.groups) {
      HIP_TRY(launch_ghost(elt, d_entries + G.e0, d_tiles + G.t0, G.t1 - G.t0, parts, s));
      HIP_TRY(launch_ghost_reduce(d_entries + G.e0, G.e1 - G.e0, parts, rows, cols, K, ld, diag ? 1 : 0,
                                  wrote ? 1 : 0, s));
      wrote = true;
    }
  }
  if (!wrote) HIP_TRY(launch_fill_rows(K, diag ? 1 : rows, diag ? rows : cols, diag ? rows : ld, s));
  if (P.mat.empty()) return DATTRI_OK;
  float* g1 = (float*)(ws + P.off_g1);
  float* g2 = P.reuse_g ? g1 : (float*)(ws + P.off_g2);
  float* dparts = (float*)(ws + P.off_dparts);
  float* oparts = (float*)(ws + P.off_oparts);
  if (!P.xents.empty()) {  // every one-pass layer: one launch per chunk of examples, then the tile sums
    XOneArgs x;
    x.entries = (const XOneEntry*)(tab + P.off_xents);
    x.slot_entry = (const int32_t*)(tab + P.off_xslots);
    x.n_slots = (int)P.xslot.size();
    x.diag = diag ? 1 : 0;
    x.parts = oparts;
    for (int j0 = 0; j0 < (diag ? 1 : nb); j0 += std::max(1, P.ob)) {
      const int cj = diag ? 0 : std::min(P.ob, nb - j0);
      for (int i0 = 0; i0 < na; i0 += P.oa) {
        const int ci = std::min(P.oa, na - i0);
        const XOneShape sh = xone_shape(a->xcost, x.n_slots, ci, cj, P.xT1, P.xT2, diag);
        x.i0 = i0; x.ci = ci; x.ipw = sh.ipw; x.j0 = j0; x.cj = cj;
        HIP_TRY(launch_xone(x, s));
        HIP_TRY(launch_kacc(oparts, x.n_slots, ci, diag ? ci : cj, K, ld, i0, j0, diag ? 1 : 0, 1, s));
      }
    }
  }
  for (size_t m = 0; m < P.mat.size(); ++m) {
    const Layer &La = a->layers[P.mat[m]], &Lb = b->layers[P.mat[m]];
    const int64_t D = (int64_t)La.d_in * La.d_out;
    if (D == 0 || P.one[m]) continue;
    const int nchunks = (int)cdiv(D, kDotChunk);
    if (diag) {
      for (int i0 = 0; i0 < na; i0 += P.ca) {
        const int ci = std::min(P.ca, na - i0);
        HIP_TRY(launch_gradient(elt, grad_args(La, elt, i0, ci, g1), s));
        HIP_TRY(launch_gdot(g1, ci, g1, ci, D, kDotChunk, 1, dparts, s));
        HIP_TRY(launch_kacc(dparts, nchunks, ci, ci, K, 1, i0, 0, 1, 1, s));
      }
      continue;
    }
    for (int j0 = 0; j0 < nb; j0 += P.cb) {
      const int cj = std::min(P.cb, nb - j0);
      if (!P.reuse_g) HIP_TRY(launch_gradient(elt, grad_args(Lb, elt, j0, cj, g2), s));
      for (int i0 = 0; i0 < na; i0 += P.ca) {
        const int ci = std::min(P.ca, na - i0);
        HIP_TRY(launch_gradient(elt, grad_args(La, elt, i0, ci, g1), s));
        HIP_TRY(launch_gdot(g1, ci, g2, cj, D, kDotChunk, 0, dparts, s));
        HIP_TRY(launch_kacc(dparts, nchunks, ci, cj, K, ld, i0, j0, 0, 1, s));
      }
    }
  }
  return DATTRI_OK;
}

}  // namespace

extern "C" {

dattri_status dattri_set_crossgram_cost_model(dattri_ctx* ctx, const dattri_crossgram_cost_model* m) {
  reset_error();
  if (!ctx || !m) return fail(DATTRI_E_INVALID_ARG, "ctx or model is NULL");
  const double v[] = {m->ghost_tflops, m->ghost_gbs, m->build_tflops, m->build_gbs, m->dot_gbs, m->onepass_tflops};
  for (double x : v)
    if (!(x > 0) || !std::isfinite(x)) return fail(DATTRI_E_INVALID_ARG, "rates must be finite and > 0");
  if (!(m->launch_us >= 0) || !std::isfinite(m->launch_us) || !(m->ghost_layer_us >= 0) ||
      !std::isfinite(m->ghost_layer_us))
    return fail(DATTRI_E_INVALID_ARG, "launch_us and ghost_layer_us must be finite and >= 0");
  ctx->xcost = *m;
  return DATTRI_OK;
}

dattri_status dattri_get_crossgram_cost_model(const dattri_ctx* ctx, dattri_crossgram_cost_model* m) {
  reset_error();
  if (!ctx || !m) return fail(DATTRI_E_INVALID_ARG, "ctx or model is NULL");
  *m = ctx->xcost;
  return DATTRI_OK;
}

dattri_status dattri_cross_gram_costs(int64_t n_a, int64_t n_b, int32_t T_a, int32_t T_b, int32_t d_in,
                                      int32_t d_out, int32_t elt_bytes, int64_t* factored_flops,
                                      int64_t* materialized_flops, int64_t* factored_bytes,
                                      int64_t* materialized_bytes) {
  reset_error();
  if (n_a < 0 || n_b < 0 || T_a < 0 || T_b < 0 || d_in < 0 || d_out < 0)
    return fail(DATTRI_E_INVALID_ARG, "sizes must be >= 0");
  if (elt_bytes != 2 && elt_bytes != 4) return fail(DATTRI_E_INVALID_ARG, "elt_bytes must be 2 or 4");
  const XCounts c = xcounts(n_a, n_b, T_a, T_b, d_in, d_out, elt_bytes);
  if (factored_flops) *factored_flops = c.f_flops;
  if (materialized_flops) *materialized_flops = c.m_flops;
  if (factored_bytes) *factored_bytes = c.f_bytes;
  if (materialized_bytes) *materialized_bytes = c.m_bytes;
  return DATTRI_OK;
}

dattri_status dattri_cross_gram_route(const dattri_ctx* a, const dattri_ctx* b, int32_t layer,
                                      dattri_route* chosen, double* pred_factored_us,
                                      double* pred_materialized_us) {
  reset_error();
  dattri_status st = check_pair(a, b);
  if (st != DATTRI_OK) return st;
  if (layer < 0 || layer >= (int32_t)a->layers.size())
    return fail(DATTRI_E_INVALID_ARG, "layer %d out of range", layer);
  const Layer &La = a->layers[layer], &Lb = b->layers[layer];
  double f, m;
  xpredict(a->xcost, La.n, Lb.n, La.T, Lb.T, La.d_in, La.d_out, a->elt, false, xone_ok(La, Lb, a->elt), &f, &m);
  if (chosen) *chosen = f <= m ? DATTRI_ROUTE_FACTORED : DATTRI_ROUTE_MATERIALIZED;
  if (pred_factored_us) *pred_factored_us = f;
  if (pred_materialized_us) *pred_materialized_us = m;
  return DATTRI_OK;
}

dattri_status dattri_cross_gram_workspace_bytes(const dattri_ctx* a, const dattri_ctx* b,
                                                dattri_route route, size_t* bytes) {
  reset_error();
  if (!bytes) return fail(DATTRI_E_INVALID_ARG, "bytes is NULL");
  dattri_status st = check_pair(a, b);
  if (st != DATTRI_OK) return st;
  XPlan P;
  st = build_xplan(a, b, route, false, P);
  if (st != DATTRI_OK) return st;
  *bytes = P.total;
  return DATTRI_OK;
}

dattri_status dattri_cross_gram(dattri_ctx* a, dattri_ctx* b, float* K, int64_t ld_k, void* workspace,
                                size_t ws_bytes, dattri_route route, void* stream) {
  reset_error();
  dattri_status st = check_pair(a, b);
  if (st != DATTRI_OK) return st;
  const int na = a->layers[0].n, nb = b->layers[0].n;
  if (ld_k < nb) return fail(DATTRI_E_INVALID_ARG, "ld_k=%lld is below n_b=%d", (long long)ld_k, nb);
  if ((int64_t)na * nb == 0) return DATTRI_OK;
  if (!K) return fail(DATTRI_E_INVALID_ARG, "K is NULL");
  XPlan P;
  st = build_xplan(a, b, route, false, P);
  if (st != DATTRI_OK) return st;
  st = check_ws(workspace, ws_bytes, P.total);
  if (st != DATTRI_OK) return st;
  return run_xplan(a, b, P, false, K, ld_k, (uint8_t*)workspace, (hipStream_t)stream);
}

dattri_status dattri_sq_norms_workspace_bytes(const dattri_ctx* ctx, dattri_route route, size_t* bytes) {
  reset_error();
  if (!bytes) return fail(DATTRI_E_INVALID_ARG, "bytes is NULL");
  dattri_status st = check_pair(ctx, ctx);
  if (st != DATTRI_OK) return st;
  XPlan P;
  st = build_xplan(ctx, ctx, route, true, P);
  if (st != DATTRI_OK) return st;
  *bytes = P.total;
  return DATTRI_OK;
}

dattri_status dattri_gradient_sq_norms(dattri_ctx* ctx, float* out, void* workspace, size_t ws_bytes,
                                       dattri_route route, void* stream) {
  reset_error();
  dattri_status st = check_pair(ctx, ctx);
  if (st != DATTRI_OK) return st;
  const int n = ctx->layers[0].n;
  if (n == 0) return DATTRI_OK;
  if (!out) return fail(DATTRI_E_INVALID_ARG, "out is NULL");
  XPlan P;
  st = build_xplan(ctx, ctx, route, true, P);
  if (st != DATTRI_OK) return st;
  st = check_ws(workspace, ws_bytes, P.total);
  if (st != DATTRI_OK) return st;
  return run_xplan(ctx, ctx, P, true, out, 1, (uint8_t*)workspace, (hipStream_t)stream);
}

}  // extern "C"
