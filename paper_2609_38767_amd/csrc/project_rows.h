// Streaming projection of row blocks onto 16-column tiles of a packed
// projection map: the building block of the factored route's kernels.
#pragma once
#include "device_common.h"
#include "internal.h"

namespace dattri {
namespace dev {

constexpr int kPanel = 4;  // k-blocks per LDS panel of projection fragments

// k-blocks of factor fragments prefetched ahead: about 8 KiB in flight per
// wave where the register budget of two waves per SIMD allows it, else 4 KiB.
constexpr int pd_of(int rt, int na, int nb) { return (rt >= 4 || na * (rt + nb) >= 24) ? 2 : 4; }

// Projection fragment source of up to NT output tiles: fragment (kb, t) of the
// packed map lives at base[t] + kb * stride[t] (bytes).
template <int NT>
struct FragSrc {
  const uint8_t* base[NT];
  int64_t stride[NT];
  int nt;  // tiles in use
};

// One operand fragment of X: row `row` (zero if >= nrows), EPL consecutive
// columns from `col` (zero past d), rows ld elements apart.
template <int ELT>
__device__ inline i32x4 load_frag_ld(rsrc_t r, int row, int nrows, int col, int d, int64_t ld,
                                     bool aligned) {
  constexpr int EPL = 16 / ELT;
  const int64_t row_off = (int64_t)row * ld;
  const bool row_ok = row < nrows;
  if (aligned) {
    const uint32_t off = (row_ok && col < d) ? (uint32_t)((row_off + col) * ELT) : kOOB;
    return load16(r, off);
  }
  uint32_t w[EPL];
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const uint32_t off = (row_ok && (col + j) < d) ? (uint32_t)((row_off + col + j) * ELT) : kOOB;
    w[j] = ELT == 2 ? load2(r, off) : load4(r, off);
  }
  i32x4 v;
  if (ELT == 2) {
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = (int32_t)(w[2 * j] | (w[2 * j + 1] << 16));
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = (int32_t)w[j];
  }
  return v;
}

// acc[rt][t] += X[rows, 0:d] * P[0:d, tile t] over all k-blocks of the d
// columns.  X rows r_wave + rt*16 + (lane & 15) of descriptor `r`, ld elements
// apart (rows >= nrows and columns >= d read as zero).  All 256 threads must
// call this together.
template <int ELT, bool AL, int RT, int NT, int NTL, int kPD>
__device__ inline void project_rows(const rsrc_t r, int r_wave, int nrows, int d, int64_t ld,
                                    const FragSrc<NT>& P, f32x4 (&acc)[RT][NT],
                                    uint8_t (*pan)[kPanel][NTL][kFragBytes]) {
  constexpr int EPL = 16 / ELT, KR = 4 * EPL;
  static_assert(kPanel % kPD == 0, "ring slots must be static inside a panel");
  // A panel holds kPanel * NT fragments of 1 KiB; fragment f = w + 4*i is
  // copied by wave w (one 16-byte load per lane), so every index is static.
  constexpr int NF = kPanel * NT;
  constexpr int CPT = (NF + kWaves - 1) / kWaves;  // fragments per wave
  static_assert(NT <= NTL, "panel too small");
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, m16 = lane & 15;
  const int wave = tid >> 6;
  const int nkb = (d + KR - 1) / KR;
  const int npan = (nkb + kPanel - 1) / kPanel;

  auto load_panel = [&](int p, i32x4 (&st)[CPT]) {
#pragma unroll
    for (int i = 0; i < CPT; ++i)
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const int f = w + kWaves * i, t = f % NT, kbl = f / NT;
        if (f < NF && wave == w) {
          const int kb = min(p * kPanel + kbl, nkb - 1);
          st[i] = (t < P.nt) ? *(const i32x4*)(P.base[t] + kb * P.stride[t] + lane * 16)
                             : i32x4{0, 0, 0, 0};
        }
      }
  };
  auto store_panel = [&](int buf, const i32x4 (&st)[CPT]) {
#pragma unroll
    for (int i = 0; i < CPT; ++i)
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const int f = w + kWaves * i, t = f % NT, kbl = f / NT;
        if (f < NF && wave == w) *(i32x4*)(&pan[buf][kbl][t][lane * 16]) = st[i];
      }
  };
  auto load_x = [&](int kb, i32x4 (&x)[RT]) {
    const int col = kb * KR + g * EPL;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) x[rt] = load_frag_ld<ELT>(r, r_wave + rt * 16 + m16, nrows, col, d, ld, AL);
  };

  i32x4 stage[CPT];
  i32x4 ring[kPD][RT];
  load_panel(0, stage);
#pragma unroll
  for (int s = 0; s < kPD; ++s) load_x(s, ring[s]);
  store_panel(0, stage);
  lds_barrier();
  for (int p = 0; p < npan; ++p) {
    const int buf = p & 1;
    if (p + 1 < npan) load_panel(p + 1, stage);
#pragma unroll
    for (int kbl = 0; kbl < kPanel; ++kbl) {
      const int kb = p * kPanel + kbl;
      if (kb < nkb) {
        i32x4 x[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) x[rt] = ring[kbl % kPD][rt];
        load_x(kb + kPD, ring[kbl % kPD]);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          if (t < P.nt) {
            const i32x4 pf = *(const i32x4*)(&pan[buf][kbl][t][lane * 16]);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) acc[rt][t] = frag_mma<ELT>(x[rt], pf, acc[rt][t]);
          }
        }
      }
    }
    if (p + 1 < npan) store_panel(buf ^ 1, stage);
    lds_barrier();
  }
}

}  // namespace dev
}  // namespace dattri
