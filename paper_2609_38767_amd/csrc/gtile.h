// One tile of a weight gradient (Eq. (1)) for bf16 factor blocks,
//   G[u0 .. u0 + 64 WM, v0 .. v0 + 64 WN] = sum_t g_t a_t^T   (float32),
// over a run of token rows, accumulated in MFMA registers.  Shared by the
// kernel that writes G (gradient_tr.hip) and the one-pass materialized-route
// kernel that projects each tile from its accumulators (gfused.hip).
//
// The contraction runs over tokens, the strided axis of both factors.  Token
// rows are loaded with coalesced 16-byte reads and stored in LDS as they are
// ([token][feature], rows padded by 32 bytes so the four rows one transposing
// read touches fall into different banks).  MFMA operands, which need eight
// consecutive tokens of one feature per lane, are read with the gfx950 LDS
// transpose read (ds_read_b64_tr_b16): within each group of 16 lanes, when lane
// 4r + a addresses row k0 + r at features m0 + 4a .. m0 + 4a + 3, lane j
// receives rows k0 .. k0 + 3 of feature m0 + j; two such reads give the 8
// tokens of a v_mfma_f32_32x32x16_bf16 operand.
//
// 4 waves in a 2 x 2 grid, each wave a (32 WM) x (32 WN) block of the tile
// (WM x WN MFMA tiles); stages of 32 tokens are double-buffered in LDS with
// the next stage prefetched into registers.  Rows past `rows` and features
// past d read zero (buffer range checks).
#pragma once
#include "device_common.h"
#include "internal.h"

namespace dattri {
namespace dev {

typedef short i16x4 __attribute__((ext_vector_type(4)));
#define DATTRI_LDS16(p) ((__attribute__((address_space(3))) ::dattri::dev::i16x4*)(p))

constexpr int kTrTokens = 32;  // tokens per stage

template <int WM, int WN>
struct GTile {
  static constexpr int TM = 64 * WM, TN = 64 * WN;         // tile rows (d_out side) x columns (d_in side)
  static constexpr int PB = TM * 2 + 32, PA = TN * 2 + 32;  // LDS row pitch in bytes
  static constexpr int CB = kTrTokens * TM / 8 / 256;      // 16-byte chunks per thread per stage (B side)
  static constexpr int CA = kTrTokens * TN / 8 / 256;      // (A side)
  static constexpr int kLdsBytes = 2 * kTrTokens * (PB + PA);
  static_assert(CB >= 1 && CA >= 1, "tile");
};

// One stage of token rows in registers: this thread's 16-byte chunks of the
// B rows (d_out side) and the A rows (d_in side).
template <int WM, int WN>
struct GStage {
  i32x4 b[GTile<WM, WN>::CB], a[GTile<WM, WN>::CA];
};

// Buffer resources over the token rows [0, rows) of the blocks whose row 0 is
// at b_rows / a_rows; rows past `rows` and features past d read zero.
struct GRows {
  rsrc_t rb, ra;
  int d_out, d_in;
};

__device__ inline GRows g_rows(const uint8_t* b_rows, const uint8_t* a_rows, int rows, int d_out, int d_in) {
  return GRows{make_rsrc(b_rows, (uint32_t)((int64_t)rows * d_out * 2)),
               make_rsrc(a_rows, (uint32_t)((int64_t)rows * d_in * 2)), d_out, d_in};
}

// Issue the loads of token rows t0 .. t0 + 31 of tile (u0, v0) into st.
template <int WM, int WN>
__device__ inline void g_load(const GRows& r, int t0, int u0, int v0, GStage<WM, WN>& st) {
  using C = GTile<WM, WN>;
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < C::CB; ++i) {
    const int c = tid + 256 * i, row = c / (C::TM / 8), fc = c % (C::TM / 8);
    const int u = u0 + fc * 8;
    const uint32_t off = u < r.d_out ? (uint32_t)(((int64_t)(t0 + row) * r.d_out + u) * 2) : kOOB;
    st.b[i] = load16(r.rb, off);
  }
#pragma unroll
  for (int i = 0; i < C::CA; ++i) {
    const int c = tid + 256 * i, row = c / (C::TN / 8), fc = c % (C::TN / 8);
    const int v = v0 + fc * 8;
    const uint32_t off = v < r.d_in ? (uint32_t)(((int64_t)(t0 + row) * r.d_in + v) * 2) : kOOB;
    st.a[i] = load16(r.ra, off);
  }
}

// acc[i][j] = G block (i, j) of this wave over token rows [0, rows) of tile
// (u0, v0).  On entry st holds (or has loads in flight for) the tile's first
// stage, rows 0 .. 31; the later stages are prefetched one ahead.  With
// next_u0 >= 0 the last stage also issues the loads of the first stage of
// tile (next_u0, next_v0) into st, so a caller walking a run of tiles keeps a
// load in flight across the tile boundary.  lds: GTile<WM, WN>::kLdsBytes of
// shared memory.  All 256 threads call this together; it ends with a barrier
// (lds may be reused after it).
template <int WM, int WN>
__device__ inline void g_tile_from(const GRows& r, int rows, int u0, int v0, int next_u0, int next_v0,
                                   uint8_t* lds, GStage<WM, WN>& st, f32x16 (&acc)[WM][WN]) {
  using C = GTile<WM, WN>;
  uint8_t* Bs[2] = {lds, lds + kTrTokens * C::PB};
  uint8_t* As[2] = {lds + 2 * kTrTokens * C::PB, lds + 2 * kTrTokens * C::PB + kTrTokens * C::PA};
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wu = wave >> 1, wv = wave & 1;

#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  auto swrite = [&](int sb) {
#pragma unroll
    for (int i = 0; i < C::CB; ++i) {
      const int c = tid + 256 * i, row = c / (C::TM / 8), fc = c % (C::TM / 8);
      *(i32x4*)(Bs[sb] + row * C::PB + fc * 16) = st.b[i];
    }
#pragma unroll
    for (int i = 0; i < C::CA; ++i) {
      const int c = tid + 256 * i, row = c / (C::TN / 8), fc = c % (C::TN / 8);
      *(i32x4*)(As[sb] + row * C::PA + fc * 16) = st.a[i];
    }
  };
  // transposed operand of K step ks (16 tokens) for the 32 features starting
  // at local column m: lane 16q + 4r + a reads row 16ks + 8(q/2) + 4h + r at
  // features m + 16(q%2) + 4a, h = 0, 1
  const int q = lane >> 4, rr = (lane >> 2) & 3, aa = lane & 3;
  auto frag = [&](const uint8_t* base, int pitch, int m, int ks) {
    const int row = ks * 16 + 8 * (q >> 1) + rr;
    const uint8_t* p = base + row * pitch + (m + 16 * (q & 1) + 4 * aa) * 2;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(DATTRI_LDS16(p));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(DATTRI_LDS16(p + 4 * pitch));
    const i32x4 w = {__builtin_bit_cast(int, __builtin_shufflevector(lo, lo, 0, 1)),
                     __builtin_bit_cast(int, __builtin_shufflevector(lo, lo, 2, 3)),
                     __builtin_bit_cast(int, __builtin_shufflevector(hi, hi, 0, 1)),
                     __builtin_bit_cast(int, __builtin_shufflevector(hi, hi, 2, 3))};
    return w;
  };

  const int nst = (rows + kTrTokens - 1) / kTrTokens;
  if (nst > 0) swrite(0);
  __syncthreads();
  for (int kk = 0; kk < nst; ++kk) {
    const int sb = kk & 1;
    if (kk + 1 < nst)
      g_load(r, (kk + 1) * kTrTokens, u0, v0, st);
    else if (next_u0 >= 0)
      g_load(r, 0, next_u0, next_v0, st);
#pragma unroll
    for (int ks = 0; ks < kTrTokens / 16; ++ks) {
      i32x4 fa[WM], fb[WN];
#pragma unroll
      for (int i = 0; i < WM; ++i) fa[i] = frag(Bs[sb], C::PB, wu * 32 * WM + i * 32, ks);
#pragma unroll
      for (int j = 0; j < WN; ++j) fb[j] = frag(As[sb], C::PA, wv * 32 * WN + j * 32, ks);
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[i]),
                                                             __builtin_bit_cast(bf16x8, fb[j]), acc[i][j], 0, 0, 0);
    }
    if (kk + 1 < nst) swrite(sb ^ 1);
    __syncthreads();
  }
  if (nst == 0 && next_u0 >= 0) g_load(r, 0, next_u0, next_v0, st);
}

// The same for a single tile: loads its first stage, then runs it.
template <int WM, int WN>
__device__ inline void g_tile(const uint8_t* b_rows, const uint8_t* a_rows, int rows, int d_out, int d_in,
                              int u0, int v0, uint8_t* lds, f32x16 (&acc)[WM][WN]) {
  const GRows r = g_rows(b_rows, a_rows, rows, d_out, d_in);
  GStage<WM, WN> st;
  if (rows > 0) g_load(r, 0, u0, v0, st);
  g_tile_from(r, rows, u0, v0, -1, 0, lds, st, acc);
}

}  // namespace dev
}  // namespace dattri
