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
#include <type_traits>

#include "device_common.h"
#include "internal.h"

namespace dattri {
namespace dev {

typedef short i16x4 __attribute__((ext_vector_type(4)));

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
  typedef __attribute__((address_space(3))) uint8_t lds_u8;
  typedef __attribute__((address_space(3))) i32x4 lds_i32x4;
  // LDS addresses as 32-bit offsets from one local-address-space base: a
  // generic pointer per access would cost a null check and 64-bit arithmetic
  lds_u8* const base = (lds_u8*)lds;
  constexpr uint32_t kB0 = 0, kB1 = kTrTokens * C::PB;
  constexpr uint32_t kA0 = 2 * kTrTokens * C::PB, kA1 = kA0 + kTrTokens * C::PA;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wu = wave >> 1, wv = wave & 1;

  // this thread's fixed offsets within a stage buffer: the 16-byte chunks it
  // stores, and the rows and features its transposed reads start at (lane
  // 16q + 4r + a reads row 8(q/2) + r of a 16-token step at features
  // m + 16(q%2) + 4a, and the same 4 rows further for the second half)
  uint32_t wb[C::CB], wa[C::CA];
#pragma unroll
  for (int i = 0; i < C::CB; ++i) {
    const int c = tid + 256 * i;
    wb[i] = (uint32_t)((c / (C::TM / 8)) * C::PB + (c % (C::TM / 8)) * 16);
  }
#pragma unroll
  for (int i = 0; i < C::CA; ++i) {
    const int c = tid + 256 * i;
    wa[i] = (uint32_t)((c / (C::TN / 8)) * C::PA + (c % (C::TN / 8)) * 16);
  }
  const int q = lane >> 4, rr = (lane >> 2) & 3, aa = lane & 3;
  const uint32_t rb_lane = (uint32_t)((8 * (q >> 1) + rr) * C::PB + (wu * 32 * WM + 16 * (q & 1) + 4 * aa) * 2);
  const uint32_t ra_lane = (uint32_t)((8 * (q >> 1) + rr) * C::PA + (wv * 32 * WN + 16 * (q & 1) + 4 * aa) * 2);

  auto swrite = [&](int sb) {
    const uint32_t ob = sb ? kB1 : kB0, oa = sb ? kA1 : kA0;
#pragma unroll
    for (int i = 0; i < C::CB; ++i) *(lds_i32x4*)(base + ob + wb[i]) = st.b[i];
#pragma unroll
    for (int i = 0; i < C::CA; ++i) *(lds_i32x4*)(base + oa + wa[i]) = st.a[i];
  };
  // transposed operand of K step ks (16 tokens), 32-feature block i
  auto frag = [&](uint32_t off, int pitch) {
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(base + off));
    const i16x4 hi =
        __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(base + off + 4 * pitch));
    const i32x4 w = {__builtin_bit_cast(int, __builtin_shufflevector(lo, lo, 0, 1)),
                     __builtin_bit_cast(int, __builtin_shufflevector(lo, lo, 2, 3)),
                     __builtin_bit_cast(int, __builtin_shufflevector(hi, hi, 0, 1)),
                     __builtin_bit_cast(int, __builtin_shufflevector(hi, hi, 2, 3))};
    return w;
  };
  // one K step of the stage in buffer sb; the first step of a tile starts
  // its accumulators from a zero operand instead of zeroed registers
  auto step = [&](int sb, int ks, auto first) {
    i32x4 fa[WM], fb[WN];
    const uint32_t ob = (sb ? kB1 : kB0) + rb_lane + (uint32_t)(ks * 16 * C::PB);
    const uint32_t oa = (sb ? kA1 : kA0) + ra_lane + (uint32_t)(ks * 16 * C::PA);
#pragma unroll
    for (int i = 0; i < WM; ++i) fa[i] = frag(ob + i * 64, C::PB);
#pragma unroll
    for (int j = 0; j < WN; ++j) fb[j] = frag(oa + j * 64, C::PA);
    const f32x16 zero = {};
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[i]),
                                                           __builtin_bit_cast(bf16x8, fb[j]),
                                                           decltype(first)::value ? zero : acc[i][j], 0, 0, 0);
  };
  using first_t = std::integral_constant<bool, true>;
  using next_t = std::integral_constant<bool, false>;

  const int nst = (rows + kTrTokens - 1) / kTrTokens;
  if (nst > 0) swrite(0);
  __syncthreads();
  if (nst == 0) {  // uniform: no token rows, G is zero
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
    if (next_u0 >= 0) g_load(r, 0, next_u0, next_v0, st);
    return;
  }
  for (int kk = 0; kk < nst; ++kk) {
    const int sb = kk & 1;
    // one call site for both prefetches (the next stage, or the first stage of
    // the next tile), so the stage registers are loaded in place
    const bool more = kk + 1 < nst;
    if (more || next_u0 >= 0)
      g_load(r, more ? (kk + 1) * kTrTokens : 0, more ? u0 : next_u0, more ? v0 : next_v0, st);
    if (kk == 0)
      step(sb, 0, first_t{});
    else
      step(sb, 0, next_t{});
#pragma unroll
    for (int ks = 1; ks < kTrTokens / 16; ++ks) step(sb, ks, next_t{});
    if (kk + 1 < nst) swrite(sb ^ 1);
    __syncthreads();
  }
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
