// One 128 x 128 tile of a weight gradient (Eq. (1)) for bf16 factor blocks,
//   G[u0 .. u0 + 127, v0 .. v0 + 127] = sum_t g_t a_t^T   (float32),
// over a run of token rows, accumulated in MFMA registers.  Shared by the
// kernel that writes G (gradient_tr.hip), the one-pass materialized-route
// kernel that projects each tile from its accumulators (gfused.hip) and the
// one-pass materialized cross-Gram kernel (xone.hip).
//
// The contraction runs over tokens, the strided axis of both factors.  MFMA
// operands need eight consecutive tokens of one feature per lane; they are
// read from token rows in LDS with the gfx950 LDS transpose read
// (ds_read_b64_tr_b16): within each group of 16 lanes, when lane 4r + a
// addresses row k0 + r at features m0 + 4a .. m0 + 4a + 3, lane j receives
// rows k0 .. k0 + 3 of feature m0 + j; two such reads give the 8 tokens of a
// v_mfma_f32_32x32x16_bf16 operand.  4 waves in a 2 x 2 grid, each a 64 x 64
// block of the tile (2 x 2 MFMA tiles); rows past `rows` and features past d
// read zero (buffer range checks).
#pragma once
#include <type_traits>

#include "device_common.h"
#include "internal.h"

namespace dattri {
namespace dev {

typedef short i16x4 __attribute__((ext_vector_type(4)));

constexpr int kTrTokens = 32;  // tokens per stage

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

// The token rows are streamed into LDS by direct loads (buffer_load ... lds,
// no registers) through a ring of kGDmaStages stages, kGDmaStages - 1 of them
// in flight while one is contracted (one stage in flight, staged through
// registers, left the 8 MFMA of a stage waiting on memory latency).
//
// A stage holds 32 token rows of each side, 256 bytes (128 features) per row,
// rows unpadded: one direct load moves 1 KiB, 4 whole rows, lane l's 16 bytes
// landing in slot l % 16 of row l / 16.  The 16-byte chunks of token row t are
// XOR-swizzled by gswz(t) = 2 (t % 4) + 8 (t % 2) (each lane fetches the chunk
// that belongs in its slot), so the four rows that one transposing read takes
// 32 bytes from (16 lanes) lie in four different 32-byte bank groups, and the
// 64-byte pieces of a 32-lane half in four different 64-byte ones.
//
// Every wave issues exactly kGDmaOps direct loads per stage (2 per side), so
// stage k has landed when at most kGDmaOps x (stages issued after k) of the
// wave's loads are in flight; one barrier per stage then publishes all waves'
// loads and, since each wave's reads of the previous stage have finished
// (lgkmcnt(0) before the barrier), frees that stage's slot for the next load.
constexpr int kGDmaStages = 4;  // the waits below assume 2 stages in flight behind the current one
constexpr int kGDmaOps = 4;
static_assert(kGDmaStages == 4, "ring depth");
struct GDma {
  static constexpr int kRowBytes = 256;
  static constexpr int kSide = kTrTokens * kRowBytes;  // 8 KiB per side and stage
  static constexpr int kStage = 2 * kSide;             // B side, then A side
  static constexpr int kBytes = kGDmaStages * kStage;  // 64 KiB
};

__device__ constexpr int gswz(int t) { return 2 * (t & 3) + 8 * (t & 1); }

// acc[i][j] = G block (i, j) of this wave over token rows [0, rows) of the
// 128 x 128 tile (u0, v0); r as from g_rows over 16-byte aligned rows.  lds:
// GDma::kBytes of shared memory.  All 256 threads call this together.  Other
// vector-memory operations of the caller still in flight only lengthen the
// counted waits (a wait for at most N outstanding then covers more of the
// older loads).  Ends with a barrier (lds may be reused after it).
__device__ inline void g_tile_dma(const GRows& r, int rows, int u0, int v0, uint8_t* lds,
                                  f32x16 (&acc)[2][2]) {
  typedef __attribute__((address_space(3))) uint8_t lds_u8;
  lds_u8* const base = (lds_u8*)lds;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wu = wave >> 1, wv = wave & 1;
  auto stage_barrier = [] { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };

  // direct loads of this wave: 1 KiB blocks 2 wave and 2 wave + 1 of each
  // side, token rows 4 ib .. 4 ib + 3; this lane's row and logical chunk
  const int row0 = 8 * wave + (lane >> 4), row1 = row0 + 4;
  const int c0 = (lane & 15) ^ gswz(row0), c1 = (lane & 15) ^ gswz(row1);
  const bool bu0 = u0 + 8 * c0 < r.d_out, bu1 = u0 + 8 * c1 < r.d_out;
  const bool av0 = v0 + 8 * c0 < r.d_in, av1 = v0 + 8 * c1 < r.d_in;
  auto issue = [&](int st) {
    uint8_t* sb = lds + (st & (kGDmaStages - 1)) * GDma::kStage;
    const int t0 = st * kTrTokens;
    const bool ok0 = t0 + row0 < rows, ok1 = t0 + row1 < rows;
    const uint32_t ob0 = ok0 && bu0 ? (uint32_t)(((int64_t)(t0 + row0) * r.d_out + u0 + 8 * c0) * 2) : kOOB;
    const uint32_t ob1 = ok1 && bu1 ? (uint32_t)(((int64_t)(t0 + row1) * r.d_out + u0 + 8 * c1) * 2) : kOOB;
    const uint32_t oa0 = ok0 && av0 ? (uint32_t)(((int64_t)(t0 + row0) * r.d_in + v0 + 8 * c0) * 2) : kOOB;
    const uint32_t oa1 = ok1 && av1 ? (uint32_t)(((int64_t)(t0 + row1) * r.d_in + v0 + 8 * c1) * 2) : kOOB;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r.rb, DATTRI_LDS_PTR(sb + (2 * wave) * 1024), 16, ob0, 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r.rb, DATTRI_LDS_PTR(sb + (2 * wave + 1) * 1024), 16, ob1, 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r.ra, DATTRI_LDS_PTR(sb + GDma::kSide + (2 * wave) * 1024), 16, oa0,
                                             0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r.ra, DATTRI_LDS_PTR(sb + GDma::kSide + (2 * wave + 1) * 1024), 16,
                                             oa1, 0, 0, 0);
  };

  // transposed reads: lane 16q + 4rr + aa takes token row 8(q/2) + rr (and 4
  // further for the second half) at features m + 16(q%2) + 4aa of block m
  const int q = lane >> 4, rr = (lane >> 2) & 3, aa = lane & 3;
  const uint32_t rowoff = (uint32_t)((8 * (q >> 1) + rr) * GDma::kRowBytes + (aa & 1) * 8);
  uint32_t bo[2], ao[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    bo[i] = rowoff + (uint32_t)(((8 * wu + 4 * i + 2 * (q & 1) + (aa >> 1)) ^ gswz(rr)) << 4);
    ao[i] = GDma::kSide + rowoff + (uint32_t)(((8 * wv + 4 * i + 2 * (q & 1) + (aa >> 1)) ^ gswz(rr)) << 4);
  }
  // The transposing reads are issued as inline assembly and waited for by
  // hand: the compiler cannot tell which LDS bytes the intrinsic reads, so it
  // would wait for every direct load in flight (vmcnt(0)) before each one,
  // draining the ring.  LDS offsets are 32-bit addresses within the block.
  const uint32_t lds0 = (uint32_t)(uintptr_t)base;
  // the two reads of the operand of the 32-feature block at LDS address
  // addr, K step KS of the stage: token rows 16 KS + (0..3) of the lane's
  // group and, 4 rows further, 16 KS + (4..7).  The results are only read
  // after the wait that covers them takes them as operands (tie), so no
  // copy of a register the LDS has not yet written can be placed before it.
  struct Raw {
    i16x4 lo, hi;
  };
  auto rd = [](uint32_t addr, auto ks) {
    constexpr int o = decltype(ks)::value * 16 * GDma::kRowBytes;
    Raw x;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(x.lo) : "v"(addr), "i"(o));
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(x.hi) : "v"(addr), "i"(o + 4 * GDma::kRowBytes));
    return x;
  };
  auto tie = [](Raw (&x)[4], auto n) {
    asm volatile("s_waitcnt lgkmcnt(%8)"
                 : "+v"(x[0].lo), "+v"(x[0].hi), "+v"(x[1].lo), "+v"(x[1].hi), "+v"(x[2].lo), "+v"(x[2].hi),
                   "+v"(x[3].lo), "+v"(x[3].hi)
                 : "i"(decltype(n)::value));
  };
  auto op = [](const Raw& x) {
    const i32x4 w = {__builtin_bit_cast(int, __builtin_shufflevector(x.lo, x.lo, 0, 1)),
                     __builtin_bit_cast(int, __builtin_shufflevector(x.lo, x.lo, 2, 3)),
                     __builtin_bit_cast(int, __builtin_shufflevector(x.hi, x.hi, 0, 1)),
                     __builtin_bit_cast(int, __builtin_shufflevector(x.hi, x.hi, 2, 3))};
    return w;
  };
  using ks0_t = std::integral_constant<int, 0>;
  using ks1_t = std::integral_constant<int, 1>;
  // both K steps of a stage: 16 reads in flight, the first step's MFMA once
  // its 8 have landed (LDS returns in order), the second's after the rest.
  // x[0..1]: B-side blocks (rows of the wave's G block), x[2..3]: A side.
  auto stage = [&](uint32_t so, auto first) {
    uint32_t ad[4];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      ad[i] = lds0 + so + bo[i];
      ad[2 + i] = lds0 + so + ao[i];
    }
    Raw x0[4], x1[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) x0[i] = rd(ad[i], ks0_t{});
#pragma unroll
    for (int i = 0; i < 4; ++i) x1[i] = rd(ad[i], ks1_t{});
    tie(x0, std::integral_constant<int, 8>{});
    const f32x16 zero = {};
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, op(x0[i])),
                                                           __builtin_bit_cast(bf16x8, op(x0[2 + j])),
                                                           decltype(first)::value ? zero : acc[i][j], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);  // the first step's MFMA stay ahead of the second wait
    tie(x1, std::integral_constant<int, 0>{});
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, op(x1[i])),
                                                           __builtin_bit_cast(bf16x8, op(x1[2 + j])), acc[i][j], 0,
                                                           0, 0);
  };
  using first_t = std::integral_constant<bool, true>;
  using next_t = std::integral_constant<bool, false>;

  const int nst = (rows + kTrTokens - 1) / kTrTokens;
  if (nst <= 0) {  // uniform: no token rows, G is zero
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int x = 0; x < 16; ++x) acc[i][j][x] = 0.f;
    stage_barrier();
    return;
  }
#pragma unroll
  for (int p = 0; p < kGDmaStages - 1; ++p)
    if (p < nst) issue(p);
  for (int k = 0; k < nst; ++k) {
    const int ahead = nst - 1 - k;  // stages after k already issued: min(ahead, kGDmaStages - 2)
    if (ahead >= 2)
      wait_vmcnt_dma<2 * kGDmaOps>();
    else if (ahead == 1)
      wait_vmcnt_dma<kGDmaOps>();
    else
      wait_vmcnt_dma<0>();
    stage_barrier();
    if (k + kGDmaStages - 1 < nst) issue(k + kGDmaStages - 1);
    const uint32_t so = (uint32_t)((k & (kGDmaStages - 1)) * GDma::kStage);
    if (k == 0)
      stage(so, first_t{});
    else
      stage(so, next_t{});
  }
  stage_barrier();
}

}  // namespace dev
}  // namespace dattri
