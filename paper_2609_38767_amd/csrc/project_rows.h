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

// ---------------------------------------------------------------------------
// The same projection for bf16 blocks with 16-byte aligned rows, streamed
// through LDS by direct loads (buffer_load ... lds, no registers): each load
// instruction moves 8 rows x 128 bytes (2 k-blocks of 8 rows), so every L2
// request carries 128 bytes of a row instead of the 64 a register operand
// load gets (16 rows x 64 bytes), and many more bytes can be in flight per CU.
//
// A stage is 2 k-blocks (64 columns).  Each wave streams only its own RT x 16
// rows, into a private double buffer (RT x 16 x 128 bytes per stage), rows
// 128 bytes apart with their 16-byte chunks XOR-swizzled by (row & 7) so the
// MFMA fragment reads (16 rows x 16 bytes per lane group) spread over the
// banks: each lane fetches the chunk that lands in its fixed LDS slot.  The
// stage's 2 x NT projection fragments (NT / 2 per wave; NT = 2, 4 or 6, so
// the maps of up to three layers that share the input block ride along) go by
// direct load into a 3-slot ring shared by the workgroup.  Every wave issues
// exactly kDmaOps loads per stage, so "stage s has landed" is vmcnt(kDmaOps) while
// stage s + 1 is in flight and vmcnt(0) otherwise (any extra load issued later
// would only make that wait longer); one barrier per stage then publishes the
// shared fragments.  The wave's reads of a buffer finish (lgkmcnt(0)) before
// the load of stage s + 2 into it is issued, and the map slot it refills was
// last read in stage s - 1, before every wave passed stage s's barrier.
// K-blocks are contracted in the order of project_rows, so results are
// bitwise those of the register path.
template <int RT, int NT>
struct DmaLds {
  static_assert((2 * NT) % kWaves == 0 && 2 * NT <= 3 * kWaves, "NT / 2 projection fragments per wave and stage");
  static constexpr int kRowBytes = 128;                      // 2 k-blocks of 32 bf16
  static constexpr int kWaveStage = RT * 16 * kRowBytes;     // bytes per wave and stage
  static constexpr int kLoads = RT * 16 / 8;                 // 1 KiB row-group loads per stage
  static constexpr int kMapLoads = 2 * NT / kWaves;          // this wave's fragments per stage
  static constexpr int kDmaOps = kLoads + kMapLoads;
  static constexpr int kMapOff = kWaves * 2 * kWaveStage;
  static constexpr int kMapStage = 2 * NT * kFragBytes;
  static constexpr int kBytes = kMapOff + 3 * kMapStage;
};

template <int RT, int NT>
__device__ inline void project_rows_dma(const rsrc_t r, int r_wave, int nrows, int d, int64_t ld,
                                        const FragSrc<NT>& P, f32x4 (&acc)[RT][NT], uint8_t* lds) {
  using C = DmaLds<RT, NT>;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, m16 = lane & 15;
  const int wave = tid >> 6;
  const int nkb = (d + 31) / 32;
  const int nst = (nkb + 1) / 2;
  uint8_t* own = lds + wave * 2 * C::kWaveStage;
  // this wave's projection fragments of every stage: fragment f = wave *
  // kMapLoads + i of the stage is k-block 2s + f / NT of tile f % NT
  int f_kbl[C::kMapLoads], f_t[C::kMapLoads];
  int64_t f_stride[C::kMapLoads];
  const uint8_t* f_base[C::kMapLoads];  // (descriptors are built per load: no arrays of rsrc_t)
#pragma unroll
  for (int i = 0; i < C::kMapLoads; ++i) {
    const int f = wave * C::kMapLoads + i;
    f_kbl[i] = f / NT;
    f_t[i] = f % NT;
    // a select chain, not P.base[f_t[i]]: a runtime index would put the
    // arrays in memory (the compiler promotes them to LDS)
    const uint8_t* base = P.base[0];
    int64_t stride = P.stride[0];
#pragma unroll
    for (int t = 1; t < NT; ++t)
      if (f_t[i] == t) {
        base = P.base[t];
        stride = P.stride[t];
      }
    f_stride[i] = stride;
    f_base[i] = base;
  }

  auto issue = [&](int s) {
    uint8_t* xs = own + (s & 1) * C::kWaveStage;
#pragma unroll
    for (int i = 0; i < C::kLoads; ++i) {
      const int row_l = i * 8 + (lane >> 3);
      const int c = (lane & 7) ^ (row_l & 7);  // the logical chunk that lands in this lane's slot
      const int row = r_wave + row_l, col = s * 64 + c * 8;
      const uint32_t off = (row < nrows && col < d) ? (uint32_t)(((int64_t)row * ld + col) * 2) : kOOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, DATTRI_LDS_PTR(xs + i * 1024), 16, off, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < C::kMapLoads; ++i) {
      const int kb = 2 * s + f_kbl[i];
      uint8_t* ms = lds + C::kMapOff + (s % 3) * C::kMapStage + (f_kbl[i] * NT + f_t[i]) * kFragBytes;
      const uint32_t moff = (f_t[i] < P.nt && kb < nkb) ? (uint32_t)(kb * f_stride[i] + lane * 16) : kOOB;
      const rsrc_t rp = make_rsrc(f_base[i], (uint32_t)((int64_t)nkb * f_stride[i]));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rp, DATTRI_LDS_PTR(ms), 16, moff, 0, 0, 0);
    }
  };

  // the stage barrier: this wave's LDS reads done, then s_barrier.  An inline
  // barrier, because a fenced one (lds_barrier) makes the compiler wait for
  // every outstanding direct load (vmcnt(0)), the prefetched stage included.
  auto stage_barrier = [] { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };
  if (nst > 0) issue(0);
  if (nst > 1) issue(1);
  for (int s = 0; s < nst; ++s) {
    if (s + 1 < nst)
      wait_vmcnt_dma<C::kDmaOps>();
    else
      wait_vmcnt_dma<0>();
    stage_barrier();
    const uint8_t* xs = own + (s & 1) * C::kWaveStage;
    const uint8_t* ms = lds + C::kMapOff + (s % 3) * C::kMapStage;
#pragma unroll
    for (int kbl = 0; kbl < 2; ++kbl) {
      if (2 * s + kbl < nkb) {  // uniform
        i32x4 x[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          const int row_l = rt * 16 + m16;
          x[rt] = *(const i32x4*)(xs + row_l * C::kRowBytes + (((kbl * 4 + g) ^ (row_l & 7)) << 4));
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          if (t < P.nt) {
            const i32x4 pf = *(const i32x4*)(ms + (kbl * NT + t) * kFragBytes + lane * 16);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) acc[rt][t] = frag_mma<2>(x[rt], pf, acc[rt][t]);
          }
        }
      }
    }
    if (s + 2 < nst) {
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this wave's reads of the buffer are done
      issue(s + 2);
    }
  }
  stage_barrier();  // every wave is done with the ring before the next call refills it
}

}  // namespace dev
}  // namespace dattri
