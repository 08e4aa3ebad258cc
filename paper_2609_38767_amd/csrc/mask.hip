// Random coordinate masks of the weight gradient, gathered from the factors
// (App. A.2 "Random maps": entry (r, c) of DW is sum_t g_{t,r} a_{t,c}, Eq. 1,
// so the kept entries need |M| products per token position and DW is never
// formed).
//
// One workgroup per (mask layer, example, token chunk, group of up to
// kMaskGroup = 16384 entries).  Each stage holds consecutive token rows of A
// and of B.  For 16-byte rows it holds, of each row, only the 16-byte-aligned
// slice that covers the group's entries (a layer's entries are dealt to its
// groups in order along the wider side of DW, so a group of a layer with g
// groups stages about 1/g of that side), packed densely so that more tokens
// fit a stage; the slices are moved by direct global-to-LDS loads (1 KiB per
// wave instruction, no registers) into one of two buffers while the other is
// gathered.  Rows that are not 16-byte multiples take a plain copy of whole
// rows into one buffer.  Every thread owns 64 entries (each (r, c) pair
// packed in one register) and adds b[r_e] * a[c_e] for each staged token, in
// token order (deterministic); the products of bf16 values are exact in
// float32 (bf16 layers up to 32768 wide take them through v_dot2_f32_bf16,
// gather_rows_b16).  Every group restages the narrow side's token rows, so
// groups are made as large as two waves per SIMD allow: ten masks of 8192
// entries take 5 groups instead of 10.  The entries come in the slot order
// of the layer's table, arranged at bind time so that the 32 lanes of a
// half-wave mostly read distinct LDS banks, and each sum is written at the
// entry's position in mask order.  Whole groups and the partial last group of a layer run in
// separate launches (the partial one bounds its slots).
//
// Whole groups of bf16 layers whose slices fit 8 KiB take mask_fixed_kernel
// instead: it stages token pairs, so each 32-bit LDS read serves two tokens
// of an entry (half the reads per product of the kernel above), and keeps
// every slice at a fixed place so that no address is formed per token.
#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

template <int ELT>
__device__ inline float lds_elem(const uint8_t* p, int i) {
  if (ELT == 2) return bf16_bits_to_f32(((const uint16_t*)p)[i]);
  return ((const float*)p)[i];
}

// Copies `bytes` bytes from global src to LDS dst (both 16-byte aligned when
// AL; bytes a multiple of 16 when AL, of ELT otherwise).
template <int ELT, bool AL>
__device__ inline void copy_rows(uint8_t* dst, const uint8_t* src, int64_t bytes) {
  if (AL) {
    const int64_t n16 = bytes / 16;
    for (int64_t i = threadIdx.x; i < n16; i += 256) ((i32x4*)dst)[i] = ((const i32x4*)src)[i];
  } else {
    const int64_t n = bytes / ELT;
    for (int64_t i = threadIdx.x; i < n; i += 256) {
      if (ELT == 2)
        ((uint16_t*)dst)[i] = ((const uint16_t*)src)[i];
      else
        ((uint32_t*)dst)[i] = ((const uint32_t*)src)[i];
    }
  }
}

#define LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

__device__ inline void wait_vm0() {  // vmcnt(0), other counters untouched
  __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));
}

// Direct global-to-LDS copy of `bytes` (whole token rows, 16-byte aligned)
// from byte offset `off` of descriptor r into dst: one 1 KiB chunk per wave
// instruction, lane l moving bytes 16 l .. 16 l + 15 of its chunk; chunks are
// dealt to the 4 waves in turn.  Bytes past the descriptor's range land as
// zero.  dst must have room for the size rounded up to 1 KiB.
__device__ inline void dma_block(const rsrc_t r, uint32_t off, int bytes, uint8_t* dst, int wave, int lane) {
  const int chunks = (bytes + 1023) >> 10;
  for (int c = wave; c < chunks; c += 4)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LDS_PTR(dst + c * 1024), 16, off + c * 1024 + lane * 16, 0, 0, 0);
}

// Direct copy of the byte slice [s0, s0 + seg) of nt consecutive token rows
// (row bytes apart, from token ts) into dst as [nt][seg], seg a multiple of 16:
// 16-byte chunk i of that image is token i / n16, chunk i % n16 (n16 = seg /
// 16; the quotient is the high word of i * magic, magic = ceil(2^32 / n16),
// exact for i < 2^17 and n16 < 2^13).  One 1 KiB run of chunks per wave
// instruction, dealt to the 4 waves in turn; chunks past the image land as
// zero, so dst needs room for nt * seg rounded up to 1 KiB.
__device__ inline void dma_slices(const rsrc_t r, int ts, int nt, int row, int s0, int seg, uint32_t magic,
                                  uint8_t* dst, int wave, int lane) {
  const int n16 = seg >> 4, total = nt * n16, runs = (total + 63) >> 6;
  for (int c = wave; c < runs; c += 4) {
    const int i = c * 64 + lane;
    const int u = n16 == 1 ? i : (int)__umulhi((uint32_t)i, magic);
    const uint32_t off = i < total ? (uint32_t)((ts + u) * row + s0 + 16 * (i - u * n16)) : kOOB;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LDS_PTR(dst + c * 1024), 16, off, 0, 0, 0);
  }
}

// acc[j] += b[r_j] * a[c_j] over the nt staged token rows (token order);
// rc[j] = r_j << 16 | c_j.  FULL: every slot holds an entry.  Else the slots
// j < 8 * ceil(nj / 8) are gathered (nj uniform over the workgroup, so each
// block test is a scalar branch); lanes past the group's entries hold rc = 0
// (element 0 of each staged row) and their sums are never stored.  The empty
// asm keeps the unpacked offsets out of registers across tokens (they would
// double the register footprint and halve the waves per SIMD).
template <int ELT, bool FULL>
__device__ __forceinline__ void gather_rows(const uint8_t* sa, const uint8_t* sb, int nt, int a_row, int b_row,
                                            int nj, uint32_t (&rc)[kMaskPerThread],
                                            float (&acc)[kMaskPerThread]) {
  for (int t = 0; t < nt; ++t) {
    const uint8_t* ar = sa + t * a_row;
    const uint8_t* br = sb + t * b_row;
#pragma unroll
    for (int jb = 0; jb < kMaskPerThread; jb += 8) {
      if (FULL || jb < nj) {
#pragma unroll
        for (int j = jb; j < jb + 8; ++j) {
          asm volatile("" : "+v"(rc[j]));
          acc[j] = fmaf(lds_elem<ELT>(br, (int)(rc[j] >> 16)), lds_elem<ELT>(ar, (int)(rc[j] & 0xFFFFu)), acc[j]);
        }
      }
    }
  }
}

// The same for bf16 layers whose token rows are at most 64 KiB (both d <=
// 32768): rc[j] holds the entry's byte offsets within a staged row, 2 r_j << 16
// | 2 c_j, so each LDS address is one add of a 16-bit field (SDWA), and each
// value is read zero-extended: as a bf16 pair (value, 0), v_dot2_f32_bf16
// gives value_b * value_a + acc with the product exact and one rounding, the
// same as the float32 FMA, with no conversion.  3 vector instructions per
// multiply-add instead of 7.
template <bool FULL>
__device__ __forceinline__ void gather_rows_b16(const uint8_t* sa, const uint8_t* sb, int nt, int a_row, int b_row,
                                                int nj, uint32_t (&rc)[kMaskPerThread],
                                                float (&acc)[kMaskPerThread]) {
  typedef __attribute__((address_space(3))) uint8_t lds_u8;
  typedef __attribute__((address_space(3))) uint16_t lds_u16;
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const uint32_t a0 = (uint32_t)(uintptr_t)(lds_u8*)sa, b0 = (uint32_t)(uintptr_t)(lds_u8*)sb;
  for (int t = 0; t < nt; ++t) {
    const uint32_t ar = a0 + (uint32_t)(t * a_row), br = b0 + (uint32_t)(t * b_row);
#pragma unroll
    for (int jb = 0; jb < kMaskPerThread; jb += 8) {
      if (FULL || jb < nj) {
#pragma unroll
        for (int j = jb; j < jb + 8; ++j) {
          asm volatile("" : "+v"(rc[j]));  // as in gather_rows: no unpacked offsets held across tokens
          const uint32_t vb = *(const lds_u16*)(uintptr_t)(br + (rc[j] >> 16));
          const uint32_t va = *(const lds_u16*)(uintptr_t)(ar + (rc[j] & 0xFFFFu));
          acc[j] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, vb), __builtin_bit_cast(bf16x2, va),
                                                   acc[j], false);
        }
      }
    }
  }
}

template <int ELT, bool AL, bool FULL, bool B16>
__global__ __launch_bounds__(256, 2) void mask_kernel(const MaskItem* __restrict__ items,
                                                   const MaskTask* __restrict__ tasks,
                                                   float* __restrict__ partials) {
  extern __shared__ __align__(1024) uint8_t stage[];
  const MaskItem it = items[blockIdx.x];
  if (it.task < 0) return;  // padding item
  const MaskTask& M = tasks[it.task];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, ex = it.example;
  int t_eff = M.T;
  if (M.lengths) t_eff = min(max(M.lengths[ex], 0), M.T);
  const int t0 = it.chunk * M.chunk_tokens, t1 = min(t_eff, t0 + M.chunk_tokens);
  const int e0 = it.group * kMaskGroup, ne = min(kMaskGroup, M.m - e0);
  const int nj = (ne + 255) / 256;  // slots per thread holding entries (uniform)
  // entry (r, c) packed as r << 16 | c (both below 2^16: a staged token row
  // of A and B fits in LDS); B16 (bf16 rows of at most 64 KiB): as byte
  // offsets 2 r << 16 | 2 c
  static_assert(!B16 || ELT == 2, "byte-offset gather is bf16 only");
  constexpr uint32_t sh = B16 ? 1u : 0u;
  const int a_row = M.d_in * ELT, b_row = M.d_out * ELT;
  const uint8_t* ga = (const uint8_t*)M.A + ((int64_t)ex * M.T) * a_row;
  const uint8_t* gb = (const uint8_t*)M.B + ((int64_t)ex * M.T) * b_row;
  // Aligned rows: the staged part of each token row is the group's slice
  // from the table (16-byte aligned, covering its columns c of A and rows r
  // of B); entries address the slices.  Else whole rows.
  int sa0 = 0, sb0 = 0, seg_a = a_row, seg_b = b_row;
  if (AL) {
    const int32_t* sl = M.slices + 4 * it.group;
    sa0 = sl[0]; seg_a = sl[1]; sb0 = sl[2]; seg_b = sl[3];
  }
  const uint32_t rb = (uint32_t)(sb0 / ELT), cb = (uint32_t)(sa0 / ELT);
  uint32_t rc[kMaskPerThread];
  float acc[kMaskPerThread];
#pragma unroll
  for (int j = 0; j < kMaskPerThread; ++j) {
    const int e = tid + 256 * j;
    rc[j] = e < ne ? (((uint32_t)M.rows[e0 + e] - rb) << (16 + sh)) | (((uint32_t)M.cols[e0 + e] - cb) << sh) : 0u;
    acc[j] = 0.f;
  }

  auto gather = [&](const uint8_t* sa, const uint8_t* sb, int nt, int a_stride, int b_stride) {
    if constexpr (B16)
      gather_rows_b16<FULL>(sa, sb, nt, a_stride, b_stride, nj, rc, acc);
    else
      gather_rows<ELT, FULL>(sa, sb, nt, a_stride, b_stride, nj, rc, acc);
  };

  if (AL) {
    // two stage buffers of the planned size (stage_tokens whole rows, each
    // part rounded up to 1 KiB); each holds [A slices | B slices] of as many
    // tokens as fit (at least stage_tokens, at most 16)
    const int buf = ((M.stage_tokens * a_row + 1023) & ~1023) + ((M.stage_tokens * b_row + 1023) & ~1023);
    auto fits = [&](int t) { return ((t * seg_a + 1023) & ~1023) + ((t * seg_b + 1023) & ~1023) <= buf; };
    int TS = M.stage_tokens;
    while (TS < 16 && fits(TS + 1)) ++TS;
    const int a_part = (TS * seg_a + 1023) & ~1023;
    const uint32_t mag_a = (uint32_t)(0xFFFFFFFFu / (uint32_t)(seg_a >> 4)) + 1u;
    const uint32_t mag_b = (uint32_t)(0xFFFFFFFFu / (uint32_t)(seg_b >> 4)) + 1u;
    // descriptors end at row t1: rows past the chunk land as zero
    const rsrc_t r_a = make_rsrc(ga, (uint32_t)((int64_t)t1 * a_row));
    const rsrc_t r_b = make_rsrc(gb, (uint32_t)((int64_t)t1 * b_row));
    const int n_st = t1 > t0 ? (t1 - t0 + TS - 1) / TS : 0;
    const bool whole = seg_a == a_row && seg_b == b_row;  // uniform: contiguous stages
    auto issue = [&](int st) {
      const int ts = t0 + st * TS, nt = min(TS, t1 - ts);
      uint8_t* sa = stage + (st & 1) * buf;
      if (whole) {
        dma_block(r_a, (uint32_t)(ts * a_row), nt * a_row, sa, wave, lane);
        dma_block(r_b, (uint32_t)(ts * b_row), nt * b_row, sa + a_part, wave, lane);
      } else {
        dma_slices(r_a, ts, nt, a_row, sa0, seg_a, mag_a, sa, wave, lane);
        dma_slices(r_b, ts, nt, b_row, sb0, seg_b, mag_b, sa + a_part, wave, lane);
      }
    };
    if (n_st > 0) issue(0);
    for (int st = 0; st < n_st; ++st) {  // uniform trip count
      wait_vm0();        // this wave's loads of stage st have landed
      __syncthreads();   // every wave's have; the other buffer's readers are done
      if (st + 1 < n_st) issue(st + 1);
      const uint8_t* sa = stage + (st & 1) * buf;
      gather(sa, sa + a_part, min(TS, t1 - (t0 + st * TS)), seg_a, seg_b);
    }
  } else {
    const int TS = M.stage_tokens;
    uint8_t* sa = stage;
    uint8_t* sb = stage + (((int64_t)TS * a_row + 15) & ~(int64_t)15);
    for (int ts = t0; ts < t1; ts += TS) {  // uniform trip count
      const int nt = min(TS, t1 - ts);
      __syncthreads();  // the previous stage's readers are done
      copy_rows<ELT, false>(sa, ga + (int64_t)ts * a_row, (int64_t)nt * a_row);
      copy_rows<ELT, false>(sb, gb + (int64_t)ts * b_row, (int64_t)nt * b_row);
      __syncthreads();
      gather(sa, sb, nt, a_row, b_row);
    }
  }
  float* dst = partials + M.partial_base + ((int64_t)ex * M.n_chunks + it.chunk) * M.m;
#pragma unroll
  for (int j = 0; j < kMaskPerThread; ++j)
    if (tid + 256 * j < ne) dst[M.pos[e0 + tid + 256 * j]] = acc[j];
}

// Fixed-slot gather: whole groups of bf16 layers with 16-byte rows whose slices
// fit kMaskSlot bytes.  A stage is kMaskSlotPairs token pairs (t, t + 1), held
// in one of two buffers (kFixBuf bytes each) as pair rows: feature f of the A
// slice at byte mask_pair_offset(f) of the pair's A row is the bf16 pair
// (A[t][f], A[t + 1][f]), its B row likewise.  So one 32-bit LDS read per side
// serves both tokens of an entry, and v_dot2_f32_bf16 adds both products (exact
// in float32) to the entry's sum.  The pairs are formed in registers (16 bytes
// of each of two token rows per thread and side, interleaved by 16-bit halves,
// written as two 16-byte chunks into the two halves of the pair row, see
// mask_pair_offset) while the next stage's loads are in flight.  Every entry
// keeps both LDS offsets in one register (16 bits each), unpacked once per
// stage into the buffer's addresses; the pair offsets are instruction
// immediates.  A pair's tokens past the chunk's end read as zero (the
// descriptors end there) and add nothing.  512 threads hold the group's 16384
// entries (slot e to thread e % 512 at step e / 512: the table's half-waves are
// still 32 consecutive slots); one workgroup per CU.
constexpr int kFixSide = 2 * kMaskSlot;                  // bytes of a pair row
constexpr int kFixPairRows = 2 * kFixSide;               // A row | B row of one pair
constexpr int kFixBuf = kMaskSlotPairs * kFixPairRows;   // one stage
static_assert(2 * kFixBuf == (int)kMaskSlotLds, "two stage buffers");
static_assert((kMaskSlotPairs - 1) * kFixPairRows + 2 * kFixSide <= 65536, "pair offsets are DS immediates");
constexpr int kFixThreads = 512;
constexpr int kFixPer = kMaskGroup / kFixThreads;  // entries per thread
static_assert(kMaskSlot / 16 == kFixThreads, "one 16-byte chunk of each slice per thread");

template <int P>
__device__ __forceinline__ void gather_pairs(const uint8_t* stage, const uint32_t (&rc)[kFixPer],
                                             float (&acc)[kFixPer]) {
  typedef __attribute__((address_space(3))) uint8_t lds_u8;
  typedef __attribute__((address_space(3))) uint32_t lds_u32;
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const lds_u8* sp = (const lds_u8*)stage + P * kFixBuf;
#pragma unroll
  for (int j = 0; j < kFixPer; ++j) {
    uint32_t x = rc[j];
    asm volatile("" : "+v"(x));  // unpack per stage: no unpacked offsets held across stages
    const lds_u8* pb = sp + (x >> 16);
    const lds_u8* pa = sp + (x & 0xFFFFu);
#pragma unroll
    for (int q = 0; q < kMaskSlotPairs; ++q) {
      const uint32_t vb = *(const lds_u32*)(pb + q * kFixPairRows);
      const uint32_t va = *(const lds_u32*)(pa + q * kFixPairRows);
      acc[j] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, vb), __builtin_bit_cast(bf16x2, va),
                                               acc[j], false);
    }
  }
}

// 16 bytes at token rows t and t + 1 (x0, x1) -> 8 pairs (x0.h[f], x1.h[f]),
// features 0..3 in lo, 4..7 in hi
__device__ __forceinline__ void pair_halves(const i32x4& x0, const i32x4& x1, i32x4& lo, i32x4& hi) {
  uint32_t o[8];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const uint32_t a = (uint32_t)x0[w], b = (uint32_t)x1[w];
    o[2 * w] = (a & 0xFFFFu) | (b << 16);
    o[2 * w + 1] = (a >> 16) | (b & 0xFFFF0000u);
  }
  lo = i32x4{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
  hi = i32x4{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
}

__global__ __launch_bounds__(kFixThreads, 2) void mask_fixed_kernel(const MaskItem* __restrict__ items,
                                                                    const MaskTask* __restrict__ tasks,
                                                                    float* __restrict__ partials) {
  extern __shared__ __align__(1024) uint8_t stage[];
  const MaskItem it = items[blockIdx.x];
  if (it.task < 0) return;  // padding item
  const MaskTask& M = tasks[it.task];
  const int tid = threadIdx.x, ex = it.example;
  int t_eff = M.T;
  if (M.lengths) t_eff = min(max(M.lengths[ex], 0), M.T);
  const int t0 = it.chunk * M.chunk_tokens;
  const int t1 = __builtin_amdgcn_readfirstlane(min(t_eff, t0 + M.chunk_tokens));
  const int e0 = it.group * kMaskGroup;
  const int a_row = __builtin_amdgcn_readfirstlane(M.d_in * 2), b_row = __builtin_amdgcn_readfirstlane(M.d_out * 2);
  const int32_t* sl = M.slices + 4 * it.group;
  const int sa0 = __builtin_amdgcn_readfirstlane(sl[0]), seg_a = __builtin_amdgcn_readfirstlane(sl[1]);
  const int sb0 = __builtin_amdgcn_readfirstlane(sl[2]), seg_b = __builtin_amdgcn_readfirstlane(sl[3]);
  // entry (r, c): byte offsets of its pair-row words in a stage, B << 16 | A
  uint32_t rc[kFixPer];
  float acc[kFixPer];
#pragma unroll
  for (int j = 0; j < kFixPer; ++j) {
    const int e = e0 + tid + kFixThreads * j;
    rc[j] = ((uint32_t)kFixSide + mask_pair_offset((uint32_t)(M.rows[e] - sb0 / 2))) << 16 |
            mask_pair_offset((uint32_t)(M.cols[e] - sa0 / 2));
    acc[j] = 0.f;
  }
  const uint8_t* ga = (const uint8_t*)M.A + ((int64_t)ex * M.T) * a_row;
  const uint8_t* gb = (const uint8_t*)M.B + ((int64_t)ex * M.T) * b_row;
  // descriptors end at row t1: token rows past the chunk read as zero
  const rsrc_t r_a = make_rsrc(ga, (uint32_t)((int64_t)t1 * a_row));
  const rsrc_t r_b = make_rsrc(gb, (uint32_t)((int64_t)t1 * b_row));
  // this thread's 16-byte chunk of each slice (features 8 tid .. 8 tid + 7);
  // a chunk past its slice starts at 2^31, which with any token row's offset
  // added stays past the descriptor's range (below 2^31 bytes), so it loads
  // as zero into pair-row space no entry reads: no branches, so the loads'
  // wait counts stay exact
  constexpr uint32_t kPast = 0x80000000u;
  const uint32_t ca = tid < (seg_a >> 4) ? (uint32_t)(sa0 + 16 * tid) : kPast;
  const uint32_t cb = tid < (seg_b >> 4) ? (uint32_t)(sb0 + 16 * tid) : kPast;
  constexpr int kTok = 2 * kMaskSlotPairs;  // tokens per stage
  const int n_st = t1 > t0 ? (t1 - t0 + kTok - 1) / kTok : 0;
  i32x4 xa[kTok], xb[kTok];  // the next stage's token rows (this thread's chunks)
  auto at = [](uint32_t chunk, int row_off) {  // formed per load, not held in registers
    asm volatile("" : "+v"(chunk));
    return chunk + (uint32_t)row_off;
  };
  auto load = [&](int st) {
    const int ts = t0 + kTok * st;
#pragma unroll
    for (int u = 0; u < kTok; ++u) {
      xa[u] = load16(r_a, at(ca, (ts + u) * a_row));
      xb[u] = load16(r_b, at(cb, (ts + u) * b_row));
    }
  };
  auto store = [&](int p) {
    uint8_t* buf = stage + p * kFixBuf;
#pragma unroll
    for (int q = 0; q < kMaskSlotPairs; ++q) {
      i32x4 lo, hi;
      pair_halves(xa[2 * q], xa[2 * q + 1], lo, hi);
      *(i32x4*)(buf + q * kFixPairRows + 16 * tid) = lo;
      *(i32x4*)(buf + q * kFixPairRows + kMaskSlot + 16 * tid) = hi;
      pair_halves(xb[2 * q], xb[2 * q + 1], lo, hi);
      *(i32x4*)(buf + q * kFixPairRows + kFixSide + 16 * tid) = lo;
      *(i32x4*)(buf + q * kFixPairRows + kFixSide + kMaskSlot + 16 * tid) = hi;
    }
  };
  if (n_st > 0) {
    load(0);
    store(0);
  }
  for (int st = 0; st < n_st; st += 2) {  // uniform trip count; buffers 0 and 1 in turn
    __syncthreads();  // buffer 0 written; buffer 1's readers are done
    if (st + 1 < n_st) load(st + 1);
    gather_pairs<0>(stage, rc, acc);
    if (st + 1 >= n_st) break;
    store(1);
    __syncthreads();
    if (st + 2 < n_st) load(st + 2);
    gather_pairs<1>(stage, rc, acc);
    if (st + 2 < n_st) store(0);
  }
  float* dst = partials + M.partial_base + ((int64_t)ex * M.n_chunks + it.chunk) * M.m;
  const int32_t* pos = M.pos + e0;
  uint32_t t = (uint32_t)tid;
  asm volatile("" : "+v"(t));  // the entry indices are formed here, not held through the loop
#pragma unroll
  for (int j = 0; j < kFixPer; ++j) dst[pos[t + (uint32_t)kFixThreads * j]] = acc[j];
}

hipError_t launch_mask_fixed(const MaskItem* items, int n_items, const MaskTask* tasks, float* partials,
                             hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute((const void*)mask_fixed_kernel,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaskSlotLds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(mask_fixed_kernel, dim3((unsigned)n_items), dim3(kFixThreads), kMaskSlotLds, s, items, tasks,
                     partials);
  return hipGetLastError();
}

template <int ELT, bool AL, bool FULL, bool B16>
static hipError_t launch_mask_t(const MaskItem* items, int n_items, const MaskTask* tasks, size_t lds_bytes,
                                float* partials, hipStream_t s) {
  if (lds_bytes > 64 * 1024) {  // dynamic LDS beyond 64 KiB must be allowed per kernel
    const hipError_t e = hipFuncSetAttribute((const void*)mask_kernel<ELT, AL, FULL, B16>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((mask_kernel<ELT, AL, FULL, B16>), dim3((unsigned)n_items), dim3(256), lds_bytes, s, items,
                     tasks, partials);
  return hipGetLastError();
}

hipError_t launch_mask(int elt, int aligned, int full, int b16, const MaskItem* items, int n_items,
                       const MaskTask* tasks, size_t lds_bytes, float* partials, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
#define DATTRI_MASK_CASE(E, A, F, B) \
  if (elt == E && (bool)aligned == A && (bool)full == F && (bool)b16 == B) \
    return launch_mask_t<E, A, F, B>(items, n_items, tasks, lds_bytes, partials, s);
  DATTRI_MASK_CASE(2, true, true, true)
  DATTRI_MASK_CASE(2, true, false, true)
  DATTRI_MASK_CASE(2, false, true, true)
  DATTRI_MASK_CASE(2, false, false, true)
  DATTRI_MASK_CASE(2, true, true, false)
  DATTRI_MASK_CASE(2, true, false, false)
  DATTRI_MASK_CASE(2, false, true, false)
  DATTRI_MASK_CASE(2, false, false, false)
  DATTRI_MASK_CASE(4, true, true, false)
  DATTRI_MASK_CASE(4, true, false, false)
  DATTRI_MASK_CASE(4, false, true, false)
  DATTRI_MASK_CASE(4, false, false, false)
#undef DATTRI_MASK_CASE
  return hipErrorInvalidValue;
}

}  // namespace dattri
