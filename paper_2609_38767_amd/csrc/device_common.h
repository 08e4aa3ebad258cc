// Device helpers for gfx950: MFMA wrappers, buffer-resource loads with
// hardware bounds checks, and bf16 conversion.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dattri {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

// Raw buffer descriptor over [base, base + bytes).  Loads at byte offsets
// >= bytes return zero (CDNA buffer range checking), which masks ragged
// token rows and feature tails without branches.
// Every caller passes a wave-uniform base and size; readfirstlane makes that
// visible to the compiler so the descriptor lives in SGPRs (no per-lane
// "waterfall" loop around each buffer load).
__device__ inline rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t p = (uint64_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)p);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
  const uint32_t n = __builtin_amdgcn_readfirstlane(bytes);
  return __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), (short)0, (int)n,
                                           0x00020000);
}
constexpr uint32_t kOOB = 0xFFFFFFF0u;  // an offset no descriptor here covers

// LDS destination of a direct load (buffer_load ... lds): lane l's 16 bytes
// land at p + 16 l.
#define DATTRI_LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

// Wait until at most N vector-memory operations of this wave are in flight
// (direct loads count until their data is in LDS); other counters untouched.
template <int N>
__device__ inline void wait_vmcnt_dma() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

__device__ inline i32x4 load16(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
typedef int i32x2 __attribute__((ext_vector_type(2)));
__device__ inline i32x2 load8(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(i32x2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}
__device__ inline uint32_t load4(rsrc_t r, uint32_t off) {
  return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
__device__ inline uint32_t load2(rsrc_t r, uint32_t off) {
  return (uint32_t)(uint16_t)__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}

// One 16-byte operand fragment: EPL = 16 / ELT consecutive elements of row
// `row` starting at column `col` of a row-major [nrows, d] block.  Rows
// >= nrows and columns >= d read as zero (their offsets are sent out of the
// descriptor's range, so 32-bit offsets never wrap into valid rows).
// `aligned` means d*ELT and the base are multiples of 16, so a fragment is
// either wholly inside or wholly outside the row.
template <int ELT>
__device__ inline i32x4 load_frag(rsrc_t r, int row, int nrows, int col, int d, bool aligned) {
  constexpr int EPL = 16 / ELT;
  const int64_t row_off = (int64_t)row * d;
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
    v[0] = (int)(w[0] | (w[1] << 16));
    v[1] = (int)(w[2] | (w[3] << 16));
    v[2] = (int)(w[4] | (w[5] << 16));
    v[3] = (int)(w[6] | (w[7] << 16));
  } else {
    v[0] = (int)w[0]; v[1] = (int)w[1]; v[2] = (int)w[2]; v[3] = (int)w[3];
  }
  return v;
}

// One 16-byte fragment of row `row` at column `col` of a block whose rows
// are `ld` elements apart and hold d valid elements; d*ELT, ld*ELT and the
// base are multiples of 16.  Rows >= nrows and columns >= d read as zero.
template <int ELT>
__device__ inline i32x4 load_frag_ld(rsrc_t r, int row, int nrows, int col, int d, int ld) {
  const uint32_t off = (row < nrows && col < d) ? (uint32_t)(((int64_t)row * ld + col) * ELT) : kOOB;
  return load16(r, off);
}

__device__ inline f32x4 mfma_f32_4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// acc[16x16] += A_frag (16 rows x K) * B_frag (K x 16 cols), where each lane's
// 16-byte fragment holds its K-slice: one 16x16x32 bf16 MFMA, or four
// 16x16x4 f32 MFMAs (element j of every lane forms the j-th K=4 step).  The
// same K-slot order is used for both operands, so the sum covers all K.
template <int ELT>
__device__ inline f32x4 frag_mma(i32x4 a, i32x4 b, f32x4 c);

template <>
__device__ inline f32x4 frag_mma<2>(i32x4 a, i32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// The whole 16-byte fragment is reinterpreted as four floats first: taking
// __builtin_bit_cast(float, v[j]) of single vector elements inside an unrolled
// loop was compiled to read element 0 for every j.
template <>
__device__ inline f32x4 frag_mma<4>(i32x4 a, i32x4 b, f32x4 c) {
  const f32x4 fa = __builtin_bit_cast(f32x4, a);
  const f32x4 fb = __builtin_bit_cast(f32x4, b);
  c = mfma_f32_4(fa[0], fb[0], c);
  c = mfma_f32_4(fa[1], fb[1], c);
  c = mfma_f32_4(fa[2], fb[2], c);
  c = mfma_f32_4(fa[3], fb[3], c);
  return c;
}

// Workgroup barrier that orders LDS accesses only.  __syncthreads() also
// fences global memory, which makes the compiler wait for every outstanding
// global load (vmcnt(0)) and would drain register prefetch pipelines.
__device__ inline void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ inline float bf16_bits_to_f32(uint32_t h) { return __builtin_bit_cast(float, h << 16); }

__device__ inline uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Element (v, c) of a fragment-major packed projection map (see internal.h),
// converted to float; rows >= d or columns >= k read as zero.
template <int ELT>
__device__ inline float packed_elem(const uint8_t* P, int v, int c, int d, int k) {
  if (v >= d || c >= k) return 0.f;
  constexpr int EPL = 16 / ELT, KR = 4 * EPL;
  const int nt_all = (k + 15) >> 4;
  const int kb = v / KR, w = v % KR, g = w / EPL, j = w % EPL;
  const int64_t off = (((int64_t)kb * nt_all + (c >> 4)) * 64 + 16 * g + (c & 15)) * 16 + j * ELT;
  if (ELT == 2) return bf16_bits_to_f32(*(const uint16_t*)(P + off));
  return *(const float*)(P + off);
}

}  // namespace dev
}  // namespace dattri
