// Random coordinate masks of the weight gradient, gathered from the factors
// (App. A.2 "Random maps": entry (r, c) of DW is sum_t g_{t,r} a_{t,c}, Eq. 1,
// so the kept entries need |M| products per token position and DW is never
// formed).
//
// One workgroup per (mask layer, example, token chunk, group of up to
// kMaskGroup = 16384 entries).  Each stage holds `stage_tokens` consecutive
// token rows of A and of B: consecutive rows of an example are one contiguous
// block in HBM, so for 16-byte rows the stage is moved by direct global-to-LDS
// loads (1 KiB per wave instruction, no registers) into one of two buffers
// while the other is gathered; rows that are not 16-byte multiples take a
// plain copy into one buffer.  Every thread owns 64 entries (each (r, c) pair
// packed in one register) and adds b[r_e] * a[c_e] for each staged token, in
// token order (deterministic); the products of bf16 values are exact in
// float32 (bf16 layers up to 32768 wide take them through v_dot2_f32_bf16,
// gather_rows_b16).  Every group restages the chunk's token rows, so groups are made
// as large as two waves per SIMD allow: ten masks of 8192 entries take 5
// groups instead of 10.  The entries come in the slot order of the layer's
// table, arranged at bind time so that the 32 lanes of a half-wave mostly
// read distinct LDS banks, and each sum is written at the entry's position in
// mask order.  Whole groups and the partial last group of a layer run in
// separate launches (the partial one bounds its slots).
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

// Direct global-to-LDS copy of `bytes` (a whole stage part, 16-byte aligned)
// from byte offset `off` of descriptor r into dst: one 1 KiB chunk per wave
// instruction, lane l moving bytes 16 l .. 16 l + 15 of its chunk; chunks are
// dealt to the 4 waves in turn.  Bytes past the descriptor's range land as
// zero.  dst must have room for the size rounded up to 1 KiB.
__device__ inline void dma_block(const rsrc_t r, uint32_t off, int bytes, uint8_t* dst, int wave, int lane) {
  const int chunks = (bytes + 1023) >> 10;
  for (int c = wave; c < chunks; c += 4)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LDS_PTR(dst + c * 1024), 16, off + c * 1024 + lane * 16, 0, 0, 0);
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
  uint32_t rc[kMaskPerThread];
  float acc[kMaskPerThread];
#pragma unroll
  for (int j = 0; j < kMaskPerThread; ++j) {
    const int e = tid + 256 * j;
    rc[j] = e < ne ? ((uint32_t)M.rows[e0 + e] << (16 + sh)) | ((uint32_t)M.cols[e0 + e] << sh) : 0u;
    acc[j] = 0.f;
  }
  const int TS = M.stage_tokens;
  const int a_row = M.d_in * ELT, b_row = M.d_out * ELT;
  const uint8_t* ga = (const uint8_t*)M.A + ((int64_t)ex * M.T) * a_row;
  const uint8_t* gb = (const uint8_t*)M.B + ((int64_t)ex * M.T) * b_row;

  auto gather = [&](const uint8_t* sa, const uint8_t* sb, int nt) {
    if constexpr (B16)
      gather_rows_b16<FULL>(sa, sb, nt, a_row, b_row, nj, rc, acc);
    else
      gather_rows<ELT, FULL>(sa, sb, nt, a_row, b_row, nj, rc, acc);
  };

  if (AL) {
    // two stage buffers, each [A rows | B rows], parts rounded up to 1 KiB
    const int a_part = (TS * a_row + 1023) & ~1023, b_part = (TS * b_row + 1023) & ~1023;
    const int buf = a_part + b_part;
    // descriptors end at row t1: rows past the chunk land as zero
    const rsrc_t r_a = make_rsrc(ga, (uint32_t)((int64_t)t1 * a_row));
    const rsrc_t r_b = make_rsrc(gb, (uint32_t)((int64_t)t1 * b_row));
    const int n_st = t1 > t0 ? (t1 - t0 + TS - 1) / TS : 0;
    auto issue = [&](int st) {
      const int ts = t0 + st * TS, nt = min(TS, t1 - ts);
      uint8_t* sa = stage + (st & 1) * buf;
      dma_block(r_a, (uint32_t)(ts * a_row), nt * a_row, sa, wave, lane);
      dma_block(r_b, (uint32_t)(ts * b_row), nt * b_row, sa + a_part, wave, lane);
    };
    if (n_st > 0) issue(0);
    for (int st = 0; st < n_st; ++st) {  // uniform trip count
      wait_vm0();        // this wave's loads of stage st have landed
      __syncthreads();   // every wave's have; the other buffer's readers are done
      if (st + 1 < n_st) issue(st + 1);
      const uint8_t* sa = stage + (st & 1) * buf;
      gather(sa, sa + a_part, min(TS, t1 - (t0 + st * TS)));
    }
  } else {
    uint8_t* sa = stage;
    uint8_t* sb = stage + (((int64_t)TS * a_row + 15) & ~(int64_t)15);
    for (int ts = t0; ts < t1; ts += TS) {  // uniform trip count
      const int nt = min(TS, t1 - ts);
      __syncthreads();  // the previous stage's readers are done
      copy_rows<ELT, false>(sa, ga + (int64_t)ts * a_row, (int64_t)nt * a_row);
      copy_rows<ELT, false>(sb, gb + (int64_t)ts * b_row, (int64_t)nt * b_row);
      __syncthreads();
      gather(sa, sb, nt);
    }
  }
  float* dst = partials + M.partial_base + ((int64_t)ex * M.n_chunks + it.chunk) * M.m;
#pragma unroll
  for (int j = 0; j < kMaskPerThread; ++j)
    if (tid + 256 * j < ne) dst[M.pos[e0 + tid + 256 * j]] = acc[j];
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
