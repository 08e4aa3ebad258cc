// bf16 scoring GEMM for large problems: S = Q X^T, Q [n_q, F], X [n_train, F]
// (both K-contiguous), float32 accumulate and output.
//
// Workgroup tile 256 x 256, 8 waves (two per SIMD) in a 2 x 4 grid of
// 128 x 64 each (4 x 2 MFMA 32x32x16 tiles = 128 float32 accumulators per
// lane).  32x32x16 is used because on gfx950 it keeps the matrix pipe full
// from one wave, which 16x16x32 does not; the second wave per SIMD covers the
// other's waits on LDS, loads and barriers.  K advances
// 32 elements per stage through a 4-stage LDS ring filled by direct
// global->LDS loads (buffer_load ... lds, 16 bytes per lane): no staging
// registers, three stages in flight while one is multiplied, and operand
// fragments double-buffered in registers across stage boundaries.  Each stage
// buffer is its own __shared__ object so the compiler tracks the loads into it
// separately; each wave waits for its own loads of a stage (vmcnt) and a
// barrier then publishes the stage to the workgroup.  LDS rows are
// 64 bytes (32 bf16) with the 16-byte chunk index XOR-swizzled by (row/2)%4,
// so the 16-byte fragment reads of a wave hit distinct banks; the swizzle is
// applied on the global side (each lane picks the chunk that lands in its
// fixed LDS slot).  Tiles are ordered per XCD as in the 128 x 128 kernel.
#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

constexpr int kSB = 256;         // tile rows (both operands)
constexpr int kSK = 32;          // K elements per stage
constexpr int kSRow = kSK * 2;   // bytes per LDS row per stage
constexpr int kStageBytes = kSB * kSRow;  // 16 KiB per operand per stage

#define LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // gfx9 s_waitcnt: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] << 14
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Barrier publishing LDS stages written by direct loads.  A memory fence here
// would make the compiler wait for every outstanding direct load (they are
// LDS writes), including the later stages still meant to be in flight; each
// wave instead waits for its own loads of the stage with wait_vmcnt<> first.
// The "memory" clobber keeps the compiler from moving LDS accesses across it.
__device__ inline void stage_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ inline int swz(int row, int chunk) { return row * kSRow + ((chunk ^ ((row >> 1) & 3)) << 4); }

// One stage: 16 KiB of Q rows and 16 KiB of X rows, 16 wave-loads of 1 KiB
// each per operand; wave w issues loads j = 2w, 2w+1 of both.
__device__ inline void issue_stage(const rsrc_t rq, const rsrc_t rx, int F, int kk, uint8_t* dq,
                                   uint8_t* dx, int wave, int lane) {
  const int row_in = lane >> 2, phys = lane & 3;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int j = wave * 2 + i;
    const int row = j * 16 + row_in;
    const int chunk = phys ^ ((row >> 1) & 3);
    const int col = kk * kSK + chunk * 8;
    // out-of-range columns get an offset beyond the descriptor (reads zero);
    // computed with a mask, not a branch, so every lane issues the same loads
    const uint32_t oob = (uint32_t)-(int32_t)(col >= F);
    const uint32_t off = ((uint32_t)((row * F + col) * 2) & ~oob) | (kOOB & oob);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rq, LDS_PTR(dq + j * 1024), 16, off, 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, LDS_PTR(dx + j * 1024), 16, off, 0, 0, 0);
  }
}

__global__ __launch_bounds__(512, 1) void score_gemm_256_kernel(const uint8_t* __restrict__ Q,
                                                                const uint8_t* __restrict__ X,
                                                                float* __restrict__ S, int n_q,
                                                                int n_train, int F, int n_qt,
                                                                int n_xt) {
  __shared__ __align__(1024) uint8_t q0[kStageBytes], q1[kStageBytes], q2[kStageBytes], q3[kStageBytes];
  __shared__ __align__(1024) uint8_t x0[kStageBytes], x1[kStageBytes], x2[kStageBytes], x3[kStageBytes];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;

  const int nb = n_qt * n_xt, b = blockIdx.x;
  const int n_full = nb / kXcds * kXcds;
  const int L = b < n_full ? (b % kXcds) * (n_full / kXcds) + b / kXcds : b;
  const int qt = L % n_qt, xt = L / n_qt;
  const int qrow0 = qt * kSB, xrow0 = xt * kSB;
  const int rows_q = min(kSB, n_q - qrow0), rows_x = min(kSB, n_train - xrow0);
  const rsrc_t rq = make_rsrc(Q + (int64_t)qrow0 * F * 2, (uint32_t)((int64_t)rows_q * F * 2));
  const rsrc_t rx = make_rsrc(X + (int64_t)xrow0 * F * 2, (uint32_t)((int64_t)rows_x * F * 2));

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // Stages are padded to a multiple of 4 so the loop is branch-free (stages
  // past F load zeros: their offsets are out of range); every stage issues the
  // same 4 direct loads per wave.  Four stages are in flight: at the start of
  // stage kk the wave waits for stage kk+1, crosses the barrier, and refills
  // the buffer stage kk came from with stage kk+4.  Fragments are
  // double-buffered in registers: the 12 fragment reads of stage kk+1 and the
  // 4 direct loads are interleaved with the 16 MFMAs of stage kk, so LDS and
  // load latency hide under matrix work.
  const int nk = ((F + kSK - 1) / kSK + 3) & ~3;
  issue_stage(rq, rx, F, 0, q0, x0, wave, lane);
  issue_stage(rq, rx, F, 1, q1, x1, wave, lane);
  issue_stage(rq, rx, F, 2, q2, x2, wave, lane);
  issue_stage(rq, rx, F, 3, q3, x3, wave, lane);

  // 32x32x16 operand fragments: lane l holds row (l % 32), K elements
  // 8*(l/32) .. +8 of a 16-wide K step; a 32-wide stage has two K steps (kh).
  i32x4 fa0[8], fb0[4], fa1[8], fb1[4];  // [tile * 2 + kh]
  const int r32 = lane & 31, kg = lane >> 5;
  auto read_frags = [&](const uint8_t* cq, const uint8_t* cx, i32x4 (&af)[8], i32x4 (&bf)[4]) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) af[t * 2 + kh] = *(const i32x4*)(cq + swz(wm * 128 + t * 32 + r32, kh * 2 + kg));
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) bf[t * 2 + kh] = *(const i32x4*)(cx + swz(wn * 64 + t * 32 + r32, kh * 2 + kg));
  };
  // K half outermost: 16 independent accumulators between the two MFMAs that
  // update the same tile, so no MFMA waits on its predecessor's result.
  auto mma_all = [&](const i32x4 (&af)[8], const i32x4 (&bf)[4]) {
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, af[i * 2 + kh]),
                                                             __builtin_bit_cast(bf16x8, bf[j * 2 + kh]),
                                                             acc[i][j], 0, 0, 0);
  };
  wait_vmcnt<12>();  // stage 0 landed (stages 1..3 may be in flight)
  stage_barrier();
  read_frags(q0, x0, fa0, fb0);

  // stage kk: fragments (ca, cb) in registers; stage kk+1 is in (nq, nx) and
  // is read into (na, nb_); (dq, dx) held stage kk and receives stage kk+4.
  auto stage = [&](int kk, const i32x4 (&ca)[8], const i32x4 (&cb)[4], i32x4 (&na)[8],
                   i32x4 (&nb_)[4], const uint8_t* nq, const uint8_t* nx, uint8_t* dq, uint8_t* dx) {
    wait_vmcnt<8>();  // this wave's loads of stage kk+1 have landed
    stage_barrier();   // ... and every other wave's; stage kk's buffer is free
    issue_stage(rq, rx, F, kk + 4, dq, dx, wave, lane);
    read_frags(nq, nx, na, nb_);
    mma_all(ca, cb);
    // interleave: 8 x {1 direct load, 2 MFMA, 1 fragment read, 2 MFMA, 1 read}
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read (direct load)
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
    }
  };
  for (int kk = 0; kk < nk; kk += 4) {
    stage(kk + 0, fa0, fb0, fa1, fb1, q1, x1, q0, x0);
    stage(kk + 1, fa1, fb1, fa0, fb0, q2, x2, q1, x1);
    stage(kk + 2, fa0, fb0, fa1, fb1, q3, x3, q2, x2);
    stage(kk + 3, fa1, fb1, fa0, fb0, q0, x0, q3, x3);
  }
  wait_vmcnt<0>();  // the padding loads issued past the end

  // 32x32 C layout: lane l, element v holds row 8*(v/4) + 4*(l/32) + v%4,
  // column l % 32; for each v, 32 lanes store 128 contiguous bytes of a row.
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int x = xrow0 + wn * 64 + j * 32 + r32;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int q = qrow0 + wm * 128 + i * 32 + 8 * (v >> 2) + 4 * kg + (v & 3);
        if (q < n_q && x < n_train) __builtin_nontemporal_store(acc[i][j][v], &S[(int64_t)q * n_train + x]);
      }
    }
}

hipError_t launch_score_gemm_256(const void* Q, const void* X, float* S, int64_t n_q,
                                 int64_t n_train, int64_t F, hipStream_t s) {
  if (n_q <= 0 || n_train <= 0) return hipSuccess;
  const int n_qt = (int)((n_q + kSB - 1) / kSB), n_xt = (int)((n_train + kSB - 1) / kSB);
  const int64_t nb = (int64_t)n_qt * n_xt;
  if (nb > INT32_MAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(score_gemm_256_kernel, dim3((unsigned)nb), dim3(512), 0, s, (const uint8_t*)Q,
                     (const uint8_t*)X, S, (int)n_q, (int)n_train, (int)F, n_qt, n_xt);
  return hipGetLastError();
}

}  // namespace dattri
