// bf16 scoring GEMM for large problems: S = Q X^T, Q [n_q, F], X [n_train, F]
// (both K-contiguous, rows ldq / ldx elements apart), float32 accumulate and
// output.
//
// Workgroup tile 256 x 256, 8 waves (two per SIMD) in a 2 x 4 grid of
// 128 x 64 each (4 x 2 MFMA 32x32x16 tiles = 128 float32 accumulators per
// lane).  32x32x16 keeps the matrix pipe full from one wave, which 16x16x32
// does not; the second wave per SIMD covers the other's waits.  K advances 64
// elements per stage.  Operands reach LDS by direct global->LDS loads
// (buffer_load ... lds, 16 bytes per lane, 8 lanes per 128-byte row segment:
// whole cache lines per request) into 32 KiB stage buffers: two for the query
// rows (L2/MALL-resident, loaded one stage ahead) and three for the training
// rows (streamed from HBM, loaded two stages ahead); 160 KiB in all.  Inside a
// stage the operand fragments of K step s+1 are read from LDS while the MFMAs
// of step s run; the last step's MFMAs are held back past the stage barrier so
// they cover the first fragment reads of the next stage.  LDS rows are 128
// bytes (64 bf16) with the 16-byte chunk index XOR-swizzled by row % 8, so
// every 8 consecutive lanes of a fragment read hit distinct banks; the swizzle
// is applied on the global side of the direct loads (each lane fetches the
// chunk that lands in its fixed LDS slot).  Tiles are ordered per XCD: the 8
// query tiles of a training tile run on one XCD, 32 tiles in flight per XCD
// share their operands through its L2.  When the tiles alone would leave CUs
// idle, K is split over a second grid dimension and the float32 partial tiles
// are summed in split order by a second kernel.
//
// What bounds it on MI355X: the operand loads (64 KiB per stage per CU); with
// loads removed the same loop runs at 86% of the bf16 MFMA peak, with the
// fragment reads alone at the same rate.
#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

constexpr int kSB = 256;         // tile rows (both operands)
constexpr int kSK = 64;          // K elements per stage
constexpr int kSRow = kSK * 2;   // bytes per LDS row per stage
constexpr int kStageBytes = kSB * kSRow;  // 32 KiB per operand per stage

#define LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

__device__ inline void stage_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ inline int swz(int row, int chunk) { return row * kSRow + ((chunk ^ (row & 7)) << 4); }

// One stage: 32 KiB of Q rows and 32 KiB of X rows, 32 wave-loads of 1 KiB
// (8 rows x 128 bytes) per operand; wave w issues loads j = 4w .. 4w+3 of both.
template <bool IS_X>
__device__ inline void issue_half(const rsrc_t r, int F, int ld, int kk, uint8_t* d, int wave, int lane) {
  const int row_in = lane >> 3, phys = lane & 7;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int j = wave * 4 + i;
    const int row = j * 8 + row_in;
    const int chunk = phys ^ (row & 7);
    const int col = kk * kSK + chunk * 8;
    const uint32_t oob = (uint32_t)-(int32_t)(col >= F);
    const uint32_t off = (((uint32_t)(row * ld + col) * 2u) & ~oob) | (kOOB & oob);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LDS_PTR(d + j * 1024), 16, off, 0, 0, 0);
  }
}

// Grid (tiles, K splits): split y runs stages [y*sps, (y+1)*sps) (stages past
// F read zeros) and writes its float32 tile to out + y*n_q*n_train.
__global__ __launch_bounds__(512, 1) void score_gemm_256_kernel(const uint8_t* __restrict__ Q,
                                                                const uint8_t* __restrict__ X,
                                                                float* __restrict__ out, int n_q,
                                                                int n_train, int F, int ldq, int ldx,
                                                                int n_qt, int n_xt, int sps) {
  __shared__ __align__(1024) uint8_t q0[kStageBytes], q1[kStageBytes];
  __shared__ __align__(1024) uint8_t x0[kStageBytes], x1[kStageBytes], x2[kStageBytes];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;

  const int nb = n_qt * n_xt, b = blockIdx.x;
  const int n_full = nb / kXcds * kXcds;
  const int L = b < n_full ? (b % kXcds) * (n_full / kXcds) + b / kXcds : b;
  const int qt = L % n_qt, xt = L / n_qt;
  const int qrow0 = qt * kSB, xrow0 = xt * kSB;
  const int rows_q = min(kSB, n_q - qrow0), rows_x = min(kSB, n_train - xrow0);
  // ranges end at the last row's F-th element (padding after it need not exist)
  const rsrc_t rq = make_rsrc(Q + (int64_t)qrow0 * ldq * 2, (uint32_t)(((int64_t)(rows_q - 1) * ldq + F) * 2));
  const rsrc_t rx = make_rsrc(X + (int64_t)xrow0 * ldx * 2, (uint32_t)(((int64_t)(rows_x - 1) * ldx + F) * 2));

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // this split's stages (past F they load zeros)
  const int nk = sps, k0 = blockIdx.y * sps;
  float* S = out + (int64_t)blockIdx.y * n_q * n_train;
  const int r32 = lane & 31, kg = lane >> 5;
  // fragments of one 16-wide K step: lane l holds row l % 32, K 8*(l/32)..+8
  auto read_frags = [&](const uint8_t* cq, const uint8_t* cx, int s, i32x4 (&af)[4], i32x4 (&bf)[2]) {
#pragma unroll
    for (int t = 0; t < 4; ++t) af[t] = *(const i32x4*)(cq + swz(wm * 128 + t * 32 + r32, 2 * s + kg));
#pragma unroll
    for (int t = 0; t < 2; ++t) bf[t] = *(const i32x4*)(cx + swz(wn * 64 + t * 32 + r32, 2 * s + kg));
  };
  auto mma = [&](const i32x4 (&af)[4], const i32x4 (&bf)[2]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, af[i]),
                                                           __builtin_bit_cast(bf16x8, bf[j]), acc[i][j], 0, 0, 0);
  };
  auto interleave_step = [&]() {
    // the 6 fragment reads of the next step over the first 6 of 8 MFMAs
#pragma unroll
    for (int i = 0; i < 6; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
  };

  issue_half<false>(rq, F, ldq, k0, q0, wave, lane);
  issue_half<true>(rx, F, ldx, k0, x0, wave, lane);
  issue_half<true>(rx, F, ldx, k0 + 1, x1, wave, lane);
  issue_half<false>(rq, F, ldq, k0 + 1, q1, wave, lane);
  issue_half<true>(rx, F, ldx, k0 + 2, x2, wave, lane);
  wait_vmcnt<12>();  // Q and X of stage 0 landed
  stage_barrier();
  i32x4 fa0[4], fb0[2], fa1[4], fb1[2];
  read_frags(q0, x0, 0, fa0, fb0);

  // stage kk lives in (cq, cx); its buffers receive Q(kk+2) and X(kk+3)
  auto stage = [&](int kk, uint8_t* cq, uint8_t* cx, const uint8_t* nq, const uint8_t* nx) {
    read_frags(cq, cx, 1, fa1, fb1);
    mma(fa0, fb0);
    interleave_step();
    read_frags(cq, cx, 2, fa0, fb0);
    mma(fa1, fb1);
    interleave_step();
    read_frags(cq, cx, 3, fa1, fb1);
    mma(fa0, fb0);
    interleave_step();
    wait_vmcnt<4>();   // Q(kk+1) and X(kk+1) landed (X(kk+2) may be in flight)
    stage_barrier();
    issue_half<false>(rq, F, ldq, k0 + kk + 2, cq, wave, lane);
    issue_half<true>(rx, F, ldx, k0 + kk + 3, cx, wave, lane);
    read_frags(nq, nx, 0, fa0, fb0);
    mma(fa1, fb1);
#pragma unroll
    for (int i = 0; i < 6; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM (direct loads)
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
    }
    __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);  // VMEM (direct loads)
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
  };
  // buffers rotate with period 6 (Q over 2, X over 3); the last nk % 6
  // stages repeat the first steps of the rotation
  int kk = 0;
  for (; kk + 6 <= nk; kk += 6) {
    stage(kk, q0, x0, q1, x1);
    stage(kk + 1, q1, x1, q0, x2);
    stage(kk + 2, q0, x2, q1, x0);
    stage(kk + 3, q1, x0, q0, x1);
    stage(kk + 4, q0, x1, q1, x2);
    stage(kk + 5, q1, x2, q0, x0);
  }
  const int rem = nk - kk;  // uniform
  if (rem > 0) stage(kk, q0, x0, q1, x1);
  if (rem > 1) stage(kk + 1, q1, x1, q0, x2);
  if (rem > 2) stage(kk + 2, q0, x2, q1, x0);
  if (rem > 3) stage(kk + 3, q1, x0, q0, x1);
  if (rem > 4) stage(kk + 4, q0, x1, q1, x2);
  wait_vmcnt<0>();  // the prefetches issued past the last stage

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

// Sum of the K-split partial tiles, in split order (deterministic).
__global__ __launch_bounds__(256) void splitk_sum_kernel(const float* __restrict__ part, int ks,
                                                         int64_t n, float* __restrict__ S) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float s = part[i];
  for (int y = 1; y < ks; ++y) s += part[(int64_t)y * n + i];
  S[i] = s;
}

int score_ksplit(int elt, int64_t n_q, int64_t n_train, int64_t F) {
  if (elt != 2 || n_q * n_train < kBigGemmMin || n_q <= 0 || n_train <= 0 || F <= 0) return 1;
  const int64_t tiles = ((n_q + kSB - 1) / kSB) * ((n_train + kSB - 1) / kSB);
  const int64_t nk = (F + kSK - 1) / kSK;
  int64_t ks = std::min<int64_t>({256 / std::max<int64_t>(tiles, 1), 16, nk / 2});
  if (ks <= 1) return 1;
  const int64_t sps = (nk + ks - 1) / ks;
  return (int)((nk + sps - 1) / sps);
}

hipError_t launch_score_gemm_256(const void* Q, int64_t ldq, const void* X, int64_t ldx, float* S,
                                 int64_t n_q, int64_t n_train, int64_t F, float* partials,
                                 hipStream_t s) {
  if (n_q <= 0 || n_train <= 0) return hipSuccess;
  const int n_qt = (int)((n_q + kSB - 1) / kSB), n_xt = (int)((n_train + kSB - 1) / kSB);
  const int64_t nb = (int64_t)n_qt * n_xt;
  if (nb > INT32_MAX) return hipErrorInvalidValue;
  const int64_t nk = (F + kSK - 1) / kSK;
  const int ks = score_ksplit(2, n_q, n_train, F);
  const int sps = ks > 1 ? (int)((nk + ks - 1) / ks) : (int)nk;
  if (ks > 1 && !partials) return hipErrorInvalidValue;
  hipLaunchKernelGGL(score_gemm_256_kernel, dim3((unsigned)nb, (unsigned)ks), dim3(512), 0, s,
                     (const uint8_t*)Q, (const uint8_t*)X, ks > 1 ? partials : S, (int)n_q,
                     (int)n_train, (int)F, (int)ldq, (int)ldx, n_qt, n_xt, sps);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || ks == 1) return e;
  const int64_t n = n_q * n_train;
  hipLaunchKernelGGL(splitk_sum_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, partials, ks,
                     n, S);
  return hipGetLastError();
}

}  // namespace dattri
