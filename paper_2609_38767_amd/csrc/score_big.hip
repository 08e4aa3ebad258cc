// bf16 scoring GEMM for large problems: S = (Q diag(d)) X^T, Q [n_q, F] rows
// ldq elements apart, X [n_train, F] rows ldx apart, float32 accumulate and
// output.
//
// Query preparation: pack_queries_kernel scales Q by d (when given) in float32,
// rounds once to bf16 and writes it in MFMA A-fragment order: block (rb, ks)
// of 1 KiB holds rows 32 rb .. 32 rb + 31 and features 16 ks .. 16 ks + 15,
// lane l owning row 32 rb + l % 32, features 16 ks + 8 (l / 32) .. + 7 (the
// operand layout of v_mfma_f32_32x32x16_bf16); rows past n_q and features past
// F are zero.  Each wave then loads its query fragments straight into
// registers with one coalesced 1 KiB load per fragment.
//
// GEMM: workgroup tile 256 x 256, 4 waves (one per SIMD) in a 2 x 2 grid of
// 128 x 128 (4 x 4 MFMA 32x32x16 tiles = 256 float32 accumulators per lane,
// held in AGPRs).  Only the training rows pass through LDS: direct
// global->LDS loads (16 bytes per lane, 8 lanes per 128-byte row segment) fill
// three 32 KiB stage buffers of K = 64, two stages ahead, spread over the four
// K steps of a stage; rows are XOR-swizzled by 16-byte chunk so fragment reads
// are conflict-free.  Query fragments run five K steps ahead in a six-slot
// register ring.  The last K step's MFMAs are held back past the stage barrier
// to cover the next stage's first fragment reads.  Workgroups are ordered per
// XCD (all 8 query tiles of a training tile on one XCD, 32 tiles in flight per
// XCD share operands through its L2).  When the tiles alone would leave CUs
// idle, K is split over a second grid dimension and the float32 partial tiles
// are summed in split order by a second kernel.
//
// What bounds it on MI355X: per shader cycle the matrix cores are about 80%
// busy (91% with the operand loads removed), but under this load the chip
// throttles its clock to about 1.7 GHz (2.0 GHz for MFMA work alone), against
// the 2.4 GHz the dense bf16 peak assumes.  Keeping the query operand out of
// LDS halves LDS traffic (fragment reads plus DMA writes, 96 KiB per stage
// instead of 192 KiB) compared with staging both operands there.
#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

constexpr int kSB = 256;         // tile rows (both operands)
constexpr int kSK = 64;          // K elements per stage
constexpr int kSRow = kSK * 2;   // bytes per LDS row per stage
constexpr int kStageBytes = kSB * kSRow;  // 32 KiB per stage buffer

#define LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

__device__ inline void stage_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ inline int swz(int row, int chunk) { return row * kSRow + ((chunk ^ (row & 7)) << 4); }

// K steps of 16 features per packed query row block (a whole number of stages)
inline int64_t qpack_ksteps(int64_t F) { return (F + kSK - 1) / kSK * 4; }

int64_t score_qpack_bytes(int64_t n_q, int64_t F) {
  const int64_t n_rb = (n_q + kSB - 1) / kSB * (kSB / 32);
  return n_rb * qpack_ksteps(F) * 1024;
}

__global__ __launch_bounds__(256) void pack_queries_kernel(const uint16_t* __restrict__ Q, int64_t ldq,
                                                           const float* __restrict__ d, int n_q, int F,
                                                           int nks, int64_t n_lanes,
                                                           uint8_t* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_lanes;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int lane = (int)(i & 63);
    const int64_t blk = i >> 6;
    const int rb = (int)(blk / nks), ks = (int)(blk % nks);
    const int row = rb * 32 + (lane & 31), k = ks * 16 + 8 * (lane >> 5);
    uint32_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint32_t v = 0;
      if (row < n_q && k + e < F) {
        v = Q[(int64_t)row * ldq + k + e];
        if (d) v = f32_to_bf16_bits(bf16_bits_to_f32(v) * d[k + e]);
      }
      h[e] = v;
    }
    const i32x4 w = {(int)(h[0] | (h[1] << 16)), (int)(h[2] | (h[3] << 16)), (int)(h[4] | (h[5] << 16)),
                     (int)(h[6] | (h[7] << 16))};
    *(i32x4*)(out + i * 16) = w;
  }
}

// Two of this wave's eight direct loads of one training-row stage (loads 2s,
// 2s + 1): each lane fetches the 16-byte chunk that lands in its fixed
// swizzled LDS slot; features past F read zero.
__device__ inline void xload2(const rsrc_t r, int F, int ld, int kk, uint8_t* d, int wave, int lane, int s) {
  const int row_in = lane >> 3, phys = lane & 7;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int j = wave * 8 + 2 * s + i;
    const int row = j * 8 + row_in;
    const int chunk = phys ^ (row & 7);
    const int col = kk * kSK + chunk * 8;
    const uint32_t oob = (uint32_t)-(int32_t)(col >= F);
    const uint32_t off = (((uint32_t)(row * ld + col) * 2u) & ~oob) | (kOOB & oob);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LDS_PTR(d + j * 1024), 16, off, 0, 0, 0);
  }
}

// Grid (tiles, K splits): split y runs stages [y*sps, (y+1)*sps) and writes its
// float32 tile to out + y*n_q*n_train.
__global__ __launch_bounds__(256, 1) void score_gemm_256_kernel(const uint8_t* __restrict__ Qp,
                                                                const uint8_t* __restrict__ X,
                                                                float* __restrict__ out, int n_q,
                                                                int n_train, int F, int ldx, int nks,
                                                                int n_qt, int n_xt, int sps) {
  __shared__ __align__(1024) uint8_t x0[kStageBytes], x1[kStageBytes], x2[kStageBytes];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  const int nb = n_qt * n_xt, b = blockIdx.x;
  const int n_full = nb / kXcds * kXcds;
  const int L = b < n_full ? (b % kXcds) * (n_full / kXcds) + b / kXcds : b;
  const int qt = L % n_qt, xt = L / n_qt;
  const int qrow0 = qt * kSB, xrow0 = xt * kSB;
  const int rows_x = min(kSB, n_train - xrow0);
  // this wave's 4 packed query row blocks; the training rows' range ends at
  // the last row's F-th element (padding after it need not exist)
  const rsrc_t rq = make_rsrc(Qp + (int64_t)(qt * 8 + wm * 4) * nks * 1024, (uint32_t)(4 * nks * 1024));
  const rsrc_t rx = make_rsrc(X + (int64_t)xrow0 * ldx * 2, (uint32_t)(((int64_t)(rows_x - 1) * ldx + F) * 2));

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int nk = sps, k0 = blockIdx.y * sps;
  float* S = out + (int64_t)blockIdx.y * n_q * n_train;
  const int r32 = lane & 31, kg = lane >> 5;
  i32x4 ar[6][4];  // query fragments of six K steps (loaded five steps ahead)
  auto aload = [&](int g, i32x4 (&dst)[4]) {  // K step g of this split
    const int ks = k0 * 4 + g;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint32_t off = ks < nks ? (uint32_t)((t * nks + ks) * 1024 + lane * 16) : kOOB;
      dst[t] = load16(rq, off);
    }
  };
  // training fragments of K step s: lane l holds row l % 32, K 8*(l/32)..+8
  auto read_b = [&](const uint8_t* cx, int s, i32x4 (&bf)[4]) {
#pragma unroll
    for (int t = 0; t < 4; ++t) bf[t] = *(const i32x4*)(cx + swz(wn * 128 + t * 32 + r32, 2 * s + kg));
  };
  auto mma = [&](const i32x4 (&af)[4], const i32x4 (&bf)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, af[i]),
                                                           __builtin_bit_cast(bf16x8, bf[j]), acc[i][j], 0, 0, 0);
  };
  // one K step: 16 MFMAs with the next step's 4 fragment reads and the 6 loads
  // (4 query fragments, 2 training-row DMA) between them
  auto sched = [&]() {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                        // MFMA
      if (i < 4) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);             // DS read
      if (i >= 4 && i < 10) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM
    }
  };

  // prologue: training rows of stages 0 and 1, query steps 0..4
#pragma unroll
  for (int s = 0; s < 4; ++s) xload2(rx, F, ldx, k0, x0, wave, lane, s);
#pragma unroll
  for (int s = 0; s < 4; ++s) xload2(rx, F, ldx, k0 + 1, x1, wave, lane, s);
  aload(0, ar[0]);
  aload(1, ar[1]);
  aload(2, ar[2]);
  aload(3, ar[3]);
  aload(4, ar[4]);
  wait_vmcnt<28>();  // stage 0's training rows landed (8 + 20 later loads may be in flight)
  stage_barrier();
  i32x4 b0[4], b1[4];
  read_b(x0, 0, b0);

  // stage kk: training rows in cx (stage kk+1 in nx); X(kk+2) is loaded into
  // fx.  The query ring slot of K step 4kk+s is (4kk+s) % 6, static because
  // three stages are unrolled (p = kk % 3).
  auto stage = [&](int kk, int p, const uint8_t* cx, const uint8_t* nx, uint8_t* fx) {
    const int g = 4 * kk;
    read_b(cx, 1, b1);
    aload(g + 5, ar[(4 * p + 5) % 6]);
    xload2(rx, F, ldx, k0 + kk + 2, fx, wave, lane, 0);
    mma(ar[(4 * p) % 6], b0);
    sched();
    read_b(cx, 2, b0);
    aload(g + 6, ar[(4 * p + 6) % 6]);
    xload2(rx, F, ldx, k0 + kk + 2, fx, wave, lane, 1);
    mma(ar[(4 * p + 1) % 6], b1);
    sched();
    read_b(cx, 3, b1);
    aload(g + 7, ar[(4 * p + 7) % 6]);
    xload2(rx, F, ldx, k0 + kk + 2, fx, wave, lane, 2);
    mma(ar[(4 * p + 2) % 6], b0);
    sched();
    wait_vmcnt<18>();  // X(kk+1) landed: 3 steps x 6 loads were issued after its last
    stage_barrier();
    read_b(nx, 0, b0);
    aload(g + 8, ar[(4 * p + 8) % 6]);
    xload2(rx, F, ldx, k0 + kk + 2, fx, wave, lane, 3);
    mma(ar[(4 * p + 3) % 6], b1);
    sched();
  };
  int kk = 0;
  for (; kk + 3 <= nk; kk += 3) {
    stage(kk, 0, x0, x1, x2);
    stage(kk + 1, 1, x1, x2, x0);
    stage(kk + 2, 2, x2, x0, x1);
  }
  const int rem = nk - kk;  // uniform
  if (rem > 0) stage(kk, 0, x0, x1, x2);
  if (rem > 1) stage(kk + 1, 1, x1, x2, x0);
  wait_vmcnt<0>();  // the prefetches issued past the last stage

  // 32x32 C layout: lane l, element v holds row 8*(v/4) + 4*(l/32) + v%4,
  // column l % 32; for each v, 32 lanes store 128 contiguous bytes of a row.
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int x = xrow0 + wn * 128 + j * 32 + r32;
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

hipError_t launch_splitk_sum(const float* part, int ks, int64_t n, float* S, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(splitk_sum_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, part, ks, n, S);
  return hipGetLastError();
}

// 128 x 128 kernel: split K while its tiles number fewer than kSmallTarget, into
// splits of at least kSmallMinSteps K steps of 128 bytes.
constexpr int64_t kSmallTarget = 512, kSmallMinSteps = 8;

int score_ksplit(int elt, int64_t n_q, int64_t n_train, int64_t F) {
  if (F <= 0) return 1;
  if (!score_uses_big(elt, n_q, n_train)) {
    const int64_t tiles = ((n_q + 127) / 128) * ((n_train + 127) / 128);
    const int64_t nk = (F + 128 / elt - 1) / (128 / elt);
    const int64_t ks = std::min<int64_t>(kSmallTarget / std::max<int64_t>(tiles, 1), nk / kSmallMinSteps);
    if (ks <= 1) return 1;
    const int64_t sps = (nk + ks - 1) / ks;
    return (int)((nk + sps - 1) / sps);
  }
  const int64_t tiles = ((n_q + kSB - 1) / kSB) * ((n_train + kSB - 1) / kSB);
  const int64_t nk = (F + kSK - 1) / kSK;
  int64_t ks = std::min<int64_t>({256 / std::max<int64_t>(tiles, 1), 16, nk / 2});
  if (ks <= 1) return 1;
  const int64_t sps = (nk + ks - 1) / ks;
  return (int)((nk + sps - 1) / sps);
}

hipError_t launch_score_gemm_256(const void* Q, int64_t ldq, const float* d, const void* X,
                                 int64_t ldx, float* S, int64_t n_q, int64_t n_train, int64_t F,
                                 void* qpack, float* partials, hipStream_t s) {
  if (n_q <= 0 || n_train <= 0) return hipSuccess;
  if (!qpack) return hipErrorInvalidValue;
  const int n_qt = (int)((n_q + kSB - 1) / kSB), n_xt = (int)((n_train + kSB - 1) / kSB);
  const int64_t nb = (int64_t)n_qt * n_xt;
  if (nb > INT32_MAX) return hipErrorInvalidValue;
  const int64_t nks = qpack_ksteps(F);
  const int64_t n_lanes = score_qpack_bytes(n_q, F) / 16;
  const int pblocks = (int)std::min<int64_t>((n_lanes + 255) / 256, 8192);
  hipLaunchKernelGGL(pack_queries_kernel, dim3(std::max(pblocks, 1)), dim3(256), 0, s,
                     (const uint16_t*)Q, ldq, d, (int)n_q, (int)F, (int)nks, n_lanes, (uint8_t*)qpack);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t nk = (F + kSK - 1) / kSK;
  const int ks = score_ksplit(2, n_q, n_train, F);
  const int sps = ks > 1 ? (int)((nk + ks - 1) / ks) : (int)nk;
  if (ks > 1 && !partials) return hipErrorInvalidValue;
  hipLaunchKernelGGL(score_gemm_256_kernel, dim3((unsigned)nb, (unsigned)ks), dim3(256), 0, s,
                     (const uint8_t*)qpack, (const uint8_t*)X, ks > 1 ? partials : S, (int)n_q,
                     (int)n_train, (int)F, (int)ldx, (int)nks, n_qt, n_xt, sps);
  e = hipGetLastError();
  if (e != hipSuccess || ks == 1) return e;
  return launch_splitk_sum(partials, ks, n_q * n_train, S, s);
}

}  // namespace dattri
