// Kronecker-factored curvature on projected factors (K-FAC, EK-FAC):
// factor sums, their eigendecomposition, EK-FAC's eigenvalue correction and
// the preconditioning of query blocks.
//
// fsum_kernel        sum over token rows of x~ x~^T with x~ = P^T x, for one
//                    side of a layer (x = a_t with P_in, or g_t with P_out).
//                    Token rows are projected exactly as in the factored route
//                    (bf16/f32 MFMA; bf16 aligned rows streamed through LDS by
//                    direct loads, project_rows_dma, else fragments loaded into
//                    registers with map panels in LDS, project_rows); the
//                    projected tiles stay in accumulators and their outer products are summed
//                    with float32 MFMA (16x16x4), whose C layout gives every
//                    element index a K = 4 slice of token rows for both
//                    operands.  Only tiles on and above the diagonal are
//                    accumulated; the partial block is written mirrored.
// stat_reduce_kernel fixed-order sum of partial blocks into the state.
// eigen_kernel       cyclic Jacobi in float64, one workgroup per matrix: each
//                    round applies n/2 rotations on disjoint index pairs (the
//                    round-robin ordering), rows then columns of the LDS copy,
//                    and accumulates the rotations into V.
// ekfac_kernel       sum over training rows of (Q_A^T Psi Q_G)^2 (float32 MFMA,
//                    one wave per row).
// precond_kernel     Q_A [(Q_A^T Psi Q_G) / (E + delta)] Q_G^T per query block.
// token_kernel       per-token contributions a~_t^T R g~_t over the kept rows
//                    (float32 MFMA, 32 token positions per wave).
#include <math.h>

#include "device_common.h"
#include "internal.h"
#include "project_rows.h"

namespace dattri {
using namespace dev;

// ------------------------------------------------------------ factor sums
constexpr int fsum_rt(int nt) { return nt <= 2 ? 4 : 2; }
// bf16 sides with aligned rows and 2 or 4 map tiles stream their factor rows
// through LDS by direct loads (project_rows_dma), as the factored route does
constexpr bool fsum_dma(int elt, bool aligned, int nt) { return elt == 2 && aligned && (nt == 2 || nt == 4); }

template <int ELT, bool AL, int NT>
__global__ __launch_bounds__(256, 2) void fsum_kernel(const FsumItem* __restrict__ items,
                                                      const FsumOp* __restrict__ ops,
                                                      float* __restrict__ partials) {
  constexpr int RT = fsum_rt(NT);
  constexpr int PD = AL ? (RT >= 4 ? 2 : 4) : 2;
  constexpr bool kDma = fsum_dma(ELT, AL, NT);
  constexpr int kPanBytes = 2 * kPanel * NT * kFragBytes;
  constexpr int kSmem = kDma ? DmaLds<RT, kDma ? NT : 2>::kBytes : kPanBytes;
  static_assert(kSmem <= 80 * 1024, "two workgroups per CU");
  __shared__ __align__(1024) uint8_t smem[kSmem];
  auto pan = reinterpret_cast<uint8_t(*)[kPanel][NT][kFragBytes]>(smem);
  const FsumItem it = items[blockIdx.x];
  if (it.n_units <= 0) return;  // padding item of the XCD-interleaved order
  const FsumOp& O = ops[it.op];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, m16 = lane & 15;
  const int nt = O.nt, d = O.d, T = O.T;

  FragSrc<NT> P;
  P.nt = nt;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    P.base[t] = (const uint8_t*)O.P + (int64_t)(t < nt ? t : 0) * kFragBytes;
    P.stride[t] = (int64_t)nt * kFragBytes;
  }
  f32x4 cov[NT][NT];
#pragma unroll
  for (int a = 0; a < NT; ++a)
#pragma unroll
    for (int b = 0; b < NT; ++b) cov[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int u = it.unit0; u < it.unit0 + it.n_units; ++u) {
    const int ex = u / O.n_chunks, ch = u - ex * O.n_chunks;
    int t_eff = T;
    if (O.lengths) t_eff = min(max(O.lengths[ex], 0), T);
    const int row_begin = ch * O.chunk_rows;
    const int row_end = min(row_begin + O.chunk_rows, t_eff);
    const int rows_valid = max(row_end, 0);
    const uint8_t* base = (const uint8_t*)O.X + (size_t)ex * T * d * ELT;
    const rsrc_t r = make_rsrc(base, (uint32_t)((int64_t)rows_valid * d * ELT));
    // sub-chunks: a uniform trip count for all waves (barriers inside)
    for (int sub = row_begin; sub < row_end; sub += kWaves * RT * 16) {
      const int r_wave = sub + wave * RT * 16;
      f32x4 acc[RT][NT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[rt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
      if constexpr (kDma)
        project_rows_dma<RT, NT>(r, r_wave, rows_valid, d, d, P, acc, smem);
      else
        project_rows<ELT, AL, RT, NT, NT, PD>(r, r_wave, rows_valid, d, d, P, acc, pan);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int ta = 0; ta < NT; ++ta)
#pragma unroll
            for (int tb = ta; tb < NT; ++tb)
              if (tb < nt) cov[ta][tb] = mfma_f32_4(acc[rt][ta][j], acc[rt][tb][j], cov[ta][tb]);
    }
  }

  // partial block (nt*16)^2 of this wave; 16x16 C layout: lane (g, n) holds
  // rows 4g..4g+3 of column n
  const int kp = nt * 16;
  float* dst = partials + O.partial_base + ((int64_t)it.part * kWaves + wave) * kp * kp;
#pragma unroll
  for (int ta = 0; ta < NT; ++ta)
#pragma unroll
    for (int tb = ta; tb < NT; ++tb) {
      if (tb < nt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          dst[(ta * 16 + 4 * g + i) * kp + tb * 16 + m16] = cov[ta][tb][i];
          if (tb != ta) dst[(tb * 16 + m16) * kp + ta * 16 + 4 * g + i] = cov[ta][tb][i];
        }
      }
    }
}

int fsum_nt_instance(int nt_req) { return nt_req <= 1 ? 1 : (nt_req <= 2 ? 2 : 4); }
int fsum_rows_per_wave(int nt_inst) { return fsum_rt(nt_inst); }

hipError_t launch_fsum(int elt, int aligned, int nt, const FsumItem* items, int n_items,
                       const FsumOp* ops, float* partials, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
#define DATTRI_FSUM(E, A, N)                                                                   \
  if (elt == E && (aligned != 0) == A && nt == N) {                                            \
    hipLaunchKernelGGL((fsum_kernel<E, A, N>), dim3(n_items), dim3(256), 0, s, items, ops, partials); \
    return hipGetLastError();                                                                  \
  }
  DATTRI_FSUM(2, true, 1) DATTRI_FSUM(2, true, 2) DATTRI_FSUM(2, true, 4)
  DATTRI_FSUM(2, false, 1) DATTRI_FSUM(2, false, 2) DATTRI_FSUM(2, false, 4)
  DATTRI_FSUM(4, true, 1) DATTRI_FSUM(4, true, 2) DATTRI_FSUM(4, true, 4)
  DATTRI_FSUM(4, false, 1) DATTRI_FSUM(4, false, 2) DATTRI_FSUM(4, false, 4)
#undef DATTRI_FSUM
  return hipErrorInvalidValue;
}

// ------------------------------------------------------------- reductions
__global__ __launch_bounds__(256) void stat_reduce_kernel(const StatTask* __restrict__ tasks,
                                                          const float* __restrict__ parts,
                                                          uint8_t* __restrict__ state) {
  __shared__ float red[4][64];
  const StatTask t = tasks[blockIdx.x];
  const int el = threadIdx.x & 63, pl = threadIdx.x >> 6;
  const int n_out = t.rows * t.cols;
  float* dst = (float*)(state + t.dst_off);
  const float* base = parts + t.part_base;
  for (int e0 = blockIdx.y * 64; e0 < n_out; e0 += gridDim.y * 64) {  // uniform trip count
    const int e = e0 + el;
    float s = 0.f;
    if (e < n_out) {
      const int r = e / t.cols, c = e - r * t.cols;
      const float* p = base + (int64_t)r * t.ldp + c;
      const int64_t step = t.part_floats;
      int q = pl;
      for (; q + 12 < t.n_parts; q += 16) {
        const float v0 = p[q * step], v1 = p[(q + 4) * step], v2 = p[(q + 8) * step],
                    v3 = p[(q + 12) * step];
        s = (((s + v0) + v1) + v2) + v3;
      }
      for (; q < t.n_parts; q += 4) s += p[q * step];
    }
    red[pl][el] = s;
    __syncthreads();
    if (pl == 0 && e < n_out) dst[e] += ((red[0][el] + red[1][el]) + red[2][el]) + red[3][el];
    __syncthreads();
  }
  if (blockIdx.y == 0 && threadIdx.x == 0 && t.count_off >= 0) {
    int64_t add = t.count_add;
    if (t.lengths) {
      add = 0;
      for (int i = 0; i < t.n_len; ++i) add += min(max(t.lengths[i], 0), t.T);
    }
    *(int64_t*)(state + t.count_off) += add;
  }
}

hipError_t launch_stat_reduce(const StatTask* tasks, int n_tasks, int max_out, const float* parts,
                              uint8_t* state, hipStream_t s) {
  if (n_tasks <= 0) return hipSuccess;
  const int zb = (max(max_out, 1) + 63) / 64;
  hipLaunchKernelGGL(stat_reduce_kernel, dim3(n_tasks, zb < 64 ? zb : 64), dim3(256), 0, s, tasks,
                     parts, state);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void zero_kernel(i32x4* p, int64_t n16) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n16) p[i] = i32x4{0, 0, 0, 0};
}

hipError_t launch_zero(void* p, int64_t bytes, hipStream_t s) {
  if (bytes <= 0) return hipSuccess;
  if (bytes % 16 || (uintptr_t)p % 16) return hipErrorInvalidValue;
  const int64_t n16 = bytes / 16;
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)((n16 + 255) / 256)), dim3(256), 0, s, (i32x4*)p, n16);
  return hipGetLastError();
}

// ------------------------------------------------ sums of stored projected rows
constexpr int kRowTile = 64;  // token rows staged in LDS per step

__global__ __launch_bounds__(256) void rowcov_kernel(const RowOp* __restrict__ ops,
                                                     float* __restrict__ parts) {
  constexpr int K = kCurvMaxK, PER = kRowTile * K / 256;  // tile elements per thread
  __shared__ __align__(16) float R[kRowTile * K];
  const RowOp o = ops[blockIdx.y];
  if ((int)blockIdx.x >= o.n_items) return;
  const int k = o.k, tid = threadIdx.x;
  const int nb = (k + 3) / 4;                      // 4 x 4 blocks per side
  const int bi = tid / nb, bj = tid - (tid / nb) * nb;
  const bool active = bi < nb;
  const int c0 = 4 * bi, r0 = 4 * bj;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
  const int e0 = blockIdx.x * o.ex_per_item, e1 = min(o.n, e0 + o.ex_per_item);
  auto rows_of = [&](int ex) {
    return o.lengths ? min(max(o.lengths[ex], 0), o.T) : o.T;
  };
  // tiles of kRowTile rows, example by example; the next tile is loaded into
  // registers (zero past the example's rows and past column k) while the
  // current one is summed
  float st[PER];
  auto load = [&](int ex, int t0) {
    const int nr = min(kRowTile, rows_of(ex) - t0);
    const float* base = o.rows + ((int64_t)ex * o.T + t0) * o.ld + o.col0;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int e = tid + 256 * j, r = e / K, c = e % K;
      st[j] = r < nr && c < k ? base[(int64_t)r * o.ld + c] : 0.f;
    }
  };
  auto next = [&](int& ex, int& t0) {  // the tile after (ex, t0); ex == e1 when done
    t0 += kRowTile;
    while (ex < e1 && t0 >= rows_of(ex)) {
      ++ex;
      t0 = 0;
    }
  };
  int ex = e0, t0 = -kRowTile;
  next(ex, t0);
  if (ex < e1) load(ex, t0);
  while (ex < e1) {  // uniform trip count
    const int nr = min(kRowTile, rows_of(ex) - t0);
    __syncthreads();  // the previous tile's readers are done
#pragma unroll
    for (int j = 0; j < PER; ++j) R[tid + 256 * j] = st[j];
    __syncthreads();
    next(ex, t0);
    if (ex < e1) load(ex, t0);
    if (active) {
      for (int r = 0; r < nr; ++r) {
        const f32x4 a = *(const f32x4*)(R + r * K + c0);
        const f32x4 b = *(const f32x4*)(R + r * K + r0);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
      }
    }
  }
  if (active) {
    float* dst = parts + o.partial_base + (int64_t)blockIdx.x * k * k;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (c0 + i < k && r0 + j < k) dst[(c0 + i) * k + r0 + j] = acc[i][j];
  }
}

hipError_t launch_rowcov(const RowOp* ops, int n_ops, int max_items, float* parts, hipStream_t s) {
  if (n_ops <= 0 || max_items <= 0) return hipSuccess;
  if (n_ops > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(rowcov_kernel, dim3(max_items, n_ops), dim3(256), 0, s, ops, parts);
  return hipGetLastError();
}

__device__ inline float load_elem(const void* p, int bf16, int64_t i);

// ---------------------------------------------------- token-level scores
// Workgroup (TT token positions, example, QS query rows): every layer is
// staged as zero-padded tiles in LDS (the QS query blocks of 64 x 64, the
// chunk's TT x 64 a~ and g~ rows), loaded into registers one layer ahead so
// that the loads of layer l + 1 are in flight while layer l is computed.  The
// 256 / TT threads of a token split into QS query slots of PARTS parts; a part
// holds g~_t in registers and sums a~_t[c] (R g~_t)[c] over its share of c,
// reading rows of R as broadcast float4.  Each part accumulates over all
// layers in layer order and the parts are added in part order at the end
// (deterministic).  One query row takes TT = 32 (twice the workgroups, so two
// share a CU and hide each other's per-layer load latency).
// Token contributions a~_t^T R g~_t on float32 MFMA (32x32x2; layouts as
// for ekfac_kernel).  A workgroup holds kTokTokens token positions of one
// example, 32 per wave, and QS query rows; per layer, for each query,
//   Y[t][c] = sum_r g~_t[r] R[c][r]   (M = t, N = c, K = r; g~ rows and the
// query block R in LDS with 65-float rows, so every operand read is free of
// bank conflicts), and the lane holding Y[t][c] adds a~_t[c] Y[t][c], a~
// read straight from the kept rows (32 lanes read 128 contiguous bytes).  The
// next layer's rows and query blocks are loaded while a layer is computed;
// the sums over c are taken once at the end, in a fixed butterfly order.
constexpr int kTokRow = kCurvMaxK + 1;  // LDS row pitch (floats)
static_assert(kTokTokens == kWaves * 32, "32 token positions per wave");

template <int QS>
__global__ __launch_bounds__(256, QS == 1 ? 2 : 1) void token_kernel(const TokTask* __restrict__ tasks, int n_tasks,
                                                    const void* __restrict__ phi_q, int q_bf16, int64_t ld_q,
                                                    int64_t n_q, int64_t n, int T, float* __restrict__ out) {
  constexpr int K = kCurvMaxK, PER_Q = K * K / 256;
  __shared__ float R[QS][K * kTokRow];
  __shared__ float G[kWaves][32 * kTokRow];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, h = lane >> 5;
  const int tw = blockIdx.x * kTokTokens + 32 * wave;  // this wave's first token position
  const int64_t ex = blockIdx.y, q0 = (int64_t)blockIdx.z * QS;

  // prefetch registers: query block elements e = tid + 256 j (row c = e / 64,
  // col r = e % 64); g~ row j of the wave at lane r = lane; a~[t][c] for the
  // lane's C elements (t = 8 (v / 4) + 4 h + v % 4, c = 32 tc + l32)
  float rq[QS][PER_Q], rg[32], ra[2][16];
  // buffer offsets are formed at each load (not held in registers); rows past
  // the example's length and columns past k read as zero (out of range)
  auto fresh = [](uint32_t x) {
    asm volatile("" : "+v"(x));
    return x;
  };
  auto load = [&](int l) {
    const TokTask tk = tasks[l];
    const int ki = tk.k_in, ko = tk.k_out;
    int t_eff = T;
    if (tk.lengths) t_eff = min(max(tk.lengths[ex], 0), T);
    const int rows = max(0, min(t_eff, tw + 32) - tw);  // this wave's valid positions
    const rsrc_t rb = make_rsrc(tk.b_rows + ((ex * T + tw) * tk.b_ld + tk.b_col0), (uint32_t)(rows * tk.b_ld * 4));
    const rsrc_t ra_ = make_rsrc(tk.a_rows + ((ex * T + tw) * tk.a_ld + tk.a_col0), (uint32_t)(rows * tk.a_ld * 4));
    const uint32_t gb = lane < ko ? (uint32_t)lane * 4 : kOOB;
#pragma unroll
    for (int j = 0; j < 32; ++j)
      rg[j] = __builtin_bit_cast(float, load4(rb, gb == kOOB ? kOOB : fresh(gb) + (uint32_t)(j * tk.b_ld * 4)));
    const uint32_t ta = (uint32_t)((4 * h) * tk.a_ld * 4);
#pragma unroll
    for (int tc = 0; tc < 2; ++tc) {
      const int c = 32 * tc + l32;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const uint32_t off = fresh(ta + (uint32_t)c * 4) + (uint32_t)((8 * (v >> 2) + (v & 3)) * tk.a_ld * 4);
        ra[tc][v] = __builtin_bit_cast(float, load4(ra_, c < ki ? off : kOOB));
      }
    }
    const int qe = q_bf16 ? 2 : 4;
#pragma unroll
    for (int qq = 0; qq < QS; ++qq) {
      const int64_t qrow = q0 + qq;
      const rsrc_t rqs = make_rsrc((const uint8_t*)phi_q + (qrow * ld_q + tk.q_off) * qe,
                                   qrow < n_q ? (uint32_t)(ki * ko * qe) : 0u);
#pragma unroll
      for (int j = 0; j < PER_Q; ++j) {
        const int e = tid + 256 * j, c = e / K, r = e % K;
        const uint32_t off = c < ki && r < ko ? fresh((uint32_t)(c * ko + r) * qe) : kOOB;
        rq[qq][j] = q_bf16 ? bf16_bits_to_f32((uint16_t)load2(rqs, off)) : __builtin_bit_cast(float, load4(rqs, off));
      }
    }
  };

  float acc[QS][16];  // per query: the lane's share of each of its 16 token positions
#pragma unroll
  for (int qq = 0; qq < QS; ++qq)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[qq][v] = 0.f;
  if (n_tasks > 0) load(0);
  for (int l = 0; l < n_tasks; ++l) {  // uniform trip count
    __syncthreads();  // the previous layer's readers are done
#pragma unroll
    for (int j = 0; j < 32; ++j) G[wave][j * kTokRow + lane] = rg[j];
#pragma unroll
    for (int j = 0; j < PER_Q; ++j) {
      const int e = tid + 256 * j;
#pragma unroll
      for (int qq = 0; qq < QS; ++qq) R[qq][(e / K) * kTokRow + e % K] = rq[qq][j];
    }
    float a[2][16];
#pragma unroll
    for (int tc = 0; tc < 2; ++tc)
#pragma unroll
      for (int v = 0; v < 16; ++v) a[tc][v] = ra[tc][v];
    __syncthreads();
    if (l + 1 < n_tasks) load(l + 1);
    const float* g = G[wave] + l32 * kTokRow + h;
#pragma unroll
    for (int qq = 0; qq < QS; ++qq)
#pragma unroll
      for (int tc = 0; tc < 2; ++tc) {
        const float* rr = R[qq] + (32 * tc + l32) * kTokRow + h;
        f32x16 y;
#pragma unroll
        for (int v = 0; v < 16; ++v) y[v] = 0.f;
#pragma unroll
        for (int s2 = 0; s2 < K / 2; ++s2) y = __builtin_amdgcn_mfma_f32_32x32x2f32(g[2 * s2], rr[2 * s2], y, 0, 0, 0);
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[qq][v] = fmaf(a[tc][v], y[v], acc[qq][v]);
      }
  }
  // sum over c: the 32 lanes of a half hold the same 16 token positions
#pragma unroll
  for (int qq = 0; qq < QS; ++qq) {
    const int64_t q = q0 + qq;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      float x = acc[qq][v];
#pragma unroll
      for (int o = 16; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
      const int t = tw + 8 * (v >> 2) + 4 * h + (v & 3);
      if (l32 == 0 && q < n_q && t < T) out[(q * n + ex) * T + t] = x;
    }
  }
}

hipError_t launch_token_scores(const TokTask* tasks, int n_tasks, const void* phi_q, int q_bf16, int64_t ld_q,
                               int64_t n_q, int64_t n, int T, float* out, hipStream_t s) {
  if (n_tasks <= 0 || n_q <= 0 || n <= 0 || T <= 0) return hipSuccess;
  const int QS = n_q >= kTokQueries ? kTokQueries : (n_q >= 2 ? 2 : 1);  // query slots per workgroup
  const int64_t gx = (T + kTokTokens - 1) / kTokTokens, gz = (n_q + QS - 1) / QS;
  if (n > 65535 || gz > 65535) return hipErrorInvalidValue;
  const dim3 grid((unsigned)gx, (unsigned)n, (unsigned)gz);
  if (QS == 4)
    hipLaunchKernelGGL((token_kernel<4>), grid, dim3(256), 0, s, tasks, n_tasks, phi_q, q_bf16, ld_q, n_q, n, T, out);
  else if (QS == 2)
    hipLaunchKernelGGL((token_kernel<2>), grid, dim3(256), 0, s, tasks, n_tasks, phi_q, q_bf16, ld_q, n_q, n, T, out);
  else
    hipLaunchKernelGGL((token_kernel<1>), grid, dim3(256), 0, s, tasks, n_tasks, phi_q, q_bf16, ld_q, n_q, n, T, out);
  return hipGetLastError();
}

// ------------------------------------------------------------ eigensolver
constexpr int kEigLd = kCurvMaxK + 1;  // float64 row pitch: column walks spread over banks
constexpr int kEigSweeps = 32;

// Round r of the round-robin ordering of n (even) indices: pair i of the
// n/2 disjoint pairs.  Index 0 stays fixed, the others turn on a circle, so
// every pair of indices meets exactly once in n - 1 rounds.
__device__ inline void round_pair(int r, int i, int n, int* p, int* q) {
  const int L = n - 1;
  if (i == 0) {
    *p = 0;
    *q = 1 + r;
  } else {
    *p = 1 + (r + i) % L;
    *q = 1 + (r - i + L) % L;
  }
}

__device__ inline double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__global__ __launch_bounds__(256) void eigen_kernel(const EigTask* __restrict__ tasks,
                                                    uint8_t* __restrict__ state) {
  __shared__ double Am[kCurvMaxK * kEigLd];
  __shared__ double Vm[kCurvMaxK * kEigLd];
  __shared__ double rc[kCurvMaxK / 2], rs[kCurvMaxK / 2];
  __shared__ int rp[kCurvMaxK / 2], rq[kCurvMaxK / 2];
  __shared__ double red[2][4];
  __shared__ int rank[kCurvMaxK];
  const EigTask t = tasks[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int k = t.k, n = k + (k & 1), m = n / 2;
  const float* sum = (const float*)(state + t.sum_off);
  const int64_t cnt = *(const int64_t*)(state + t.count_off);
  const double scale = cnt > 0 ? 1.0 / (double)cnt : 0.0;
  for (int e = tid; e < n * n; e += 256) {
    const int i = e / n, j = e - (e / n) * n;
    double v = 0.0;
    if (i < k && j < k) v = 0.5 * ((double)sum[i * k + j] + (double)sum[j * k + i]) * scale;
    Am[i * kEigLd + j] = v;
    Vm[i * kEigLd + j] = i == j ? 1.0 : 0.0;
  }
  __syncthreads();

  for (int sweep = 0; sweep < kEigSweeps; ++sweep) {
    double off = 0.0, tot = 0.0;
    for (int e = tid; e < n * n; e += 256) {
      const int i = e / n, j = e - (e / n) * n;
      const double v = Am[i * kEigLd + j];
      tot += v * v;
      if (i != j) off += v * v;
    }
    off = wave_sum(off);
    tot = wave_sum(tot);
    if (lane == 0) {
      red[0][wave] = off;
      red[1][wave] = tot;
    }
    __syncthreads();
    off = ((red[0][0] + red[0][1]) + red[0][2]) + red[0][3];
    tot = ((red[1][0] + red[1][1]) + red[1][2]) + red[1][3];
    __syncthreads();
    if (off <= 1e-26 * tot) break;  // the same value in every thread: a uniform exit

    for (int r = 0; r < n - 1; ++r) {
      if (tid < m) {
        int p, q;
        round_pair(r, tid, n, &p, &q);
        double c = 1.0, s = 0.0;
        const double apq = Am[p * kEigLd + q];
        if (apq != 0.0) {
          // rotation in the (p, q) plane that zeroes a_pq: tan = root of
          // t^2 + 2 theta t - 1 = 0 of smaller magnitude
          const double theta = (Am[q * kEigLd + q] - Am[p * kEigLd + p]) / (2.0 * apq);
          double tn;
          if (fabs(theta) > 1e150)
            tn = 0.5 / theta;
          else
            tn = (theta >= 0.0 ? 1.0 : -1.0) / (fabs(theta) + sqrt(1.0 + theta * theta));
          c = 1.0 / sqrt(1.0 + tn * tn);
          s = tn * c;
        }
        rc[tid] = c;
        rs[tid] = s;
        rp[tid] = p;
        rq[tid] = q;
      }
      __syncthreads();
      // rows: A <- J^T A; thread (tid / 64, tid % 64) takes column tid % 64 of
      // the pairs tid / 64, + 4, ... (the pair indices were formed once above)
      if (lane < n) {
        for (int pi = wave; pi < m; pi += 4) {
          const int p = rp[pi], q = rq[pi];
          const double c = rc[pi], s = rs[pi];
          const double a = Am[p * kEigLd + lane], b = Am[q * kEigLd + lane];
          Am[p * kEigLd + lane] = c * a - s * b;
          Am[q * kEigLd + lane] = s * a + c * b;
        }
      }
      __syncthreads();
      // columns: A <- A J, V <- V J; row tid % 64 of the same pairs
      if (lane < n) {
        for (int pi = wave; pi < m; pi += 4) {
          const int p = rp[pi], q = rq[pi];
          const double c = rc[pi], s = rs[pi];
          const double a = Am[lane * kEigLd + p], b = Am[lane * kEigLd + q];
          Am[lane * kEigLd + p] = c * a - s * b;
          Am[lane * kEigLd + q] = s * a + c * b;
          const double va = Vm[lane * kEigLd + p], vb = Vm[lane * kEigLd + q];
          Vm[lane * kEigLd + p] = c * va - s * vb;
          Vm[lane * kEigLd + q] = s * va + c * vb;
        }
      }
      __syncthreads();
    }
  }

  // ascending order, ties by index
  if (tid < k) {
    const double li = Am[tid * kEigLd + tid];
    int rk = 0;
    for (int j = 0; j < k; ++j) {
      const double lj = Am[j * kEigLd + j];
      rk += (lj < li) || (lj == li && j < tid);
    }
    rank[tid] = rk;
  }
  __syncthreads();
  float* Q = (float*)(state + t.q_off);
  float* lam = (float*)(state + t.lam_off);
  for (int e = tid; e < k * k; e += 256) {
    const int row = e / k, col = e - (e / k) * k;
    Q[row * k + rank[col]] = (float)Vm[row * kEigLd + col];
  }
  if (tid < k) lam[rank[tid]] = (float)Am[tid * kEigLd + tid];
}

hipError_t launch_eigen(const EigTask* tasks, int n_tasks, uint8_t* state, hipStream_t s) {
  if (n_tasks <= 0) return hipSuccess;
  hipLaunchKernelGGL(eigen_kernel, dim3(n_tasks), dim3(256), 0, s, tasks, state);
  return hipGetLastError();
}

// -------------------------------------------------------- rotated blocks
constexpr int kLd = kCurvMaxK;  // float pitch of the LDS matrices

// c[i][j] = sum_{kk < K} L[kk][c0 + i] R[kk][r0 + j]  (LDS, rows kLd apart)
__device__ inline void mm4(const float* L, const float* R, int K, int c0, int r0, float (&c)[4][4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) c[i][j] = 0.f;
  for (int kk = 0; kk < K; ++kk) {
    const f32x4 l = *(const f32x4*)(L + kk * kLd + c0);
    const f32x4 r = *(const f32x4*)(R + kk * kLd + r0);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) c[i][j] = fmaf(l[i], r[j], c[i][j]);
  }
}

__device__ inline float load_elem(const void* p, int bf16, int64_t i) {
  return bf16 ? bf16_bits_to_f32(((const uint16_t*)p)[i]) : ((const float*)p)[i];
}

// Loads a k1 x k2 float32 matrix (row-major, dense) into an LDS matrix, and its
// transpose into T when T is not null.
__device__ inline void load_mat(float* M, float* Tr, const float* src, int k1, int k2) {
  for (int e = threadIdx.x; e < k1 * k2; e += 256) {
    const int r = e / k2, c = e - (e / k2) * k2;
    const float v = src[e];
    M[r * kLd + c] = v;
    if (Tr) Tr[c * kLd + r] = v;
  }
}

__device__ inline void zero_lds(float* M) {
  for (int e = threadIdx.x; e < kCurvMaxK * kLd; e += 256) M[e] = 0.f;
}

// EK-FAC rotation on float32 MFMA (32x32x2: lane l holds A[l % 32][l / 32]
// and B[l / 32][l % 32]; C element v of lane l is row 8 (v / 4) + 4 (l / 32)
// + v % 4, column l % 32).  One wave per training row, all k padded to 64:
//   Y1^T[b][c] = sum_a Psi[a][b] QA[a][c]  (M = b, N = c, K = a),
//   Y^T[r][c]  = sum_b QG[b][r] Y1^T[b][c] (M = r, N = c, K = b).
// The sum over b may take b in any order, so the second product's K step v
// of b-tile tb takes, in lane half h, b = 32 tb + 8 (v / 4) + 4 h + v % 4:
// its B operand is then exactly C element v of Y1^T's tile, with no data
// movement, and its A operand is QG[b][r] read from LDS.  Each wave sums
// Y^T squared over its rows; the four waves' sums are added in a fixed order.
__global__ __launch_bounds__(256, 2) void ekfac_kernel(const RotTask* __restrict__ tasks,
                                                       const uint8_t* __restrict__ state,
                                                       const void* __restrict__ phi, int phi_bf16,
                                                       int64_t ld, int64_t n, int rpb,
                                                       float* __restrict__ parts) {
  __shared__ __align__(16) float QA[kCurvMaxK * kLd];
  __shared__ __align__(16) float QG[kCurvMaxK * kLd];
  const RotTask t = tasks[blockIdx.y];
  if ((int)blockIdx.x >= t.n_blocks) return;
  const int ki = t.k_in, ko = t.k_out, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, l32 = lane & 31, h = lane >> 5;
  zero_lds(QA);
  zero_lds(QG);
  __syncthreads();
  load_mat(QA, nullptr, (const float*)(state + t.q_a), ki, ki);
  load_mat(QG, nullptr, (const float*)(state + t.q_g), ko, ko);
  __syncthreads();
  f32x16 acc[2][2];  // [r tile][c tile] of this wave's sum of Y^T squared
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[x][y][v] = 0.f;
  const int64_t e0 = (int64_t)blockIdx.x * rpb;
  const int64_t e1 = min(n, e0 + rpb);
  // Psi[a][b] for this lane: a = 2 s + h (s < 32), b = 32 tb + l32, read
  // through a descriptor over the row's block (zero outside ki x ko); the
  // offsets are formed at each load, not held in registers
  const int elt = phi_bf16 ? 2 : 4;
  const uint32_t lane_off = (uint32_t)((h * ko + l32) * elt);
  float ps[2][32];
  auto load_psi = [&](int64_t e) {
    const rsrc_t r = make_rsrc((const uint8_t*)phi + (e * ld + t.col) * elt, (uint32_t)(ki * ko * elt));
#pragma unroll
    for (int tb = 0; tb < 2; ++tb)
#pragma unroll
      for (int s2 = 0; s2 < 32; ++s2) {
        uint32_t off = lane_off;
        asm volatile("" : "+v"(off));
        off += (uint32_t)((2 * s2 * ko + 32 * tb) * elt);
        if (2 * s2 + h >= ki || 32 * tb + l32 >= ko) off = kOOB;
        ps[tb][s2] = phi_bf16 ? bf16_bits_to_f32((uint16_t)load2(r, off)) : __builtin_bit_cast(float, load4(r, off));
      }
  };
  for (int64_t e = e0 + wave; e < e1; e += kWaves) {
    load_psi(e);
    f32x16 y1[2][2];  // Y1^T [b tile][c tile]
#pragma unroll
    for (int tb = 0; tb < 2; ++tb)
#pragma unroll
      for (int tc = 0; tc < 2; ++tc) {
#pragma unroll
        for (int v = 0; v < 16; ++v) y1[tb][tc][v] = 0.f;
#pragma unroll
        for (int s2 = 0; s2 < 32; ++s2)
          y1[tb][tc] = __builtin_amdgcn_mfma_f32_32x32x2f32(ps[tb][s2], QA[(2 * s2 + h) * kLd + 32 * tc + l32],
                                                            y1[tb][tc], 0, 0, 0);
      }
#pragma unroll
    for (int tr = 0; tr < 2; ++tr)
#pragma unroll
      for (int tc = 0; tc < 2; ++tc) {
        f32x16 y;
#pragma unroll
        for (int v = 0; v < 16; ++v) y[v] = 0.f;
#pragma unroll
        for (int tb = 0; tb < 2; ++tb)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int b = 32 * tb + 8 * (v >> 2) + 4 * h + (v & 3);
            y = __builtin_amdgcn_mfma_f32_32x32x2f32(QG[b * kLd + 32 * tr + l32], y1[tb][tc][v], y, 0, 0, 0);
          }
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[tr][tc][v] = fmaf(y[v], y[v], acc[tr][tc][v]);
      }
  }
  // fixed-order sum of the four waves' blocks: slot w % 2 gets wave w, then
  // wave w + 2 adds to it, then the two slots are added (QA/QG reused)
  float* slot = (wave & 1) ? QG : QA;
  auto at = [&](int tr, int tc, int v) { return (32 * tc + l32) * kLd + 32 * tr + 8 * (v >> 2) + 4 * h + (v & 3); };
  __syncthreads();
  if (wave < 2) {
#pragma unroll
    for (int tr = 0; tr < 2; ++tr)
#pragma unroll
      for (int tc = 0; tc < 2; ++tc)
#pragma unroll
        for (int v = 0; v < 16; ++v) slot[at(tr, tc, v)] = acc[tr][tc][v];
  }
  __syncthreads();
  if (wave >= 2) {
#pragma unroll
    for (int tr = 0; tr < 2; ++tr)
#pragma unroll
      for (int tc = 0; tc < 2; ++tc)
#pragma unroll
        for (int v = 0; v < 16; ++v) slot[at(tr, tc, v)] += acc[tr][tc][v];
  }
  __syncthreads();
  // slot element (c, r) at c * kLd + r; the layer's partial block is c * ko + r
  float* dst = parts + t.part_base + (int64_t)blockIdx.x * ki * ko;
  for (int idx = tid; idx < ki * ko; idx += 256) {
    const int c = idx / ko, r = idx - (idx / ko) * ko;
    dst[idx] = QA[c * kLd + r] + QG[c * kLd + r];
  }
}

hipError_t launch_ekfac(const RotTask* tasks, int n_tasks, int max_blocks, const uint8_t* state,
                        const void* phi, int phi_bf16, int64_t ld, int64_t n, int rows_per_block,
                        float* parts, hipStream_t s) {
  if (n_tasks <= 0 || max_blocks <= 0 || n <= 0) return hipSuccess;
  if (n_tasks > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ekfac_kernel, dim3(max_blocks, n_tasks), dim3(256), 0, s, tasks, state, phi,
                     phi_bf16, ld, n, rows_per_block, parts);
  return hipGetLastError();
}

// Block sum of v over the workgroup in a fixed order (float64); every thread
// gets the same value.  Contains two barriers.
__device__ inline double block_sum(double v, double* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  const double s = ((red[0] + red[1]) + red[2]) + red[3];
  __syncthreads();
  return s;
}

constexpr int kPrecQueries = 8;  // query rows per workgroup

__global__ __launch_bounds__(256) void precond_kernel(const RotTask* __restrict__ tasks,
                                                      const uint8_t* __restrict__ state, int kind,
                                                      double rel, double abs_,
                                                      const void* __restrict__ phi_q, int in_bf16,
                                                      int64_t ld_q, int64_t n_q,
                                                      void* __restrict__ out, int out_bf16,
                                                      int64_t ld_out) {
  __shared__ __align__(16) float QA[kCurvMaxK * kLd];
  __shared__ __align__(16) float QAT[kCurvMaxK * kLd];
  __shared__ __align__(16) float QG[kCurvMaxK * kLd];
  __shared__ __align__(16) float QGT[kCurvMaxK * kLd];
  __shared__ __align__(16) float X[kCurvMaxK * kLd];
  __shared__ __align__(16) float YT[kCurvMaxK * kLd];
  __shared__ double red[4];
  const RotTask t = tasks[blockIdx.y];
  const int ki = t.k_in, ko = t.k_out, tid = threadIdx.x;
  const int nro = (ko + 3) / 4, nci = (ki + 3) / 4;
  const int ci = tid / nro, ri = tid - (tid / nro) * nro;
  const bool active = ci < nci;
  const int c0 = 4 * ci, r0 = 4 * ri;
  const float* lam_a = (const float*)(state + t.lam_a);
  const float* lam_g = (const float*)(state + t.lam_g);
  const float* sum_e = (const float*)(state + t.sum_e);
  const int64_t n_e = ((const int64_t*)(state + t.counts))[2];
  const float inv_e = n_e > 0 ? (float)(1.0 / (double)n_e) : 0.f;

  // damping: rel * mean eigenvalue of the layer + abs
  double mean;
  if (kind == 0) {
    double sa = 0.0, sg = 0.0;
    for (int i = tid; i < ki; i += 256) sa += (double)lam_a[i];
    for (int i = tid; i < ko; i += 256) sg += (double)lam_g[i];
    sa = block_sum(sa, red);
    sg = block_sum(sg, red);
    mean = sa * sg / ((double)ki * ko);
  } else {
    double se = 0.0;
    for (int i = tid; i < ki * ko; i += 256) se += (double)sum_e[i];
    se = block_sum(se, red);
    mean = n_e > 0 ? se / ((double)n_e * ki * ko) : 0.0;
  }
  const float delta = (float)(rel * mean + abs_);
  // this thread's 4 x 4 divisors E + delta
  float den[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = min(c0 + i, ki - 1), r = min(r0 + j, ko - 1);
      const float E = kind == 0 ? lam_a[c] * lam_g[r] : sum_e[c * ko + r] * inv_e;
      den[i][j] = E + delta;
    }

  zero_lds(QA);
  zero_lds(QAT);
  zero_lds(QG);
  zero_lds(QGT);
  zero_lds(X);
  zero_lds(YT);
  __syncthreads();
  load_mat(QA, QAT, (const float*)(state + t.q_a), ki, ki);
  load_mat(QG, QGT, (const float*)(state + t.q_g), ko, ko);

  const int64_t q0 = (int64_t)blockIdx.x * kPrecQueries;
  const int64_t q1 = min(n_q, q0 + kPrecQueries);
  for (int64_t q = q0; q < q1; ++q) {
    __syncthreads();  // the previous query's readers are done
    for (int idx = tid; idx < ki * ko; idx += 256) {
      const int c = idx / ko, r = idx - (idx / ko) * ko;
      X[c * kLd + r] = load_elem(phi_q, in_bf16, q * ld_q + t.col + idx);
    }
    __syncthreads();
    float y[4][4];
    if (active) {  // Y1 = Q_A^T Psi_q, stored transposed
      mm4(QA, X, ki, c0, r0, y);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) YT[(r0 + j) * kLd + c0 + i] = y[i][j];
    }
    __syncthreads();
    if (active) {  // W = (Y1 Q_G) / (E + delta), stored row-major over X
      mm4(YT, QG, ko, c0, r0, y);
    }
    __syncthreads();
    if (active) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) X[(c0 + i) * kLd + r0 + j] = y[i][j] / den[i][j];
    }
    __syncthreads();
    if (active) {  // Z1 = Q_A W, stored transposed
      mm4(QAT, X, ki, c0, r0, y);
    }
    __syncthreads();
    if (active) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) YT[(r0 + j) * kLd + c0 + i] = y[i][j];
    }
    __syncthreads();
    if (active) {  // out = Z1 Q_G^T
      mm4(YT, QGT, ko, c0, r0, y);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (c0 + i < ki && r0 + j < ko) {
            const int64_t o = q * ld_out + t.col + (int64_t)(c0 + i) * ko + r0 + j;
            if (out_bf16)
              ((uint16_t*)out)[o] = f32_to_bf16_bits(y[i][j]);
            else
              ((float*)out)[o] = y[i][j];
          }
        }
    }
  }
}

hipError_t launch_precondition(const RotTask* tasks, int n_tasks, const uint8_t* state, int kind,
                               double rel, double abs_, const void* phi_q, int in_bf16,
                               int64_t ld_q, int64_t n_q, void* out, int out_bf16, int64_t ld_out,
                               hipStream_t s) {
  if (n_tasks <= 0 || n_q <= 0) return hipSuccess;
  const int64_t qb = (n_q + kPrecQueries - 1) / kPrecQueries;
  if (n_tasks > 65535 || qb > INT32_MAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(precond_kernel, dim3((unsigned)qb, n_tasks), dim3(256), 0, s, tasks, state,
                     kind, rel, abs_, phi_q, in_bf16, ld_q, n_q, out, out_bf16, ld_out);
  return hipGetLastError();
}

}  // namespace dattri
