// Scoring: S = (Phi_q diag(d)) Phi_train^T  (GradDot, Sec. 4.1, with an
// optional positive diagonal preconditioner applied once), float32 out.
//
// Both operands are row-major with the feature axis contiguous, which is the
// K-contiguous ("NT") form MFMA wants for both sides: a lane's 16-byte fragment
// is a contiguous slice of one row.  Workgroup tile 128 x 128, 4 waves in a
// 2 x 2 grid of 64 x 64 (4 x 4 MFMA tiles each), 128 bytes of K per stage,
// double-buffered in LDS with the next stage prefetched into registers while
// the current one is multiplied.  LDS rows are XOR-swizzled by 16-byte chunk.
// Tiles are remapped so that each XCD walks a contiguous range of training
// tiles, all query tiles of one training tile back to back, so a Phi_train
// tile is fetched into that XCD's L2 once and reused by every query tile.
// When the tiles alone cannot fill the chip (few queries and training rows,
// long feature rows), the feature axis is split over grid.y: each split writes
// its partial tile, and the splits are summed in split order.
#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

// dst[r][f] = src[r][f] * d[f] for f < F; rows ld_src / ld_dst elements apart
// (the padding of dst rows is not written).
template <int ELT>
__global__ __launch_bounds__(256) void scale_rows_kernel(const uint8_t* __restrict__ src,
                                                         int64_t ld_src,
                                                         const float* __restrict__ d,
                                                         uint8_t* __restrict__ dst, int64_t ld_dst,
                                                         int64_t rows, int64_t F) {
  const int64_t n = rows * F;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / F, f = i - r * F;
    if constexpr (ELT == 2) {
      const float x = bf16_bits_to_f32(((const uint16_t*)src)[r * ld_src + f]) * d[f];
      ((uint16_t*)dst)[r * ld_dst + f] = f32_to_bf16_bits(x);
    } else {
      ((float*)dst)[r * ld_dst + f] = ((const float*)src)[r * ld_src + f] * d[f];
    }
  }
}

constexpr int kBM = 128, kBN = 128, kRowBytes = 128;  // tile rows, K bytes per stage

template <int ELT>
__global__ __launch_bounds__(256) void score_gemm_kernel(const uint8_t* __restrict__ Q,
                                                         const uint8_t* __restrict__ X,
                                                         float* __restrict__ S, int n_q,
                                                         int n_train, int F, int ldq, int ldx,
                                                         int n_qt, int n_xt, int sps) {
  constexpr int EPL = 16 / ELT;
  constexpr int BK = kRowBytes / ELT;  // K elements per stage
  __shared__ __align__(16) uint8_t smem[2][2][kBM * kRowBytes];  // [stage][Q/X] 64 KiB
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, m16 = lane & 15, wm = wave >> 1, wn = wave & 1;

  // XCD-aware tile order (dispatch round-robins workgroups over 8 XCDs)
  const int nb = n_qt * n_xt, b = blockIdx.x;
  const int n_full = nb / 8 * 8;
  const int L = b < n_full ? (b % 8) * (n_full / 8) + b / 8 : b;
  const int qt = L % n_qt, xt = L / n_qt;
  const int q0 = qt * kBM, x0 = xt * kBN;
  const int rows_q = min(kBM, n_q - q0), rows_x = min(kBN, n_train - x0);
  // ranges end at the last row's F-th element (padding after it need not exist)
  const rsrc_t rq = make_rsrc(Q + (int64_t)q0 * ldq * ELT, (uint32_t)(((int64_t)(rows_q - 1) * ldq + F) * ELT));
  const rsrc_t rx = make_rsrc(X + (int64_t)x0 * ldx * ELT, (uint32_t)(((int64_t)(rows_x - 1) * ldx + F) * ELT));

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = (F + BK - 1) / BK;
  const int k0 = blockIdx.y * sps, k1 = min(nk, k0 + sps);  // this split's K steps
  S += (int64_t)blockIdx.y * n_q * n_train;                 // its partial tile (S itself when unsplit)
  i32x4 rqv[4], rxv[4];
  auto gload = [&](int kk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + 256 * i, row = c >> 3, ch = c & 7;
      const int col = kk * BK + ch * EPL;
      rqv[i] = load_frag_ld<ELT>(rq, row, rows_q, col, F, ldq);
      rxv[i] = load_frag_ld<ELT>(rx, row, rows_x, col, F, ldx);
    }
  };
  auto swrite = [&](int st) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + 256 * i, row = c >> 3, ch = c & 7;
      const int off = row * kRowBytes + ((ch ^ (row & 7)) << 4);
      *(i32x4*)(smem[st][0] + off) = rqv[i];
      *(i32x4*)(smem[st][1] + off) = rxv[i];
    }
  };

  if (k0 < k1) {
    gload(k0);
    swrite(0);
  }
  __syncthreads();
  for (int kk = k0; kk < k1; ++kk) {
    const int st = (kk - k0) & 1;
    if (kk + 1 < k1) gload(kk + 1);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      i32x4 af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = wm * 64 + i * 16 + m16, ch = s * 4 + g;
        af[i] = *(const i32x4*)(smem[st][0] + row * kRowBytes + ((ch ^ (row & 7)) << 4));
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = wn * 64 + j * 16 + m16, ch = s * 4 + g;
        bf[j] = *(const i32x4*)(smem[st][1] + row * kRowBytes + ((ch ^ (row & 7)) << 4));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = frag_mma<ELT>(af[i], bf[j], acc[i][j]);
    }
    if (kk + 1 < k1) swrite(st ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int x = x0 + wn * 64 + j * 16 + m16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int q = q0 + wm * 64 + i * 16 + 4 * g + r;
        if (q < n_q && x < n_train) S[(int64_t)q * n_train + x] = acc[i][j][r];
      }
    }
}

// ------------------------------------------------------ cosine normalization
// inv[r] = 1 / |row r (times d, when given)|, 0 for a zero row.  One wave per
// row, 16-byte loads (rows are 16-byte aligned and F a multiple of 16 bytes).
template <int ELT>
__global__ __launch_bounds__(256) void row_inv_norms_kernel(const uint8_t* __restrict__ X, int64_t ld,
                                                            int64_t rows, int64_t F,
                                                            const float* __restrict__ d,
                                                            float* __restrict__ inv) {
  constexpr int EPL = 16 / ELT;
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;  // the whole wave leaves; no barrier below
  const uint8_t* row = X + r * ld * ELT;
  float s = 0.f;
  for (int64_t f = (int64_t)lane * EPL; f < F; f += 64 * EPL) {
    // elements named explicitly: bit-casting single vector elements inside an
    // unrolled loop was compiled to read element 0 for every index
    const i32x4 v = *(const i32x4*)(row + f * ELT);
    float x[EPL];
    if constexpr (ELT == 2) {
      const uint32_t w0 = (uint32_t)v.x, w1 = (uint32_t)v.y, w2 = (uint32_t)v.z, w3 = (uint32_t)v.w;
      x[0] = bf16_bits_to_f32(w0 & 0xFFFFu); x[1] = bf16_bits_to_f32(w0 >> 16);
      x[2] = bf16_bits_to_f32(w1 & 0xFFFFu); x[3] = bf16_bits_to_f32(w1 >> 16);
      x[4] = bf16_bits_to_f32(w2 & 0xFFFFu); x[5] = bf16_bits_to_f32(w2 >> 16);
      x[6] = bf16_bits_to_f32(w3 & 0xFFFFu); x[7] = bf16_bits_to_f32(w3 >> 16);
    } else {
      const f32x4 fv = __builtin_bit_cast(f32x4, v);
      x[0] = fv.x; x[1] = fv.y; x[2] = fv.z; x[3] = fv.w;
    }
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const float y = d ? x[j] * d[f + j] : x[j];
      s = fmaf(y, y, s);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  if (lane == 0) inv[r] = s > 0.f ? 1.f / sqrtf(s) : 0.f;
}

// S[q][j] *= iq[q] * it[j] (rows of S dense, n_train apart).
__global__ __launch_bounds__(256) void scale_scores_kernel(float* __restrict__ S, int64_t n_q, int64_t n_train,
                                                           const float* __restrict__ iq,
                                                           const float* __restrict__ it) {
  for (int64_t q = blockIdx.x; q < n_q; q += gridDim.x) {
    const float a = iq[q];
    float* row = S + q * n_train;
    for (int64_t j = threadIdx.x; j < n_train; j += 256) row[j] *= a * it[j];
  }
}

hipError_t launch_cosine_scale(int elt, const void* Q, int64_t ldq, const float* d, const void* X, int64_t ldx,
                               float* S, int64_t n_q, int64_t n_train, int64_t F, float* inv_q, float* inv_t,
                               hipStream_t s) {
  if (n_q <= 0 || n_train <= 0) return hipSuccess;
  const int64_t bq = (n_q + 3) / 4, bt = (n_train + 3) / 4;
  if (bq > INT32_MAX || bt > INT32_MAX) return hipErrorInvalidValue;
  if (elt == 2) {
    hipLaunchKernelGGL(row_inv_norms_kernel<2>, dim3((unsigned)bq), dim3(256), 0, s, (const uint8_t*)Q, ldq, n_q,
                       F, d, inv_q);
    hipLaunchKernelGGL(row_inv_norms_kernel<2>, dim3((unsigned)bt), dim3(256), 0, s, (const uint8_t*)X, ldx,
                       n_train, F, nullptr, inv_t);
  } else {
    hipLaunchKernelGGL(row_inv_norms_kernel<4>, dim3((unsigned)bq), dim3(256), 0, s, (const uint8_t*)Q, ldq, n_q,
                       F, d, inv_q);
    hipLaunchKernelGGL(row_inv_norms_kernel<4>, dim3((unsigned)bt), dim3(256), 0, s, (const uint8_t*)X, ldx,
                       n_train, F, nullptr, inv_t);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned blocks = (unsigned)std::min<int64_t>(n_q, 4096);
  hipLaunchKernelGGL(scale_scores_kernel, dim3(blocks), dim3(256), 0, s, S, n_q, n_train, inv_q, inv_t);
  return hipGetLastError();
}

hipError_t launch_scale_rows(int elt, const void* src, int64_t ld_src, const float* d, void* dst,
                             int64_t ld_dst, int64_t rows, int64_t F, hipStream_t s) {
  const int64_t n = rows * F;
  if (n <= 0) return hipSuccess;
  const int blocks = (int)std::min<int64_t>((n + 255) / 256, 65536);
  if (elt == 2)
    hipLaunchKernelGGL(scale_rows_kernel<2>, dim3(blocks), dim3(256), 0, s, (const uint8_t*)src,
                       ld_src, d, (uint8_t*)dst, ld_dst, rows, F);
  else
    hipLaunchKernelGGL(scale_rows_kernel<4>, dim3(blocks), dim3(256), 0, s, (const uint8_t*)src,
                       ld_src, d, (uint8_t*)dst, ld_dst, rows, F);
  return hipGetLastError();
}

hipError_t launch_score_gemm(int elt, const void* Q, int64_t ldq, const float* d, const void* X,
                             int64_t ldx, float* S, int64_t n_q, int64_t n_train, int64_t F,
                             void* qws, int64_t ld_ws, float* partials, hipStream_t s) {
  if (n_q <= 0 || n_train <= 0) return hipSuccess;
  if (score_uses_big(elt, n_q, n_train))
    return launch_score_gemm_256(Q, ldq, d, X, ldx, S, n_q, n_train, F, qws, partials, s);
  if (d && F > 0) {  // scaled queries, row-major in the workspace
    if (!qws) return hipErrorInvalidValue;
    hipError_t e = launch_scale_rows(elt, Q, ldq, d, qws, ld_ws, n_q, F, s);
    if (e != hipSuccess) return e;
    Q = qws;
    ldq = ld_ws;
  }
  const int n_qt = (int)((n_q + kBM - 1) / kBM), n_xt = (int)((n_train + kBN - 1) / kBN);
  const int64_t nb = (int64_t)n_qt * n_xt;
  if (nb > INT32_MAX) return hipErrorInvalidValue;
  const int64_t nk = (F + kRowBytes / elt - 1) / (kRowBytes / elt);
  const int ks = score_ksplit(elt, n_q, n_train, F);
  const int sps = ks > 1 ? (int)((nk + ks - 1) / ks) : (int)std::max<int64_t>(nk, 1);
  if (ks > 1 && !partials) return hipErrorInvalidValue;
  float* out = ks > 1 ? partials : S;
  if (elt == 2)
    hipLaunchKernelGGL(score_gemm_kernel<2>, dim3((unsigned)nb, (unsigned)ks), dim3(256), 0, s,
                       (const uint8_t*)Q, (const uint8_t*)X, out, (int)n_q, (int)n_train, (int)F, (int)ldq,
                       (int)ldx, n_qt, n_xt, sps);
  else
    hipLaunchKernelGGL(score_gemm_kernel<4>, dim3((unsigned)nb, (unsigned)ks), dim3(256), 0, s,
                       (const uint8_t*)Q, (const uint8_t*)X, out, (int)n_q, (int)n_train, (int)F, (int)ldq,
                       (int)ldx, n_qt, n_xt, sps);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || ks == 1) return e;
  return launch_splitk_sum(partials, ks, n_q * n_train, S, s);
}

}  // namespace dattri
