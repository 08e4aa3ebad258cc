// Per-query top-k of the score matrix: the k largest scores of each row,
// largest first, equal scores ordered by lower training index.
//
// One workgroup (16 waves) per query row.  Scores are mapped to order-preserving
// 32-bit keys (-0.0 folded onto +0.0).  A 4-pass, 8-bit MSB radix select finds
// the exact key K* of the k-th largest element and how many copies of K* are
// needed; a final pass in index order gathers every key > K* and the
// lowest-index copies of K* (an ordered block scan), and a bitonic sort in LDS
// orders the k winners by (key desc, index asc).
#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;

__device__ inline uint32_t score_key(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  if (u == 0x80000000u) u = 0u;  // -0.0 == +0.0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__global__ __launch_bounds__(kTopkThreads) void topk_kernel(const float* __restrict__ S,
                                                            int64_t n_train, int k,
                                                            int32_t* __restrict__ idx_out,
                                                            float* __restrict__ val_out) {
  __shared__ uint32_t hist[kTopkWaves][256];
  __shared__ uint32_t total[256];
  __shared__ uint32_t cand_key[kTopkMax];
  __shared__ int32_t cand_idx[kTopkMax];
  __shared__ uint32_t wave_cnt[kTopkWaves];
  __shared__ uint32_t s_bin, s_rem, s_gt;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t q = blockIdx.x;
  const float* row = S + q * n_train;
  const int n = (int)n_train;

  uint32_t prefix = 0, mask = 0, remaining = (uint32_t)k;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int i = tid; i < kTopkWaves * 256; i += kTopkThreads) (&hist[0][0])[i] = 0;
    __syncthreads();
    for (int i = tid; i < n; i += kTopkThreads) {
      const uint32_t key = score_key(row[i]);
      if ((key & mask) == prefix) atomicAdd(&hist[wave][(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 256) {
      uint32_t s = 0;
      for (int w = 0; w < kTopkWaves; ++w) s += hist[w][tid];
      total[tid] = s;
    }
    __syncthreads();
    if (tid == 0) {
      uint32_t cum = 0;
      int b = 255;
      for (; b > 0; --b) {
        if (cum + total[b] >= remaining) break;
        cum += total[b];
      }
      s_bin = (uint32_t)b;
      s_rem = remaining - cum;
    }
    __syncthreads();
    prefix |= s_bin << shift;
    mask |= 0xFFu << shift;
    remaining = s_rem;
    __syncthreads();
  }
  // prefix = K*; `remaining` copies of K* are needed, and all k - remaining
  // keys greater than K* are in the answer.
  const uint32_t kstar = prefix;
  const int n_gt = k - (int)remaining;
  if (tid == 0) s_gt = 0;
  __syncthreads();
  uint32_t eq_taken = 0;
  for (int base = 0; base < n; base += kTopkThreads) {
    const int i = base + tid;
    const uint32_t key = i < n ? score_key(row[i]) : 0u;
    const bool gt = i < n && key > kstar;
    const bool eq = i < n && key == kstar;
    if (gt) {
      const uint32_t slot = atomicAdd(&s_gt, 1u);
      cand_key[slot] = key;
      cand_idx[slot] = i;
    }
    const uint64_t ball = __ballot(eq);
    const uint32_t before = __popcll(ball & ((1ull << lane) - 1ull));
    if (lane == 0) wave_cnt[wave] = (uint32_t)__popcll(ball);
    __syncthreads();
    uint32_t wave_base = 0, block_cnt = 0;
    for (int w = 0; w < kTopkWaves; ++w) {
      if (w < wave) wave_base += wave_cnt[w];
      block_cnt += wave_cnt[w];
    }
    if (eq) {
      const uint32_t r = eq_taken + wave_base + before;
      if (r < remaining) {
        cand_key[n_gt + r] = key;
        cand_idx[n_gt + r] = i;
      }
    }
    eq_taken += block_cnt;
    __syncthreads();
  }
  // bitonic sort of the k candidates (padded to a power of two) by
  // (key descending, index ascending)
  int P = 1;
  while (P < k) P <<= 1;
  for (int i = k + tid; i < P; i += kTopkThreads) {
    cand_key[i] = 0u;
    cand_idx[i] = 0x7FFFFFFF;
  }
  __syncthreads();
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < P; i += kTopkThreads) {
        const int j = i ^ stride;
        if (j > i) {
          const uint32_t ki = cand_key[i], kj = cand_key[j];
          const int32_t ii = cand_idx[i], ij = cand_idx[j];
          const bool i_first = ki > kj || (ki == kj && ii < ij);
          const bool ascending_block = (i & size) == 0;  // this block sorts "first" to the front
          if (ascending_block ? !i_first : i_first) {
            cand_key[i] = kj; cand_key[j] = ki;
            cand_idx[i] = ij; cand_idx[j] = ii;
          }
        }
      }
      __syncthreads();
    }
  }
  for (int i = tid; i < k; i += kTopkThreads) {
    const int32_t j = cand_idx[i];
    idx_out[q * k + i] = j;
    val_out[q * k + i] = row[j];
  }
}

hipError_t launch_topk(const float* S, int64_t n_q, int64_t n_train, int32_t k, int32_t* idx,
                       float* val, hipStream_t s) {
  if (n_q <= 0 || k <= 0) return hipSuccess;
  if (k > kTopkMax || k > n_train || n_q > INT32_MAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(topk_kernel, dim3((unsigned)n_q), dim3(kTopkThreads), 0, s, S, n_train, k, idx,
                     val);
  return hipGetLastError();
}

}  // namespace dattri
