// Per-query top-k of the score matrix: the k largest scores of each row,
// largest first, equal scores ordered by lower training index.
//
// One workgroup (16 waves) per query row.  Scores are mapped to order-
// preserving 32-bit keys (-0.0 folded onto +0.0).
//
// Fast path (two reads of the row): a 4096-bin histogram of the top 12 key
// bits locates the bin b* that holds the k-th largest key; every element with
// bin >= b* is a candidate (all of the top k are among them), candidates are
// gathered into LDS and bitonic-sorted by (key desc, index asc), and the first
// k are the answer.  For score rows of real workloads the candidate set is a
// few hundred elements.
//
// Fallback (rows whose candidate set exceeds kCandMax, e.g. massive ties): an
// exact 4-pass 8-bit MSB radix select finds the key K* of the k-th largest
// element and how many copies of K* are needed; an ordered pass gathers every
// key > K* and the lowest-index copies of K*; then the same bitonic sort.
#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;
constexpr int kHistBits = 12;
constexpr int kHistBins = 1 << kHistBits;
constexpr int kCandMax = 2048;

__device__ inline uint32_t score_key(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  if (u == 0x80000000u) u = 0u;  // -0.0 == +0.0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Bitonic sort of ck/ci[0, P) (P a power of two <= kCandMax) by key
// descending, index ascending.  Called by all threads.
__device__ inline void sort_candidates(uint32_t* ck, int32_t* ci, int P) {
  const int tid = threadIdx.x;
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < P; i += kTopkThreads) {
        const int j = i ^ stride;
        if (j > i) {
          const uint32_t ki = ck[i], kj = ck[j];
          const int32_t ii = ci[i], ij = ci[j];
          const bool i_first = ki > kj || (ki == kj && ii < ij);
          const bool ascending_block = (i & size) == 0;  // this block puts "first" in front
          if (ascending_block ? !i_first : i_first) {
            ck[i] = kj; ck[j] = ki;
            ci[i] = ij; ci[j] = ii;
          }
        }
      }
      __syncthreads();
    }
  }
}

__global__ __launch_bounds__(kTopkThreads) void topk_kernel(const float* __restrict__ S,
                                                            int64_t n_train, int k,
                                                            int32_t* __restrict__ idx_out,
                                                            float* __restrict__ val_out) {
  // hist: the 4096-bin histogram, or 16 x 256 per-wave bins of the fallback
  __shared__ uint32_t hist[kHistBins];
  __shared__ uint32_t cand_key[kCandMax];
  __shared__ int32_t cand_idx[kCandMax];
  __shared__ uint32_t total[256];
  __shared__ uint32_t wave_cnt[kTopkWaves];
  __shared__ uint32_t s_bin, s_cand, s_rem, s_gt;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t q = blockIdx.x;
  const float* row = S + q * n_train;
  const int n = (int)n_train;

  // ---------------- fast path: histogram of the top 12 key bits
  for (int i = tid; i < kHistBins; i += kTopkThreads) hist[i] = 0;
  __syncthreads();
  for (int i = tid; i < n; i += kTopkThreads) atomicAdd(&hist[score_key(row[i]) >> (32 - kHistBits)], 1u);
  __syncthreads();
  // b* = the highest bin whose suffix count (elements in bins >= b*) reaches k:
  // 64 groups of 64 bins are summed in parallel, then one thread walks the
  // group totals and the bins of the group that holds b*
  if (tid < 64) {
    uint32_t s = 0;
    for (int b = 0; b < 64; ++b) s += hist[tid * 64 + b];
    total[tid] = s;
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t cum = 0;  // elements in bins above the current one
    int grp = 63;
    for (; grp > 0; --grp) {
      if (cum + total[grp] >= (uint32_t)k) break;
      cum += total[grp];
    }
    int b = grp * 64 + 63;
    for (; b > grp * 64; --b) {
      if (cum + hist[b] >= (uint32_t)k) break;
      cum += hist[b];
    }
    s_bin = (uint32_t)b;
    s_cand = cum + hist[b];
  }
  __syncthreads();
  const uint32_t bstar = s_bin;
  const uint32_t n_cand = s_cand;
  if (n_cand <= (uint32_t)kCandMax) {
    if (tid == 0) s_gt = 0;
    __syncthreads();
    for (int i = tid; i < n; i += kTopkThreads) {
      const uint32_t key = score_key(row[i]);
      if ((key >> (32 - kHistBits)) >= bstar) {
        const uint32_t slot = atomicAdd(&s_gt, 1u);
        cand_key[slot] = key;
        cand_idx[slot] = i;
      }
    }
    __syncthreads();
    int P = 1;
    while (P < (int)n_cand) P <<= 1;
    for (int i = (int)n_cand + tid; i < P; i += kTopkThreads) {
      cand_key[i] = 0u;
      cand_idx[i] = 0x7FFFFFFF;
    }
    __syncthreads();
    sort_candidates(cand_key, cand_idx, P);
  } else {
    // ---------------- fallback: exact radix select with ordered tie gathering
    uint32_t(*whist)[256] = reinterpret_cast<uint32_t(*)[256]>(hist);  // 16 x 256 bins
    uint32_t prefix = 0, mask = 0, remaining = (uint32_t)k;
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      for (int i = tid; i < kTopkWaves * 256; i += kTopkThreads) hist[i] = 0;
      __syncthreads();
      for (int i = tid; i < n; i += kTopkThreads) {
        const uint32_t key = score_key(row[i]);
        if ((key & mask) == prefix) atomicAdd(&whist[wave][(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (tid < 256) {
        uint32_t s = 0;
        for (int w = 0; w < kTopkWaves; ++w) s += whist[w][tid];
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
    // prefix = K*; `remaining` copies of K* are needed after the k - remaining
    // keys greater than K*
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
    int P = 1;
    while (P < k) P <<= 1;
    for (int i = k + tid; i < P; i += kTopkThreads) {
      cand_key[i] = 0u;
      cand_idx[i] = 0x7FFFFFFF;
    }
    __syncthreads();
    sort_candidates(cand_key, cand_idx, P);
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
