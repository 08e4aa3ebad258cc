// Per-query top-k of the score matrix: the k largest scores of each row,
// largest first, equal scores ordered by lower training index.
//
// One workgroup (16 waves) per query row.  Scores are mapped to order-
// preserving 32-bit keys (-0.0 folded onto +0.0); rows are read with 16-byte
// loads where they are 16-byte aligned.
//
// Sampled path (rows of at least 64K scores, one read of the row): a 4096-bin
// histogram of the top 12 key bits over a sample (64 evenly spaced runs of 256
// scores) picks a bin b_s expected to hold a few times k scores at or above
// it; one pass over the row gathers every score in bins >= b_s into LDS.  If
// at least k and at most kCandMax were gathered, the top k are among them (the
// k-th largest key is at least the smallest gathered one), and a bitonic sort
// by (key desc, index asc) gives the exact answer.  Otherwise the row falls
// through to the exact paths below.
//
// Histogram path (two reads): the same histogram over the whole row locates
// the bin holding the k-th largest key; every score in that bin or above is
// gathered and sorted.
//
// Fallback (candidate sets above kCandMax, e.g. massive ties): an exact
// 4-pass 8-bit MSB radix select finds the key K* of the k-th largest element
// and how many copies of K* are needed; an ordered pass gathers every key > K*
// and the lowest-index copies of K*; then the same bitonic sort.
#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;
constexpr int kHistBits = 12;
constexpr int kHistBins = 1 << kHistBits;
constexpr int kCandMax = 2048;
constexpr int kSampleRuns = 64, kSampleRun = 256;   // 16384 sampled scores
constexpr int64_t kSampleMinRow = (int64_t)1 << 16;  // rows this long use the sample

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
  const bool vec = ((uintptr_t)row & 15) == 0;  // uniform over the workgroup

  // f(i, score) for every score of the row, 16-byte loads (two in flight per
  // thread) where the row is aligned
  auto for_row = [&](auto&& f) {
    if (vec) {
      const f32x4* r4 = (const f32x4*)row;
      const int n4 = n >> 2;
      int j = tid;
      for (; j + kTopkThreads < n4; j += 2 * kTopkThreads) {
        const f32x4 a = r4[j], b = r4[j + kTopkThreads];
        f(4 * j, a[0]); f(4 * j + 1, a[1]); f(4 * j + 2, a[2]); f(4 * j + 3, a[3]);
        const int jb = j + kTopkThreads;
        f(4 * jb, b[0]); f(4 * jb + 1, b[1]); f(4 * jb + 2, b[2]); f(4 * jb + 3, b[3]);
      }
      if (j < n4) {
        const f32x4 a = r4[j];
        f(4 * j, a[0]); f(4 * j + 1, a[1]); f(4 * j + 2, a[2]); f(4 * j + 3, a[3]);
      }
      for (int i = 4 * n4 + tid; i < n; i += kTopkThreads) f(i, row[i]);
    } else {
      for (int i = tid; i < n; i += kTopkThreads) f(i, row[i]);
    }
  };
  auto bin_of = [](uint32_t key) { return key >> (32 - kHistBits); };
  // highest bin whose suffix count (elements in bins >= it) reaches `need`,
  // and that suffix count; 64 groups of 64 bins are summed in parallel
  auto find_bin = [&](uint32_t need) {
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
        if (cum + total[grp] >= need) break;
        cum += total[grp];
      }
      int b = grp * 64 + 63;
      for (; b > grp * 64; --b) {
        if (cum + hist[b] >= need) break;
        cum += hist[b];
      }
      s_bin = (uint32_t)b;
      s_cand = cum + hist[b];
    }
    __syncthreads();
  };
  // gather every score in bins >= b0 (at most kCandMax stored); returns the count
  auto gather = [&](uint32_t b0) {
    if (tid == 0) s_gt = 0;
    __syncthreads();
    for_row([&](int i, float v) {
      const uint32_t key = score_key(v);
      if (bin_of(key) >= b0) {
        const uint32_t slot = atomicAdd(&s_gt, 1u);
        if (slot < (uint32_t)kCandMax) {
          cand_key[slot] = key;
          cand_idx[slot] = i;
        }
      }
    });
    __syncthreads();
    return s_gt;
  };
  auto sort_first = [&](uint32_t count) {
    int P = 1;
    while (P < (int)count) P <<= 1;
    for (int i = (int)count + tid; i < P; i += kTopkThreads) {
      cand_key[i] = 0u;
      cand_idx[i] = 0x7FFFFFFF;
    }
    __syncthreads();
    sort_candidates(cand_key, cand_idx, P);
  };

  // ---------------- sampled path
  bool done = false;
  if (n_train >= kSampleMinRow) {
    for (int i = tid; i < kHistBins; i += kTopkThreads) hist[i] = 0;
    __syncthreads();
    {
      const int c = tid >> 4, sub = tid & 15;
      const int start = (int)(((int64_t)c * n / kSampleRuns) & ~(int64_t)3);
#pragma unroll
      for (int m = 0; m < kSampleRun / 64; ++m) {
        const int i = start + m * 64 + sub * 4;  // in range: start + 256 <= n
        if (vec) {
          const f32x4 v = *(const f32x4*)(row + i);
#pragma unroll
          for (int e = 0; e < 4; ++e) atomicAdd(&hist[bin_of(score_key(v[e]))], 1u);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) atomicAdd(&hist[bin_of(score_key(row[i + e]))], 1u);
        }
      }
    }
    __syncthreads();
    const int64_t n_s = (int64_t)kSampleRuns * kSampleRun;
    const uint32_t r = (uint32_t)std::min<int64_t>(n_s, (2 * (int64_t)k * n_s + n - 1) / n + 4);
    find_bin(r);
    const uint32_t bs = s_bin;
    const uint32_t count = gather(bs);
    if (count >= (uint32_t)k && count <= (uint32_t)kCandMax) {
      sort_first(count);
      done = true;
    }
    __syncthreads();
  }
  if (done) {
    for (int i = tid; i < k; i += kTopkThreads) {
      const int32_t j = cand_idx[i];
      idx_out[q * k + i] = j;
      val_out[q * k + i] = row[j];
    }
    return;
  }

  // ---------------- histogram path: histogram of the top 12 key bits
  for (int i = tid; i < kHistBins; i += kTopkThreads) hist[i] = 0;
  __syncthreads();
  for_row([&](int, float v) { atomicAdd(&hist[bin_of(score_key(v))], 1u); });
  __syncthreads();
  find_bin((uint32_t)k);
  const uint32_t bstar = s_bin;
  const uint32_t n_cand = s_cand;
  if (n_cand <= (uint32_t)kCandMax) {
    gather(bstar);
    sort_first(n_cand);
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
