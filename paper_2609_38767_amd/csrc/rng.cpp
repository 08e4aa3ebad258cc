// Seeded Gaussian projection maps (host side of the library).
//
// App. A.2 ("Factor projection", "Random maps") asks for dense Gaussian maps
// whose two sides use distinct seeds derived from a per-layer base seed, fixed
// for every gradient that is compared.  The generator is built from published
// algorithms only: SplitMix64 (Steele, Lea & Flood 2014) for seed derivation,
// Philox4x32-10 (Salmon et al., SC 2011) as a counter-based stream, and the
// Box-Muller transform (1958).  The exact recipe is in include/dattri.h
// (dattri_bind_projection).  Values are computed in double, rounded to float32
// (RNE) and, for bf16 contexts, to bf16 (RNE), then packed in the
// fragment-major device layout.
#include <cmath>
#include <cstring>
#include <thread>
#include <algorithm>
#include <unordered_set>
#include <vector>

#include "internal.h"
#include "runtime.h"

namespace dattri {

static inline uint64_t splitmix_out(uint64_t state) {
  uint64_t z = state + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

uint64_t derive_side_seed(uint64_t global_seed, int layer, int side) {
  return splitmix_out(splitmix_out(global_seed) ^ (uint64_t)(2 * (int64_t)layer + side));
}

uint64_t derive_mask_seed(uint64_t global_seed, int layer) {
  return splitmix_out(splitmix_out(global_seed) ^ ((uint64_t)1 << 63) ^ (uint64_t)(uint32_t)layer);
}

static inline void philox10(uint32_t c[4], uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
    c[1] = (uint32_t)p1;
    c[3] = (uint32_t)p0;
    c[0] = n0;
    c[2] = n2;
  }
}

void philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
  philox10(c, key[0], key[1]);
  std::memcpy(out, c, sizeof(c));
}

double gaussian_entry(uint64_t seed64, uint64_t e) {
  uint32_t c[4] = {(uint32_t)e, (uint32_t)(e >> 32), 0u, 0u};
  philox10(c, (uint32_t)seed64, (uint32_t)(seed64 >> 32));
  const uint64_t a = ((uint64_t)c[0] << 32) | c[1];
  const uint64_t b = ((uint64_t)c[2] << 32) | c[3];
  const double u1 = (double)((a >> 11) + 1) * 0x1.0p-53;
  const double u2 = (double)(b >> 11) * 0x1.0p-53;
  return std::sqrt(-2.0 * std::log(u1)) * std::cos(2.0 * M_PI * u2);
}

double rademacher_entry(uint64_t seed64, uint64_t e) {
  uint32_t c[4] = {(uint32_t)e, (uint32_t)(e >> 32), 0u, 0u};
  philox10(c, (uint32_t)seed64, (uint32_t)(seed64 >> 32));
  return (c[0] >> 31) ? -1.0 : 1.0;
}

// Masks mask_id .. mask_id + count - 1 (m entries each) of a d_out x d_in
// gradient: the distinct flat indices u of the draw stream
// u_i = (x0:x1) mod (d_out d_in), Philox counter (i lo, i hi, 0, 0) under the
// layer's mask key, first occurrences kept; mask j is run j of m consecutive
// distinct draws, sorted by u = c * d_out + r; the masks are concatenated.
// Needs (mask_id + count) * m <= d_out * d_in / 2 (checked by the caller).
void mask_entries(uint64_t seed64, int d_in, int d_out, int m, int mask_id, int count,
                  std::vector<int32_t>& rows, std::vector<int32_t>& cols) {
  const uint64_t N = (uint64_t)d_in * (uint64_t)d_out;
  const size_t need = (size_t)(mask_id + count) * (size_t)m;
  std::unordered_set<uint64_t> seen;
  seen.reserve(2 * need);
  std::vector<uint64_t> order;
  order.reserve(need);
  for (uint64_t i = 0; order.size() < need; ++i) {
    uint32_t c[4] = {(uint32_t)i, (uint32_t)(i >> 32), 0u, 0u};
    philox10(c, (uint32_t)seed64, (uint32_t)(seed64 >> 32));
    const uint64_t u = ((((uint64_t)c[0]) << 32) | c[1]) % N;
    if (seen.insert(u).second) order.push_back(u);
  }
  rows.resize((size_t)count * m);
  cols.resize((size_t)count * m);
  for (int j = 0; j < count; ++j) {
    std::vector<uint64_t> run(order.begin() + (size_t)(mask_id + j) * m,
                              order.begin() + (size_t)(mask_id + j + 1) * m);
    std::sort(run.begin(), run.end());
    for (int e = 0; e < m; ++e) {
      rows[(size_t)j * m + e] = (int32_t)(run[e] % (uint64_t)d_out);
      cols[(size_t)j * m + e] = (int32_t)(run[e] / (uint64_t)d_out);
    }
  }
}

uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

float bf16_to_f32(uint16_t h) {
  const uint32_t u = (uint32_t)h << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

float round_to_compute(double x, int elt_bytes) {
  const float f = (float)x;
  return elt_bytes == 2 ? bf16_to_f32(f32_to_bf16_rne(f)) : f;
}

// Fill `logical` (d x k float32, row-major) with the rounded map values:
// kind 0 Gaussian N(0, 1/k), kind 1 Rademacher +-1/sqrt(k).
void seeded_map(uint64_t seed64, int d, int k, int elt_bytes, int kind, float* logical) {
  const int64_t total = (int64_t)d * k;
  const double scale = 1.0 / std::sqrt((double)k);
  unsigned hw = std::thread::hardware_concurrency();
  int nth = (int)std::min<int64_t>(hw ? hw : 1, std::max<int64_t>(1, total / 65536));
  nth = std::max(1, std::min(nth, 32));
  auto work = [&](int t) {
    const int64_t b = total * t / nth, e = total * (t + 1) / nth;
    for (int64_t i = b; i < e; ++i)
      logical[i] = round_to_compute(
          (kind == 1 ? rademacher_entry(seed64, (uint64_t)i) : gaussian_entry(seed64, (uint64_t)i)) * scale,
          elt_bytes);
  };
  if (nth == 1) { work(0); return; }
  std::vector<std::thread> th;
  for (int t = 0; t < nth; ++t) th.emplace_back(work, t);
  for (auto& x : th) x.join();
}

void pack_map(const float* logical, int d, int k, int elt_bytes, std::vector<uint8_t>& packed) {
  packed.assign((size_t)packed_bytes(d, k, elt_bytes), 0);
  for (int v = 0; v < d; ++v)
    for (int c = 0; c < k; ++c) {
      const int64_t off = packed_offset(v, c, k, elt_bytes);
      const float x = logical[(int64_t)v * k + c];
      if (elt_bytes == 2) {
        const uint16_t h = f32_to_bf16_rne(x);
        std::memcpy(&packed[off], &h, 2);
      } else {
        std::memcpy(&packed[off], &x, 4);
      }
    }
}

}  // namespace dattri
