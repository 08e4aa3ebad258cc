// Factored route (Eq. (2), left side): per example and layer,
//   Psi = (A P_in)^T (B P_out),   Psi[c][r] = sum_t a~_t[c] g~_t[r],
// fused in one kernel over a work list of (input group, example, token chunk).
//
// A workgroup of 4 waves owns a chunk of token rows of one example and one
// input group (layers sharing A, e.g. q/k/v).  For each sub-chunk of
// 4 x RT x 16 rows it streams A once and each member's B once from HBM.  bf16
// blocks with aligned rows and 2-tile output maps go through LDS by direct
// loads (project_rows_dma, up to 6 input tiles, so q/k/v and gate/up share
// one pass over A).  Otherwise rows go straight into MFMA operand registers:
// 16-byte buffer loads, prefetched PD
// k-blocks ahead in a register ring (ragged rows and feature tails read as
// zero through the descriptor range).  Projection fragments are staged once
// per workgroup in LDS, one panel of KP k-blocks at a time (loaded a panel
// ahead, one LDS-only barrier per panel, so prefetched loads stay in flight), and
// shared by the 4 waves.
//
// The projected tiles A~ = A P_in and B~ = B P_out stay in accumulators, and
// the token contraction A~^T B~ is done from those registers with float32 MFMA
// (16x16x4): in the 16x16 C layout lane (g, n) holds rows 4g..4g+3 of column n,
// which for each element index is a K=4 operand slice, identically for both
// factors.  Each wave writes its float32 partial block; a second kernel sums
// partials in a fixed order (deterministic, no float atomics) and writes phi.
#include "device_common.h"
#include "internal.h"
#include "project_rows.h"

namespace dattri {
using namespace dev;

// Two waves per SIMD where the accumulators and load ring fit in 256 VGPRs.
constexpr int waves_of(int na, int nb) { return ((na * nb <= 16 && na <= 6) || na * nb <= 8) ? 2 : 1; }

// Instances that stream factor rows by direct loads into LDS: output maps of
// 2 tiles with 2, 4 or 6 input tiles (one layer, or up to three sharing their
// input block), or of 4 tiles with 2 or 4 input tiles (k = 64 layers).
constexpr bool dma_instance(int elt, bool aligned, int na, int nb) {
  return elt == 2 && aligned &&
         ((nb == 2 && (na == 2 || na == 4 || na == 6)) || (nb == 4 && (na == 2 || na == 4)));
}

// Workgroups per CU the launch bounds ask for: the direct-load instances with
// 4 or 6 map tiles on a side hold 88-100 KiB of LDS, one per CU.
constexpr int occupancy_of(int elt, bool aligned, int na, int nb) {
  return !aligned ? 1 : (dma_instance(elt, aligned, na, nb) && (na > 2 || nb > 2)) ? 1 : waves_of(na, nb);
}

// Projected rows of a wave's RT x 16 token rows, tiles [t0, t0 + nt) of acc,
// into dst rows of k floats (columns >= k and rows >= row_end are skipped).
// 16x16 C layout: lane (g, n) holds rows 4g..4g+3 of column n.
template <int RT, int NT>
__device__ inline void store_rows(const f32x4 (&acc)[RT][NT], float* dst, int k, int t0, int nt, int r_wave,
                                  int row_end, int g, int m16) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int col = (t - t0) * 16 + m16;
      if (t >= t0 && t < t0 + nt && col < k) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = r_wave + rt * 16 + 4 * g + i;
          if (row < row_end) dst[(int64_t)row * k + col] = acc[rt][t][i];
        }
      }
    }
}

template <int ELT, bool AL, int RT, int NA, int NB>
__global__ __launch_bounds__(256, occupancy_of(ELT, AL, NA, NB)) void factored_kernel(const FactItem* __restrict__ items,
                                                          const FactGroup* __restrict__ groups,
                                                          const FactMember* __restrict__ members,
                                                          float* __restrict__ partials) {
  constexpr int NTL = NA > NB ? NA : NB;
  constexpr int PD = AL ? pd_of(RT, NA, NB) : 2;
  // bf16 with aligned rows, two output map tiles and 2, 4 or 6 input map
  // tiles (one layer, or up to three sharing their input block): factor rows
  // streamed through LDS by direct loads (project_rows_dma); otherwise operand
  // loads straight into registers with projection panels in LDS (project_rows)
  constexpr bool kDma = dma_instance(ELT, AL, NA, NB);
  constexpr int kPanBytes = 2 * kPanel * NTL * kFragBytes;
  constexpr int kSmem = kDma ? DmaLds<RT, kDma ? NTL : 2>::kBytes : kPanBytes;
  __shared__ __align__(1024) uint8_t smem[kSmem];
  auto pan = reinterpret_cast<uint8_t(*)[kPanel][NTL][kFragBytes]>(smem);
  const FactItem it = items[blockIdx.x];
  if (it.example < 0) return;  // padding item of the XCD-interleaved order
  const FactGroup& G = groups[it.group];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, m16 = lane & 15;
  const int ex = it.example;
  const int T = G.T, d_in = G.d_in;
  int t_eff = T;
  if (G.lengths) t_eff = min(max(G.lengths[ex], 0), T);
  const int row_begin = it.chunk * G.chunk_rows;
  const int row_end = min(row_begin + G.chunk_rows, t_eff);
  const int rows_valid = max(row_end, 0);

  f32x4 psi[NA][NB];
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) psi[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const uint8_t* a_base = (const uint8_t*)G.A + (size_t)ex * T * d_in * ELT;
  const rsrc_t ra = make_rsrc(a_base, (uint32_t)((int64_t)rows_valid * d_in * ELT));
  FragSrc<NA> pin;
  pin.nt = G.na;
#pragma unroll
  for (int t = 0; t < NA; ++t) {
    const int tt = t < G.na ? t : 0;
    pin.base[t] = (const uint8_t*)G.ptile[tt] + (int64_t)G.ptile_local[tt] * kFragBytes;
    pin.stride[t] = (int64_t)G.ptile_nt[tt] * kFragBytes;
  }

  // sub-chunks: a uniform trip count for all waves (barriers inside)
  for (int sub = row_begin; sub < row_end; sub += kWaves * RT * 16) {
    const int r_wave = sub + wave * RT * 16;
    f32x4 acc_a[RT][NA];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int t = 0; t < NA; ++t) acc_a[rt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (kDma)
      project_rows_dma<RT, NA>(ra, r_wave, rows_valid, d_in, d_in, pin, acc_a, smem);
    else
      project_rows<ELT, AL, RT, NA, NTL, PD>(ra, r_wave, rows_valid, d_in, d_in, pin, acc_a, pan);
    // projected input rows of every member that asks for them
    for (int mi = 0; mi < G.n_members; ++mi) {
      const FactMember& M = members[G.member0 + mi];
      if (M.rows_a)
        store_rows<RT, NA>(acc_a, M.rows_a + (int64_t)ex * T * M.k_in, M.k_in, M.a_tile0, M.na, r_wave,
                           row_end, g, m16);
    }

    for (int mi = 0; mi < G.n_members; ++mi) {
      const FactMember& M = members[G.member0 + mi];
      const int d_out = M.d_out, nb = M.nb;
      const uint8_t* b_base = (const uint8_t*)M.B + (size_t)ex * T * d_out * ELT;
      const rsrc_t rb = make_rsrc(b_base, (uint32_t)((int64_t)rows_valid * d_out * ELT));
      FragSrc<NB> pout;
      pout.nt = nb;
#pragma unroll
      for (int t = 0; t < NB; ++t) {
        pout.base[t] = (const uint8_t*)M.P_out + (int64_t)(t < nb ? t : 0) * kFragBytes;
        pout.stride[t] = (int64_t)nb * kFragBytes;
      }
      f32x4 acc_b[RT][NB];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int t = 0; t < NB; ++t) acc_b[rt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
      if constexpr (kDma)
        project_rows_dma<RT, NB>(rb, r_wave, rows_valid, d_out, d_out, pout, acc_b, smem);
      else
        project_rows<ELT, AL, RT, NB, NTL, PD>(rb, r_wave, rows_valid, d_out, d_out, pout, acc_b, pan);
      if (M.rows_b)
        store_rows<RT, NB>(acc_b, M.rows_b + (int64_t)ex * T * M.k_out, M.k_out, 0, nb, r_wave, row_end, g,
                           m16);

      // K slices (rt, j) outermost: consecutive MFMAs update different psi
      // blocks, so none waits on its predecessor's result
      const int a0 = M.a_tile0, a1 = M.a_tile0 + M.na;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int ta = 0; ta < NA; ++ta) {
            if (ta >= a0 && ta < a1) {
#pragma unroll
              for (int tb = 0; tb < NB; ++tb)
                if (tb < nb) psi[ta][tb] = mfma_f32_4(acc_a[rt][ta][j], acc_b[rt][tb][j], psi[ta][tb]);
            }
          }
    }
  }

  // ---- write this wave's partial block of every member
  const int part = (ex * G.n_chunks + it.chunk) * kWaves + wave;
  for (int mi = 0; mi < G.n_members; ++mi) {
    const FactMember& M = members[G.member0 + mi];
    const int ldp = M.nb * 16;
    float* dst = partials + M.partial_base + (int64_t)part * (M.na * 16) * ldp;
    const int a0 = M.a_tile0, a1 = M.a_tile0 + M.na;
#pragma unroll
    for (int ta = 0; ta < NA; ++ta) {
      if (ta >= a0 && ta < a1) {
#pragma unroll
        for (int tb = 0; tb < NB; ++tb) {
          if (tb < M.nb) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              dst[((ta - a0) * 16 + 4 * g + i) * ldp + tb * 16 + m16] = psi[ta][tb][i];
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------ instances
// Aligned instances per (input tiles NA, output tiles NB); one unaligned
// instance (8, 4) serves any group whose rows are not 16-byte multiples.
// Rows per wave RT keeps two waves per SIMD within the register file; the
// direct-load instances keep 4 row tiles per wave however many layers share
// the input block, so grouping those layers costs no rows in flight.
constexpr int rt_of(int elt, int na, int nb) {
  return (na <= 2 && nb <= 2) || dma_instance(elt, true, na, nb) ? 4 : ((na * nb <= 16 && na <= 6) ? 2 : 1);
}

bool factored_direct_loads(int elt, int na, int nb, int aligned) { return dma_instance(elt, aligned != 0, na, nb); }

void factored_instance(int elt, int na_req, int nb_req, int aligned, int* na_inst, int* nb_inst,
                       int* rows_per_wave) {
  int na = 8, nb = 4;
  if (aligned) {
    const int na_list[] = {1, 2, 4, 6, 8};
    const int nb_list[] = {1, 2, 4};
    for (int v : na_list) if (v >= na_req) { na = v; break; }
    for (int v : nb_list) if (v >= nb_req) { nb = v; break; }
    // bf16: round 1-tile maps up to the direct-load instances (the unused
    // tile's fragments read as zero), which stream the factor rows faster
    const int na2 = na == 1 ? 2 : na, nb2 = nb == 1 ? 2 : nb;
    if (dma_instance(elt, true, na2, nb2)) {
      na = na2;
      nb = nb2;
    }
  }
  *na_inst = na;
  *nb_inst = nb;
  *rows_per_wave = aligned ? rt_of(elt, na, nb) : 1;
}

template <int ELT, bool AL, int NA, int NB>
static hipError_t launch_one(const FactItem* items, int n, const FactGroup* g, const FactMember* m,
                             float* part, hipStream_t s) {
  constexpr int RT = AL ? rt_of(ELT, NA, NB) : 1;
  hipLaunchKernelGGL((factored_kernel<ELT, AL, RT, NA, NB>), dim3(n), dim3(256), 0, s, items, g, m, part);
  return hipGetLastError();
}

hipError_t launch_factored(int elt, int na, int nb, int aligned, const FactItem* items, int n_items,
                           const FactGroup* groups, const FactMember* members, float* partials,
                           hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
#define DATTRI_FACT_CASE(E, A, B) \
  if (elt == E && na == A && nb == B) return launch_one<E, true, A, B>(items, n_items, groups, members, partials, s);
#define DATTRI_FACT_NB(E, A) DATTRI_FACT_CASE(E, A, 1) DATTRI_FACT_CASE(E, A, 2) DATTRI_FACT_CASE(E, A, 4)
#define DATTRI_FACT_ALL(E) \
  DATTRI_FACT_NB(E, 1) DATTRI_FACT_NB(E, 2) DATTRI_FACT_NB(E, 4) DATTRI_FACT_NB(E, 6) DATTRI_FACT_NB(E, 8)
  if (!aligned) {
    if (na != 8 || nb != 4) return hipErrorInvalidValue;
    if (elt == 2) return launch_one<2, false, 8, 4>(items, n_items, groups, members, partials, s);
    if (elt == 4) return launch_one<4, false, 8, 4>(items, n_items, groups, members, partials, s);
    return hipErrorInvalidValue;
  }
  DATTRI_FACT_ALL(2)
  DATTRI_FACT_ALL(4)
#undef DATTRI_FACT_ALL
#undef DATTRI_FACT_NB
#undef DATTRI_FACT_CASE
  return hipErrorInvalidValue;
}

}  // namespace dattri
