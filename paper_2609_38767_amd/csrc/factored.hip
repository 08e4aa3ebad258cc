// Factored route (Eq. (2), left side): per example and layer,
//   Psi = (A P_in)^T (B P_out),   Psi[c][r] = sum_t a~_t[c] g~_t[r],
// fused in one kernel over a work list of (input group, example, token chunk).
//
// A workgroup of 4 waves streams its token chunk of A once (shared by all
// layers of the group, e.g. q/k/v) and of each member's B once, straight from
// HBM into MFMA operand registers (16-byte buffer loads; ragged rows and
// feature tails read as zero).  Projection fragments come from L2 in the
// fragment-major layout (one coalesced 1 KiB load per wave).  The projected
// tiles A~ = A P_in and B~ = B P_out stay in accumulator registers, and the
// token contraction A~^T B~ is done from those registers with float32 MFMA
// (16x16x4): for the 16x16 C layout, lane (g, n) holds rows 4g..4g+3 of column
// n, which is exactly a K=4 operand slice per element index, for both factors.
// Each wave writes its float32 partial block; a second kernel sums partials
// in a fixed order (deterministic, no float atomics) and writes phi.
#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

template <int ELT, int RT, int NA, int NB>
__global__ __launch_bounds__(256) void factored_kernel(const FactItem* __restrict__ items,
                                                       const FactGroup* __restrict__ groups,
                                                       const FactMember* __restrict__ members,
                                                       float* __restrict__ partials) {
  constexpr int EPL = 16 / ELT;
  constexpr int KR = 4 * EPL;  // feature rows covered by one fragment
  const FactItem it = items[blockIdx.x];
  const FactGroup& G = groups[it.group];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, m16 = lane & 15;
  const int ex = it.example;
  const int T = G.T, d_in = G.d_in, na = G.na;
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
  const bool a_aligned = G.aligned != 0;
  const int nkb_a = (d_in + KR - 1) / KR;

  for (int r0 = row_begin + wave * RT * 16; r0 < row_end; r0 += kWaves * RT * 16) {
    // ---- A~ = A[rows] P_in(group), all member input tiles at once
    f32x4 acc_a[RT][NA];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int t = 0; t < NA; ++t) acc_a[rt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int kb = 0; kb < nkb_a; ++kb) {
      const int col = kb * KR + g * EPL;
      i32x4 af[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) af[rt] = load_frag<ELT>(ra, r0 + rt * 16 + m16, rows_valid, col, d_in, a_aligned);
#pragma unroll
      for (int t = 0; t < NA; ++t) {
        if (t < na) {
          const uint8_t* pb = (const uint8_t*)G.ptile[t];
          const int64_t off = (((int64_t)kb * G.ptile_nt[t] + G.ptile_local[t]) * 64 + lane) * 16;
          const i32x4 pf = *(const i32x4*)(pb + off);
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) acc_a[rt][t] = frag_mma<ELT>(af[rt], pf, acc_a[rt][t]);
        }
      }
    }
    // ---- each member: B~ = B[rows] P_out, then psi += A~^T B~ over these rows
    for (int mi = 0; mi < G.n_members; ++mi) {
      const FactMember& M = members[G.member0 + mi];
      const int d_out = M.d_out, nb = M.nb;
      const uint8_t* b_base = (const uint8_t*)M.B + (size_t)ex * T * d_out * ELT;
      const rsrc_t rb = make_rsrc(b_base, (uint32_t)((int64_t)rows_valid * d_out * ELT));
      const bool b_aligned = M.aligned != 0;
      const uint8_t* pout = (const uint8_t*)M.P_out;
      f32x4 acc_b[RT][NB];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int t = 0; t < NB; ++t) acc_b[rt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int nkb_b = (d_out + KR - 1) / KR;
      for (int kb = 0; kb < nkb_b; ++kb) {
        const int col = kb * KR + g * EPL;
        i32x4 bf[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) bf[rt] = load_frag<ELT>(rb, r0 + rt * 16 + m16, rows_valid, col, d_out, b_aligned);
#pragma unroll
        for (int t = 0; t < NB; ++t) {
          if (t < nb) {
            const i32x4 pf = *(const i32x4*)(pout + (((int64_t)kb * nb + t) * 64 + lane) * 16);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) acc_b[rt][t] = frag_mma<ELT>(bf[rt], pf, acc_b[rt][t]);
          }
        }
      }
      const int a0 = M.a_tile0, a1 = M.a_tile0 + M.na;
#pragma unroll
      for (int ta = 0; ta < NA; ++ta) {
        if (ta >= a0 && ta < a1) {
#pragma unroll
          for (int tb = 0; tb < NB; ++tb) {
            if (tb < nb) {
#pragma unroll
              for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                  psi[ta][tb] = mfma_f32_4(acc_a[rt][ta][j], acc_b[rt][tb][j], psi[ta][tb]);
            }
          }
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

// Sum the partial blocks of each (layer, example) in index order and write the
// layer block of phi: element (c, r) at column phi_offset + c*k_out + r.
__global__ __launch_bounds__(256) void reduce_kernel(const ReduceTask* __restrict__ tasks,
                                                     const float* __restrict__ partials,
                                                     void* __restrict__ phi, int phi_bf16,
                                                     int64_t ld_phi) {
  const ReduceTask t = tasks[blockIdx.y];
  const int ex_local = blockIdx.x;
  const int64_t ex = (int64_t)t.ex_begin + ex_local;
  const float* base = partials + t.partial_base + (int64_t)ex_local * t.n_parts * t.part_floats;
  const int n_out = t.k_in * t.k_out;
  for (int e = threadIdx.x; e < n_out; e += blockDim.x) {
    const int c = e / t.k_out, r = e - c * t.k_out;
    const float* p = base + c * t.ldp + r;
    float s = 0.f;
    for (int q = 0; q < t.n_parts; ++q) s += p[(int64_t)q * t.part_floats];
    const int64_t o = ex * ld_phi + t.phi_offset + e;
    if (phi_bf16)
      ((uint16_t*)phi)[o] = f32_to_bf16_bits(s);
    else
      ((float*)phi)[o] = s;
  }
}

// ------------------------------------------------------------ instances
// (NA, NB) instances compiled per element type; rows per wave (RT) shrinks as
// the accumulator footprint grows so that two waves fit per SIMD.
static int rt_for(int na, int nb) {
  if (na <= 2 && nb <= 2) return 4;
  if (na * nb <= 12) return 2;
  return 1;
}

void factored_instance(int elt, int na_req, int nb_req, int* na_inst, int* nb_inst, int* rows_per_wave) {
  (void)elt;
  const int na_list[] = {1, 2, 4, 6, 8};
  const int nb_list[] = {1, 2, 4};
  int na = 8, nb = 4;
  for (int v : na_list) if (v >= na_req) { na = v; break; }
  for (int v : nb_list) if (v >= nb_req) { nb = v; break; }
  *na_inst = na;
  *nb_inst = nb;
  *rows_per_wave = rt_for(na, nb);
}

template <int ELT, int NA, int NB>
static hipError_t launch_one(const FactItem* items, int n, const FactGroup* g, const FactMember* m,
                             float* part, hipStream_t s) {
  constexpr int RT = (NA <= 2 && NB <= 2) ? 4 : (NA * NB <= 12 ? 2 : 1);
  hipLaunchKernelGGL((factored_kernel<ELT, RT, NA, NB>), dim3(n), dim3(256), 0, s, items, g, m, part);
  return hipGetLastError();
}

#define DATTRI_FACT_CASE(E, A, B) \
  if (elt == E && na == A && nb == B) return launch_one<E, A, B>(items, n_items, groups, members, partials, s);

hipError_t launch_factored(int elt, int na, int nb, const FactItem* items, int n_items,
                           const FactGroup* groups, const FactMember* members, float* partials,
                           hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
#define DATTRI_FACT_NB(E, A) DATTRI_FACT_CASE(E, A, 1) DATTRI_FACT_CASE(E, A, 2) DATTRI_FACT_CASE(E, A, 4)
#define DATTRI_FACT_ALL(E) \
  DATTRI_FACT_NB(E, 1) DATTRI_FACT_NB(E, 2) DATTRI_FACT_NB(E, 4) DATTRI_FACT_NB(E, 6) DATTRI_FACT_NB(E, 8)
  DATTRI_FACT_ALL(2)
  DATTRI_FACT_ALL(4)
  return hipErrorInvalidValue;
}

hipError_t launch_reduce(const ReduceTask* tasks, int n_tasks, int n_examples, const float* partials,
                         void* phi, int phi_bf16, int64_t ld_phi, hipStream_t s) {
  if (n_tasks <= 0 || n_examples <= 0) return hipSuccess;
  hipLaunchKernelGGL(reduce_kernel, dim3(n_examples, n_tasks), dim3(256), 0, s, tasks, partials, phi,
                     phi_bf16, ld_phi);
  return hipGetLastError();
}

}  // namespace dattri
