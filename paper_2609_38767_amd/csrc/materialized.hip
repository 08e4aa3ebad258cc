// Materialized route: build each example's weight gradient (Eq. (1))
//   G = B^T A = sum_t g_t a_t^T            (d_out x d_in, float32)
// then project it with the Kronecker-structured map of Eq. (2), right side:
//   Psi = (P_out^T G P_in)^T,  computed as H = G P_in (d_out x k_in) and
//   Psi = H^T P_out, each workgroup contributing the rows of G it owns.
#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

// ---------------------------------------------------------------- G = B^T A
// Workgroup: 64 (u = output feature) x 64 (v = input feature) tile of G for one
// example; 4 waves in a 2 x 2 grid of 32 x 32.  The contraction runs over
// tokens, which is the strided axis of both factors, so each stage of 32
// tokens is loaded with coalesced 16-byte row reads and stored transposed in
// LDS ([feature][token], token contiguous); MFMA fragments are then 16-byte
// LDS reads.
constexpr int kGT = 32;  // tokens per stage

template <int ELT>
__global__ __launch_bounds__(256) void gradient_kernel(GradArgs a) {
  constexpr int EPL = 16 / ELT, KR = 4 * EPL;
  constexpr int ROW = kGT * ELT + 16;  // padded LDS row (bytes)
  __shared__ __align__(16) uint8_t Bs[64 * ROW];
  __shared__ __align__(16) uint8_t As[64 * ROW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, m16 = lane & 15, wu = wave >> 1, wv = wave & 1;
  const int e_local = blockIdx.z;
  const int e = a.ex_begin + e_local;
  const int u0 = blockIdx.y * 64, v0 = blockIdx.x * 64;
  int t_eff = a.T;
  if (a.lengths) t_eff = min(max(a.lengths[e], 0), a.T);
  const uint8_t* b_base = (const uint8_t*)a.B + (size_t)e * a.T * a.d_out * ELT;
  const uint8_t* a_base = (const uint8_t*)a.A + (size_t)e * a.T * a.d_in * ELT;
  const rsrc_t rb = make_rsrc(b_base, (uint32_t)((int64_t)t_eff * a.d_out * ELT));
  const rsrc_t ra = make_rsrc(a_base, (uint32_t)((int64_t)t_eff * a.d_in * ELT));
  const bool aligned = a.aligned != 0;

  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  constexpr int CH_PER_ROW = 64 / EPL;           // 16-byte chunks per 64-feature row
  constexpr int CHUNKS = kGT * CH_PER_ROW;       // per operand per stage
  for (int t0 = 0; t0 < t_eff; t0 += kGT) {
    for (int c = tid; c < CHUNKS; c += 256) {
      const int t = c / CH_PER_ROW, f = (c % CH_PER_ROW) * EPL;
      const i32x4 vb = load_frag<ELT>(rb, t0 + t, t_eff, u0 + f, a.d_out, aligned);
      const i32x4 va = load_frag<ELT>(ra, t0 + t, t_eff, v0 + f, a.d_in, aligned);
      if constexpr (ELT == 2) {
#pragma unroll
        for (int j = 0; j < EPL; ++j) {
          const int w = j >> 1, sh = (j & 1) * 16;
          *(uint16_t*)(Bs + (f + j) * ROW + t * 2) = (uint16_t)((uint32_t)vb[w] >> sh);
          *(uint16_t*)(As + (f + j) * ROW + t * 2) = (uint16_t)((uint32_t)va[w] >> sh);
        }
      } else {
#pragma unroll
        for (int j = 0; j < EPL; ++j) {
          *(int*)(Bs + (f + j) * ROW + t * 4) = vb[j];
          *(int*)(As + (f + j) * ROW + t * 4) = va[j];
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < kGT / KR; ++ks) {
      i32x4 af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *(const i32x4*)(Bs + (wu * 32 + i * 16 + m16) * ROW + (ks * KR + g * EPL) * ELT);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bf[j] = *(const i32x4*)(As + (wv * 32 + j * 16 + m16) * ROW + (ks * KR + g * EPL) * ELT);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = frag_mma<ELT>(af[i], bf[j], acc[i][j]);
    }
    __syncthreads();
  }

  float* Ge = a.G + (int64_t)e_local * a.d_out * a.d_in;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int v = v0 + wv * 32 + j * 16 + m16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int u = u0 + wu * 32 + i * 16 + 4 * g + r;
        if (u < a.d_out && v < a.d_in) Ge[(int64_t)u * a.d_in + v] = acc[i][j][r];
      }
    }
}

// --------------------------------------------------- Psi = (P_out^T G P_in)^T
// Workgroup: 64 rows of G (one 16-row slice per wave) of one example.  For
// each group of up to 8 input tiles: H = G[rows] P_in by float32 MFMA, with
// 64-row slabs of P_in converted to float32 and staged in LDS in operand order;
// then for every output tile, Psi_part = H^T P_out[rows] straight from the H
// accumulators (their C layout is a K=4 operand slice per element index).
// Each wave writes its partial block; the reduce kernel sums them in order.
constexpr int kPV = 64;  // P_in rows staged per LDS slab

template <int ELT>
__global__ __launch_bounds__(256) void gproject_kernel(GProjArgs a) {
  __shared__ __align__(16) float Ps[kPV / 16][kGProjMaxTilesIn][64][4];  // 32 KiB
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, m16 = lane & 15;
  const int ub = blockIdx.x, e = blockIdx.y;
  const int u0 = ub * kGProjRows + wave * 16;
  const float* Ge = a.G + (int64_t)e * a.d_out * a.d_in;
  const rsrc_t rg = make_rsrc(Ge, (uint32_t)((int64_t)a.d_out * a.d_in * 4));
  const bool g_aligned = (a.d_in % 4) == 0;
  const int na_all = (a.k_in + 15) >> 4, nb_all = (a.k_out + 15) >> 4;
  const int ldp = nb_all * 16;
  const int part_floats = na_all * 16 * ldp;
  float* dst = a.partials + ((int64_t)(e * a.n_ublocks + ub) * kWaves + wave) * part_floats;
  const uint8_t* pin = (const uint8_t*)a.P_in;
  const uint8_t* pout = (const uint8_t*)a.P_out;

  for (int ta0 = 0; ta0 < na_all; ta0 += kGProjMaxTilesIn) {
    const int nt = min(kGProjMaxTilesIn, na_all - ta0);
    f32x4 H[kGProjMaxTilesIn];
#pragma unroll
    for (int t = 0; t < kGProjMaxTilesIn; ++t) H[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int v0 = 0; v0 < a.d_in; v0 += kPV) {
      __syncthreads();
      for (int idx = tid; idx < (kPV / 16) * nt * 64 * 4; idx += 256) {
        const int j = idx & 3, ln = (idx >> 2) & 63, rest = idx >> 8;
        const int t = rest % nt, vs = rest / nt;
        const int v = v0 + vs * 16 + 4 * (ln >> 4) + j;
        const int c = (ta0 + t) * 16 + (ln & 15);
        Ps[vs][t][ln][j] = packed_elem<ELT>(pin, v, c, a.d_in, a.k_in);
      }
      __syncthreads();
#pragma unroll
      for (int vs = 0; vs < kPV / 16; ++vs) {
        const i32x4 gf = load_frag<4>(rg, u0 + m16, a.d_out, v0 + vs * 16 + 4 * g, a.d_in, g_aligned);
#pragma unroll
        for (int t = 0; t < kGProjMaxTilesIn; ++t) {
          if (t < nt) {
            const i32x4 pf = *(const i32x4*)&Ps[vs][t][lane][0];
            H[t] = frag_mma<4>(gf, pf, H[t]);
          }
        }
      }
    }
    for (int tb = 0; tb < nb_all; ++tb) {
      float po[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) po[i] = packed_elem<ELT>(pout, u0 + 4 * g + i, tb * 16 + m16, a.d_out, a.k_out);
#pragma unroll
      for (int t = 0; t < kGProjMaxTilesIn; ++t) {
        if (t < nt) {
          f32x4 ps = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int i = 0; i < 4; ++i) ps = mfma_f32_4(H[t][i], po[i], ps);
#pragma unroll
          for (int i = 0; i < 4; ++i) dst[((ta0 + t) * 16 + 4 * g + i) * ldp + tb * 16 + m16] = ps[i];
        }
      }
    }
  }
}

hipError_t launch_gradient(int elt, const GradArgs& a, hipStream_t s) {
  constexpr int kMaxZ = 65535;  // grid z limit: launch examples in slices
  for (int e0 = 0; e0 < a.ex_count; e0 += kMaxZ) {
    GradArgs c = a;
    c.ex_begin = a.ex_begin + e0;
    c.ex_count = min(kMaxZ, a.ex_count - e0);
    c.G = a.G + (int64_t)e0 * a.d_out * a.d_in;
    const dim3 grid((a.d_in + 63) / 64, (a.d_out + 63) / 64, c.ex_count);
    if (elt == 2)
      hipLaunchKernelGGL(gradient_kernel<2>, grid, dim3(256), 0, s, c);
    else
      hipLaunchKernelGGL(gradient_kernel<4>, grid, dim3(256), 0, s, c);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_gproject(int elt, const GProjArgs& a, hipStream_t s) {
  if (a.ex_count <= 0) return hipSuccess;
  const dim3 grid(a.n_ublocks, a.ex_count);
  if (elt == 2)
    hipLaunchKernelGGL(gproject_kernel<2>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(gproject_kernel<4>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace dattri
