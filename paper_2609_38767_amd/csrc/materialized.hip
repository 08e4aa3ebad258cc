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
// Workgroup: 128 rows of G (two 16-row tiles per wave) of one example, over one
// range of d_in's k-blocks (d_in is split when row blocks times examples alone
// give too few workgroups).  H = G[rows, range] P_in[range, :] by float32 MFMA
// (16x16x4) with no LDS staging: each lane reads its 16-byte fragment of the
// packed P_in (element j of lane (g, n) is row g*EPL + j of the k-block,
// column n) and the matching EPL columns of its G row, so the j-th MFMA step
// contracts the K slots {g*EPL + j} of both operands.  Then
// Psi_part = H^T P_out[rows] straight from the H accumulators (their C layout
// is a K=4 operand slice per element index); the four waves' parts are summed
// in LDS in wave order and the workgroup writes one partial block, which the
// reduce kernel sums with the others in index order.
constexpr int kGRT = 2;  // row tiles per wave
static_assert(kWaves * kGRT * 16 == kGProjRows, "row block");

template <int ELT>
__global__ __launch_bounds__(256, 2) void gproject_kernel(GProjArgs a) {
  constexpr int EPL = 16 / ELT, KR = 4 * EPL, NH = EPL / 4;
  constexpr int NT = kGProjMaxTilesIn;
  __shared__ float red[kWaves][NT][256];  // 32 KiB
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, m16 = lane & 15;
  const int ub = blockIdx.x / a.n_ksplit, ks = blockIdx.x - ub * a.n_ksplit;
  const int e = blockIdx.y;
  const int u0 = ub * kGProjRows + wave * kGRT * 16;
  const float* Ge = a.G + (int64_t)e * a.d_out * a.d_in;
  const rsrc_t rg = make_rsrc(Ge, (uint32_t)((int64_t)a.d_out * a.d_in * 4));
  const bool g_aligned = (a.d_in % 4) == 0;
  const int nkb = (a.d_in + KR - 1) / KR;
  const int kb_begin = ks * a.kb_per_split, kb_end = min(nkb, kb_begin + a.kb_per_split);
  const int na_all = (a.k_in + 15) >> 4, nb_all = (a.k_out + 15) >> 4;
  const int ldp = nb_all * 16;
  const int part_floats = na_all * 16 * ldp;
  float* dst = a.partials + ((int64_t)e * a.n_ublocks * a.n_ksplit + blockIdx.x) * part_floats;
  const uint8_t* pin = (const uint8_t*)a.P_in;
  const uint8_t* pout = (const uint8_t*)a.P_out;

  auto load_g = [&](int kb, f32x4 (&gf)[kGRT][NH]) {
#pragma unroll
    for (int rt = 0; rt < kGRT; ++rt)
#pragma unroll
      for (int h = 0; h < NH; ++h)
        gf[rt][h] = __builtin_bit_cast(
            f32x4, load_frag<4>(rg, u0 + rt * 16 + m16, a.d_out, kb * KR + g * EPL + 4 * h, a.d_in, g_aligned));
  };

  for (int ta0 = 0; ta0 < na_all; ta0 += NT) {
    const int nt = min(NT, na_all - ta0);
    f32x4 H[kGRT][NT];
#pragma unroll
    for (int rt = 0; rt < kGRT; ++rt)
#pragma unroll
      for (int t = 0; t < NT; ++t) H[rt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 gcur[kGRT][NH], gnext[kGRT][NH];
    if (kb_begin < kb_end) load_g(kb_begin, gcur);
    for (int kb = kb_begin; kb < kb_end; ++kb) {
      if (kb + 1 < kb_end) load_g(kb + 1, gnext);
      i32x4 pf[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t)
        pf[t] = t < nt ? *(const i32x4*)(pin + ((int64_t)(kb * na_all + ta0 + t) * 64 + lane) * 16)
                       : i32x4{0, 0, 0, 0};
      // K slot j outermost: consecutive MFMAs update different H tiles, so
      // none waits on its predecessor's result
#pragma unroll
      for (int j = 0; j < EPL; ++j) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          if (t < nt) {
            float pv;
            if (ELT == 2) {
              const uint32_t w = (uint32_t)pf[t][j / 2];
              pv = bf16_bits_to_f32((j & 1) ? (w >> 16) : (w & 0xFFFFu));
            } else {
              pv = __builtin_bit_cast(f32x4, pf[t])[j];
            }
#pragma unroll
            for (int rt = 0; rt < kGRT; ++rt) H[rt][t] = mfma_f32_4(gcur[rt][j / 4][j % 4], pv, H[rt][t]);
          }
        }
      }
#pragma unroll
      for (int rt = 0; rt < kGRT; ++rt)
#pragma unroll
        for (int h = 0; h < NH; ++h) gcur[rt][h] = gnext[rt][h];
    }
    for (int tb = 0; tb < nb_all; ++tb) {
      float po[kGRT][4];
#pragma unroll
      for (int rt = 0; rt < kGRT; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          po[rt][i] = packed_elem<ELT>(pout, u0 + rt * 16 + 4 * g + i, tb * 16 + m16, a.d_out, a.k_out);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if (t < nt) {
          f32x4 ps = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int rt = 0; rt < kGRT; ++rt)
#pragma unroll
            for (int i = 0; i < 4; ++i) ps = mfma_f32_4(H[rt][t][i], po[rt][i], ps);
          // lane (g, n): Psi rows c = 4g..4g+3 of tile t, column n of tile tb
#pragma unroll
          for (int i = 0; i < 4; ++i) red[wave][t][(4 * g + i) * 16 + m16] = ps[i];
        }
      }
      __syncthreads();
      for (int idx = tid; idx < nt * 256; idx += 256) {
        const int t = idx >> 8, w = idx & 255;
        const float s = ((red[0][t][w] + red[1][t][w]) + red[2][t][w]) + red[3][t][w];
        dst[((ta0 + t) * 16 + (w >> 4)) * ldp + tb * 16 + (w & 15)] = s;
      }
      __syncthreads();
    }
  }
}

hipError_t launch_gradient(int elt, const GradArgs& a, hipStream_t s) {
  if (elt == 2 && a.aligned) return launch_gradient_tr(a, s);
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
  if (a.n_ublocks <= 0 || a.n_ksplit <= 0) return hipErrorInvalidValue;
  const dim3 grid(a.n_ublocks * a.n_ksplit, a.ex_count);
  if (elt == 2)
    hipLaunchKernelGGL(gproject_kernel<2>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(gproject_kernel<4>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace dattri
