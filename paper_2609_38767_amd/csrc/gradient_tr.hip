// Weight gradient of Eq. (1) for bf16 factor blocks, G = B^T A = sum_t g_t a_t^T
// (d_out x d_in, float32), one example per grid z slice.
//
// The contraction runs over tokens, the strided axis of both factors.  Token
// rows are loaded with coalesced 16-byte reads and stored in LDS as they are
// ([token][feature], rows padded by 32 bytes so the four rows one transposing
// read touches fall into different banks).  MFMA operands, which need eight
// consecutive tokens of one feature per lane, are read with the gfx950 LDS
// transpose read (ds_read_b64_tr_b16): within each group of 16 lanes, when lane
// 4r + a addresses row k0 + r at features m0 + 4a .. m0 + 4a + 3, lane j
// receives rows k0 .. k0 + 3 of feature m0 + j; two such reads give the 8
// tokens of a v_mfma_f32_32x32x16_bf16 operand.
//
// Workgroup: 4 waves in a 2 x 2 grid, each wave a (32 WM) x (32 WN) block of
// G (WM x WN MFMA tiles); stages of 32 tokens are double-buffered in LDS with
// the next stage prefetched into registers.  Rows past the example's length and
// features past d read zero (buffer range checks).
#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

typedef short i16x4 __attribute__((ext_vector_type(4)));
#define LDS16(p) ((__attribute__((address_space(3))) i16x4*)(p))

constexpr int kTrTokens = 32;  // tokens per stage

template <int WM, int WN>
__global__ __launch_bounds__(256, 2) void gradient_tr_kernel(GradArgs a) {
  constexpr int TM = 64 * WM, TN = 64 * WN;         // workgroup tile: rows of G (d_out) x columns (d_in)
  constexpr int PB = TM * 2 + 32, PA = TN * 2 + 32;  // LDS row pitch in bytes
  constexpr int CB = kTrTokens * TM / 8 / 256;      // 16-byte chunks per thread per stage (B side)
  constexpr int CA = kTrTokens * TN / 8 / 256;      // (A side)
  static_assert(CB >= 1 && CA >= 1, "tile");
  __shared__ __align__(16) uint8_t Bs[2][kTrTokens * PB];
  __shared__ __align__(16) uint8_t As[2][kTrTokens * PA];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wu = wave >> 1, wv = wave & 1;
  const int e_local = blockIdx.z, e = a.ex_begin + e_local;
  const int u0 = blockIdx.y * TM, v0 = blockIdx.x * TN;
  int t_eff = a.T;
  if (a.lengths) t_eff = min(max(a.lengths[e], 0), a.T);
  const rsrc_t rb = make_rsrc((const uint8_t*)a.B + (size_t)e * a.T * a.d_out * 2,
                              (uint32_t)((int64_t)t_eff * a.d_out * 2));
  const rsrc_t ra = make_rsrc((const uint8_t*)a.A + (size_t)e * a.T * a.d_in * 2,
                              (uint32_t)((int64_t)t_eff * a.d_in * 2));

  f32x16 acc[WM][WN];
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  i32x4 pb[CB], pa[CA];
  auto gload = [&](int t0) {
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int c = tid + 256 * i, row = c / (TM / 8), fc = c % (TM / 8);
      const int u = u0 + fc * 8;
      const uint32_t off = u < a.d_out ? (uint32_t)(((int64_t)(t0 + row) * a.d_out + u) * 2) : kOOB;
      pb[i] = load16(rb, off);
    }
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int c = tid + 256 * i, row = c / (TN / 8), fc = c % (TN / 8);
      const int v = v0 + fc * 8;
      const uint32_t off = v < a.d_in ? (uint32_t)(((int64_t)(t0 + row) * a.d_in + v) * 2) : kOOB;
      pa[i] = load16(ra, off);
    }
  };
  auto swrite = [&](int st) {
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int c = tid + 256 * i, row = c / (TM / 8), fc = c % (TM / 8);
      *(i32x4*)(Bs[st] + row * PB + fc * 16) = pb[i];
    }
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int c = tid + 256 * i, row = c / (TN / 8), fc = c % (TN / 8);
      *(i32x4*)(As[st] + row * PA + fc * 16) = pa[i];
    }
  };
  // transposed operand of K step ks (16 tokens) for the 32 features starting
  // at local column m: lane 16q + 4r + a reads row 16ks + 8(q/2) + 4h + r at
  // features m + 16(q%2) + 4a, h = 0, 1
  const int q = lane >> 4, r = (lane >> 2) & 3, aa = lane & 3;
  auto frag = [&](const uint8_t* base, int pitch, int m, int ks) {
    const int row = ks * 16 + 8 * (q >> 1) + r;
    const uint8_t* p = base + row * pitch + (m + 16 * (q & 1) + 4 * aa) * 2;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS16(p));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS16(p + 4 * pitch));
    const i32x4 w = {__builtin_bit_cast(int, __builtin_shufflevector(lo, lo, 0, 1)),
                     __builtin_bit_cast(int, __builtin_shufflevector(lo, lo, 2, 3)),
                     __builtin_bit_cast(int, __builtin_shufflevector(hi, hi, 0, 1)),
                     __builtin_bit_cast(int, __builtin_shufflevector(hi, hi, 2, 3))};
    return w;
  };

  const int nst = (t_eff + kTrTokens - 1) / kTrTokens;
  if (nst > 0) {
    gload(0);
    swrite(0);
  }
  __syncthreads();
  for (int kk = 0; kk < nst; ++kk) {
    const int st = kk & 1;
    if (kk + 1 < nst) gload((kk + 1) * kTrTokens);
#pragma unroll
    for (int ks = 0; ks < kTrTokens / 16; ++ks) {
      i32x4 fa[WM], fb[WN];
#pragma unroll
      for (int i = 0; i < WM; ++i) fa[i] = frag(Bs[st], PB, wu * 32 * WM + i * 32, ks);
#pragma unroll
      for (int j = 0; j < WN; ++j) fb[j] = frag(As[st], PA, wv * 32 * WN + j * 32, ks);
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[i]),
                                                             __builtin_bit_cast(bf16x8, fb[j]), acc[i][j], 0, 0, 0);
    }
    if (kk + 1 < nst) swrite(st ^ 1);
    __syncthreads();
  }

  // 32x32 C layout: lane l, element v holds row 8*(v/4) + 4*(l/32) + v%4,
  // column l % 32 (32 lanes store 128 contiguous bytes of a row of G)
  float* Ge = a.G + (int64_t)e_local * a.d_out * a.d_in;
  const int r32 = lane & 31, kg = lane >> 5;
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j) {
      const int v = v0 + wv * 32 * WN + j * 32 + r32;
#pragma unroll
      for (int x = 0; x < 16; ++x) {
        const int u = u0 + wu * 32 * WM + i * 32 + 8 * (x >> 2) + 4 * kg + (x & 3);
        if (u < a.d_out && v < a.d_in) Ge[(int64_t)u * a.d_in + v] = acc[i][j][x];
      }
    }
}

// bf16 blocks whose rows are 16-byte aligned (the caller checks); one launch
// per slice of at most 65535 examples.
hipError_t launch_gradient_tr(const GradArgs& a, hipStream_t s) {
  constexpr int kMaxZ = 65535;
  for (int e0 = 0; e0 < a.ex_count; e0 += kMaxZ) {
    GradArgs c = a;
    c.ex_begin = a.ex_begin + e0;
    c.ex_count = min(kMaxZ, a.ex_count - e0);
    c.G = a.G + (int64_t)e0 * a.d_out * a.d_in;
    const dim3 grid((a.d_in + 127) / 128, (a.d_out + 127) / 128, c.ex_count);
    hipLaunchKernelGGL((gradient_tr_kernel<2, 2>), grid, dim3(256), 0, s, c);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace dattri
