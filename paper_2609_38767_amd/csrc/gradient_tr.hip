// Weight gradient of Eq. (1) for bf16 factor blocks, G = B^T A = sum_t g_t a_t^T
// (d_out x d_in, float32), one example per grid z slice.  Each workgroup forms
// one 128 x 128 tile of G over all of the example's tokens (g_tile_dma,
// gtile.h: token rows streamed into LDS by direct loads, MFMA operands read
// with the gfx950 transposing LDS read) and writes it.  Rows past the
// example's length and features past d read zero.
#include "device_common.h"
#include "gtile.h"
#include "internal.h"

namespace dattri {
using namespace dev;

__global__ __launch_bounds__(256, 2) void gradient_tr_kernel(GradArgs a) {
  __shared__ __align__(16) uint8_t lds[GDma::kBytes];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wu = wave >> 1, wv = wave & 1;
  const int e_local = blockIdx.z, e = a.ex_begin + e_local;
  const int u0 = blockIdx.y * 128, v0 = blockIdx.x * 128;
  int t_eff = a.T;
  if (a.lengths) t_eff = min(max(a.lengths[e], 0), a.T);
  f32x16 acc[2][2];
  const GRows r = g_rows((const uint8_t*)a.B + (size_t)e * a.T * a.d_out * 2,
                         (const uint8_t*)a.A + (size_t)e * a.T * a.d_in * 2, t_eff, a.d_out, a.d_in);
  g_tile_dma(r, t_eff, u0, v0, lds, acc);

  // 32x32 C layout: lane l, element v holds row 8*(v/4) + 4*(l/32) + v%4,
  // column l % 32 (32 lanes store 128 contiguous bytes of a row of G)
  float* Ge = a.G + (int64_t)e_local * a.d_out * a.d_in;
  const int r32 = lane & 31, kg = lane >> 5;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int v = v0 + wv * 64 + j * 32 + r32;
#pragma unroll
      for (int x = 0; x < 16; ++x) {
        const int u = u0 + wu * 64 + i * 32 + 8 * (x >> 2) + 4 * kg + (x & 3);
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
    hipLaunchKernelGGL(gradient_tr_kernel, grid, dim3(256), 0, s, c);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace dattri
