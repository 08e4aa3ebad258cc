// Materialized route of the cross-Gram matrix in one pass (Sec. 3.2
// "Factorized inner product" and "FLOP-aware routing": the route that forms
// each example's weight gradient DW = B^T A, Eq. (1), and takes Frobenius
// products), for bf16 factor blocks with 16-byte aligned rows and a small
// batch b.  DW never goes to memory: a workgroup owns one 128 x 128 tile of
// DW, one example j of batch b and a run of examples of batch a; it forms
// the tile of DW_b[j] once (g_tile_dma, gtile.h, float32 accumulators), then for
// each example i of its run forms the tile of DW_a[i] in the same register
// layout and reduces sum over the tile of DW_a[i] * DW_b[j] (for the squared
// norms, DW_a[i] * DW_a[i]): per lane over its 64 elements, then across the
// wave by a fixed butterfly, then over the four waves in wave order.  The
// tile's value goes to parts[tile][i][j] (norms: parts[tile][i]), which
// kacc_kernel sums over the tiles in a fixed order into K.
#include "device_common.h"
#include "gtile.h"
#include "internal.h"

namespace dattri {
using namespace dev;

__global__ __launch_bounds__(256, 2) void xone_kernel(XOneArgs a) {
  __shared__ __align__(16) uint8_t lds[GDma::kBytes];
  __shared__ float wsum[kWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // Workgroups go to the 8 XCDs (each with its own L2) in turn: workgroup x
  // takes tile (x % 8) * (n / 8) + x / 8, so each XCD owns one band of
  // consecutive tiles, ordered along the wider side of DW: the XCD reads its
  // band of the wider factor block once, instead of every XCD reading all of it.
  const int n_ub = (a.d_out + kXOneTile - 1) / kXOneTile, n_tiles = n_ub * a.n_vt;
  const int tile = (n_tiles % 8 == 0) ? (blockIdx.x % 8) * (n_tiles / 8) + blockIdx.x / 8 : blockIdx.x;
  const int y = blockIdx.y;
  const bool u_major = n_ub >= a.n_vt;
  const int u0 = (u_major ? tile / a.n_vt : tile % n_ub) * kXOneTile;
  const int v0 = (u_major ? tile % a.n_vt : tile / n_ub) * kXOneTile;
  const int i_begin = blockIdx.z * a.ipw, i_end = min(a.ci, i_begin + a.ipw);

  auto rows_of = [](const int32_t* len, int e, int T) { return len ? min(max(len[e], 0), T) : T; };
  auto tile_of = [&](const void* B, const void* A, const int32_t* len, int e, int T, f32x16 (&acc)[2][2]) {
    const int rows = rows_of(len, e, T);
    const GRows r = g_rows((const uint8_t*)B + (size_t)e * T * a.d_out * 2,
                           (const uint8_t*)A + (size_t)e * T * a.d_in * 2, rows, a.d_out, a.d_in);
    g_tile_dma(r, rows, u0, v0, lds, acc);
  };
  f32x16 ref[2][2];
  if (!a.diag) tile_of(a.B2, a.A2, a.len2, a.j0 + y, a.T2, ref);
  for (int i = i_begin; i < i_end; ++i) {
    f32x16 g[2][2];
    tile_of(a.B1, a.A1, a.len1, a.i0 + i, a.T1, g);
    float s = 0.f;
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int x = 0; x < 16; ++x) s = __builtin_fmaf(g[p][q][x], a.diag ? g[p][q][x] : ref[p][q][x], s);
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m);
    if (lane == 0) wsum[wave] = s;
    __syncthreads();
    if (tid == 0) {
      const float t = ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
      if (a.diag)
        a.parts[(int64_t)tile * a.ci + i] = t;
      else
        a.parts[((int64_t)tile * a.ci + i) * a.cj + y] = t;
    }
    __syncthreads();  // wsum is rewritten by the next example
  }
}

hipError_t launch_xone(const XOneArgs& a, hipStream_t s) {
  const int n_ub = (a.d_out + kXOneTile - 1) / kXOneTile;
  if (a.ci <= 0) return hipSuccess;
  if (a.d_in <= 0 || a.d_out <= 0 || a.n_vt != (a.d_in + kXOneTile - 1) / kXOneTile || a.ipw <= 0 ||
      (!a.diag && (a.cj <= 0 || a.cj > 65535)) || (int64_t)n_ub * a.n_vt > INT32_MAX)
    return hipErrorInvalidValue;
  const int nz = (a.ci + a.ipw - 1) / a.ipw;
  if (nz > 65535) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(n_ub * a.n_vt), a.diag ? 1u : (unsigned)a.cj, (unsigned)nz);
  hipLaunchKernelGGL(xone_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace dattri
