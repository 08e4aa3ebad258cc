// Materialized route of the cross-Gram matrix in one pass (Sec. 3.2
// "Factorized inner product" and "FLOP-aware routing": the route that forms
// each example's weight gradient DW = B^T A, Eq. (1), and takes Frobenius
// products), for bf16 factor blocks with 16-byte aligned rows and a small
// batch b.  DW never goes to memory: a workgroup owns one 128 x 128 tile of
// one layer's DW, one example j of batch b and a run of examples of batch a;
// it forms the tile of DW_b[j] once (g_tile_dma, gtile.h, float32
// accumulators), then for each example i of its run forms the tile of
// DW_a[i] in the same register layout and reduces sum over the tile of
// DW_a[i] * DW_b[j] (for the squared norms, DW_a[i] * DW_a[i]): per lane over
// its 64 elements, then across the wave by a fixed butterfly, then over the
// four waves in wave order.  The tile's value goes to parts[slot][i][j]
// (norms: parts[slot][i]), which kacc_kernel sums over all slots, in slot
// order, into K.  All one-pass layers of a call share one launch.
#include "device_common.h"
#include "gtile.h"
#include "internal.h"

namespace dattri {
using namespace dev;

__global__ __launch_bounds__(256, 2) void xone_kernel(XOneArgs a) {
  __shared__ __align__(16) uint8_t lds[GDma::kBytes];
  __shared__ float wsum[kWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int x = blockIdx.x, y = blockIdx.y;
  const int i_begin = blockIdx.z * a.ipw, i_end = min(a.ci, i_begin + a.ipw);
  auto put = [&](int i, float t) {
    if (a.diag)
      a.parts[(int64_t)x * a.ci + i] = t;
    else
      a.parts[((int64_t)x * a.ci + i) * a.cj + y] = t;
  };
  const XOneEntry E = a.entries[a.slot_entry[x]];
  // Workgroups go to the 8 XCDs (each with its own L2) in turn, and a layer's
  // slots start at a multiple of 8: slot s of the layer takes tile
  // (s % 8) (nslots / 8) + s / 8, so each XCD owns one band of consecutive
  // tiles, ordered along the wider side of DW, and reads its band of the
  // wider factor block once instead of every XCD reading all of it.
  const int ls = x - E.slot0, n_tiles = E.n_ub * E.n_vt;
  const int tile = (ls % 8) * (E.nslots / 8) + ls / 8;
  if (tile >= n_tiles) {  // padding slot (uniform)
    if (tid == 0)
      for (int i = i_begin; i < i_end; ++i) put(i, 0.f);
    return;
  }
  const bool u_major = E.n_ub >= E.n_vt;
  const int u0 = (u_major ? tile / E.n_vt : tile % E.n_ub) * kXOneTile;
  const int v0 = (u_major ? tile % E.n_vt : tile / E.n_ub) * kXOneTile;

  auto rows_of = [](const int32_t* len, int e, int T) { return len ? min(max(len[e], 0), T) : T; };
  auto tile_of = [&](const void* B, const void* A, const int32_t* len, int e, int T, f32x16 (&acc)[2][2]) {
    // the same for every lane; made visible as such, so the stage loop
    // branches on scalars instead of masking lanes
    const int rows = __builtin_amdgcn_readfirstlane(rows_of(len, e, T));
    const GRows r = g_rows((const uint8_t*)B + (size_t)e * T * E.d_out * 2,
                           (const uint8_t*)A + (size_t)e * T * E.d_in * 2, rows, E.d_out, E.d_in);
    g_tile_dma(r, rows, u0, v0, lds, acc);
  };
  f32x16 ref[2][2];
  if (!a.diag) tile_of(E.B2, E.A2, E.len2, a.j0 + y, E.T2, ref);
  for (int i = i_begin; i < i_end; ++i) {
    f32x16 g[2][2];
    tile_of(E.B1, E.A1, E.len1, a.i0 + i, E.T1, g);
    float s = 0.f;
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int v = 0; v < 16; ++v) s = __builtin_fmaf(g[p][q][v], a.diag ? g[p][q][v] : ref[p][q][v], s);
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m);
    if (lane == 0) wsum[wave] = s;
    __syncthreads();
    if (tid == 0) put(i, ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3]);
    __syncthreads();  // wsum is rewritten by the next example
  }
}

hipError_t launch_xone(const XOneArgs& a, hipStream_t s) {
  if (a.ci <= 0 || a.n_slots <= 0) return hipSuccess;
  if (a.ipw <= 0 || (!a.diag && (a.cj <= 0 || a.cj > 65535))) return hipErrorInvalidValue;
  const int nz = (a.ci + a.ipw - 1) / a.ipw;
  if (nz > 65535) return hipErrorInvalidValue;
  const dim3 grid((unsigned)a.n_slots, a.diag ? 1u : (unsigned)a.cj, (unsigned)nz);
  hipLaunchKernelGGL(xone_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace dattri
