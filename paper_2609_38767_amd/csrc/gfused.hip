// Materialized route in one pass for bf16 factor blocks with 16-byte aligned
// rows: per example, the weight gradient G = B^T A (Eq. (1)) is formed tile by
// tile and projected while the tile is on chip,
//   Psi = (P_out^T G P_in)^T = H^T P_out,   H = G P_in   (Eq. (2), right side),
// so G never goes to memory.
//
// Workgroup: 128 rows of G (output features u0 .. u0 + 127) of one example,
// over one chunk of its tokens and one range of its 128-column tiles (G is a
// sum over tokens and Psi a sum over the columns of G, so chunks and ranges
// give partial blocks that add up).  For each 128-column tile of G (input
// features v0 .. v0 + 127): the tile is formed over the chunk's tokens with bf16 MFMA
// (g_tile, gtile.h), written to LDS in float32, and H[rows, :] += G_tile
// P_in[v0 .. v0 + 127, :] by bf16 MFMA (16x16x32; the P_in fragment read from
// the packed map, lane (g, n) holding K slots g*8 + j of column n, so the G
// operand is the matching 8 columns of the lane's row), each G value split
// exactly into three bf16 terms (hi + mid + lo) whose products with the bf16
// map are exact in the float32 accumulation.  The next tile's first token
// stage and the next k-block's map fragments are loaded while a tile is
// projected.  After
// the last tile, Psi_part = H^T P_out[rows] from the H accumulators (their C
// layout is a K=4 operand slice per element index); the four waves' parts are
// added in LDS in wave order and the workgroup writes one partial block, which
// the reduce kernel adds to the others in index order.  Sums are float32
// throughout (bf16 products are exact in float32).
#include "device_common.h"
#include "gtile.h"
#include "internal.h"

namespace dattri {
using namespace dev;

constexpr int kGFPitch = kGFusedCols + 4;  // floats per LDS row of a tile
static_assert(kWaves * 2 * 16 == kGFusedRows, "row block: 4 waves x 2 row tiles of 16");

template <int NT>
__global__ __launch_bounds__(256, 1) void gfused_kernel(GFusedArgs a) {
  using C = GTile<2, 2>;
  static_assert(C::TM == kGFusedRows && C::TN == kGFusedCols, "tile");
  static_assert(kWaves * NT * 256 * 4 <= C::kLdsBytes, "wave sums reuse the token staging buffer");
  __shared__ __align__(16) uint8_t stage[C::kLdsBytes];
  __shared__ __align__(16) float Gs[kGFusedRows * kGFPitch];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, m16 = lane & 15, wu = wave >> 1, wv = wave & 1;
  const int r32 = lane & 31, kg = lane >> 5;
  // blockIdx.x = (row block * n_vsplit + column range) * n_tchunks + token chunk
  const int tc = blockIdx.x % a.n_tchunks, bv = blockIdx.x / a.n_tchunks;
  const int ub = bv / a.n_vsplit, vs = bv - ub * a.n_vsplit;
  const int v_begin = vs * a.vt_per_split * kGFusedCols;
  const int v_end = min(a.d_in, v_begin + a.vt_per_split * kGFusedCols);
  const int e_local = blockIdx.y, e = a.ex_begin + e_local;
  const int u0 = ub * kGFusedRows;
  int t_eff = a.T;
  if (a.lengths) t_eff = min(max(a.lengths[e], 0), a.T);
  const int t_begin = tc * a.tok_chunk;  // < T: n_tchunks = ceil(T / tok_chunk)
  const int rows = max(0, min(t_eff - t_begin, a.tok_chunk));
  const uint8_t* b_rows = (const uint8_t*)a.B + ((size_t)e * a.T + t_begin) * a.d_out * 2;
  const uint8_t* a_rows = (const uint8_t*)a.A + ((size_t)e * a.T + t_begin) * a.d_in * 2;
  const int na_all = (a.k_in + 15) >> 4, nb_all = (a.k_out + 15) >> 4;
  const int nkb = (a.d_in + 31) / 32;  // k-blocks of 32 rows of the packed bf16 P_in
  const int r_wave = wave * 32;        // this wave's rows of the block (two tiles of 16)
  const uint8_t* pin = (const uint8_t*)a.P_in;

  f32x4 H[2][NT];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int t = 0; t < NT; ++t) H[rt][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  // P_in fragments of k-block kb (zero past d_in or k_in: buffer range check)
  const rsrc_t rpin = make_rsrc(pin, (uint32_t)((int64_t)nkb * na_all * kFragBytes));
  auto pin_frags = [&](int kb, i32x4 (&pf)[NT]) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
      pf[t] = load16(rpin, (t < na_all && kb < nkb) ? (uint32_t)(((kb * na_all + t) * 64 + lane) * 16) : kOOB);
  };
  // Two float32 G values as three packed bf16 terms each: hi = v truncated to
  // bf16, mid = (v - hi) truncated, lo = v - hi - mid.  The differences are
  // exact and lo has at most 8 significant bits, so hi + mid + lo = v exactly
  // (away from the subnormal range).
  auto split2 = [](float x, float y, int& hi, int& mid, int& lo) {
    const uint32_t ux = __builtin_bit_cast(uint32_t, x), uy = __builtin_bit_cast(uint32_t, y);
    const float rx = x - __builtin_bit_cast(float, ux & 0xFFFF0000u);
    const float ry = y - __builtin_bit_cast(float, uy & 0xFFFF0000u);
    const uint32_t urx = __builtin_bit_cast(uint32_t, rx), ury = __builtin_bit_cast(uint32_t, ry);
    const uint32_t lx = __builtin_bit_cast(uint32_t, rx - __builtin_bit_cast(float, urx & 0xFFFF0000u));
    const uint32_t ly = __builtin_bit_cast(uint32_t, ry - __builtin_bit_cast(float, ury & 0xFFFF0000u));
    hi = (int)((ux >> 16) | (uy & 0xFFFF0000u));
    mid = (int)((urx >> 16) | (ury & 0xFFFF0000u));
    lo = (int)((lx >> 16) | (ly & 0xFFFF0000u));
  };

  // Token rows of the first tile, then of each next tile during the current
  // tile's last stage (g_tile_from), so the first stage of a tile is in
  // flight while the previous tile is projected.
  const GRows gr = g_rows(b_rows, a_rows, rows, a.d_out, a.d_in);
  GStage<2, 2> st;
  if (v_begin < v_end) g_load(gr, 0, u0, v_begin, st);
  for (int v0 = v_begin; v0 < v_end; v0 += kGFusedCols) {
    i32x4 pf[NT];
    pin_frags(v0 / 32, pf);  // in flight during the tile's token stages
    f32x16 acc[2][2];
    g_tile_from(gr, rows, u0, v0, v0 + kGFusedCols < v_end ? v0 + kGFusedCols : -1, stage, st, acc);
    // 32x32 C layout: lane l, element x holds tile row 8*(x/4) + 4*(l/32) + x%4
    // of block i, column l % 32 of block j
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int x = 0; x < 16; ++x)
          Gs[(wu * 64 + i * 32 + 8 * (x >> 2) + 4 * kg + (x & 3)) * kGFPitch + wv * 64 + j * 32 + r32] =
              acc[i][j][x];
    __syncthreads();
#pragma unroll
    for (int kbl = 0; kbl < kGFusedCols / 32; ++kbl) {
      const int kb = v0 / 32 + kbl;
      i32x4 pn[NT];
      if (kbl + 1 < kGFusedCols / 32) pin_frags(kb + 1, pn);
      if (kb < nkb) {  // uniform
        // the lane's 8 G values of each row tile (columns g*8 .. g*8 + 7 of
        // k-block kbl, matching the P_in fragment's K slots), as three bf16
        // terms; P_in is exactly bf16, so each term's products are exact in
        // the float32 accumulation of a bf16 MFMA
        i32x4 gs[2][3];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          const float* gp = &Gs[(r_wave + rt * 16 + m16) * kGFPitch + kbl * 32 + g * 8];
          const f32x4 g0 = *(const f32x4*)gp, g1 = *(const f32x4*)(gp + 4);
          int h[4], m[4], l[4];
          split2(g0[0], g0[1], h[0], m[0], l[0]);
          split2(g0[2], g0[3], h[1], m[1], l[1]);
          split2(g1[0], g1[1], h[2], m[2], l[2]);
          split2(g1[2], g1[3], h[3], m[3], l[3]);
          gs[rt][0] = i32x4{h[0], h[1], h[2], h[3]};
          gs[rt][1] = i32x4{m[0], m[1], m[2], m[3]};
          gs[rt][2] = i32x4{l[0], l[1], l[2], l[3]};
        }
        // fragments t >= na_all are zero, so their products leave H[., t] zero
#pragma unroll
        for (int q = 0; q < 3; ++q)
#pragma unroll
          for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) H[rt][t] = frag_mma<2>(gs[rt][q], pf[t], H[rt][t]);
      }
      if (kbl + 1 < kGFusedCols / 32)
#pragma unroll
        for (int t = 0; t < NT; ++t) pf[t] = pn[t];
    }
    __syncthreads();  // the next tile overwrites Gs and the staging buffer
  }

  // Psi_part = H^T P_out[u0 + rows]; lane (g, n): Psi rows c = 4g..4g+3 of
  // tile t, column n of tile tb.  Per output tile tb, the four packed P_out
  // fragments covering the block's 128 rows (k-blocks u0/32 .. u0/32 + 3,
  // zero past d_out) are first copied to LDS, one 16-byte load per thread.
  float* red = (float*)stage;
  uint8_t* po_lds = stage + kWaves * NT * 256 * 4;
  static_assert(kWaves * NT * 256 * 4 + 4 * kFragBytes <= C::kLdsBytes, "P_out staging fits beside the sums");
  const uint8_t* pout = (const uint8_t*)a.P_out;
  const int nkb_out = (a.d_out + 31) / 32;
  const int ldp = nb_all * 16;
  const int part_floats = na_all * 16 * ldp;
  float* dst =
      a.partials + ((int64_t)e_local * a.n_ublocks * a.n_vsplit * a.n_tchunks + blockIdx.x) * part_floats;
  for (int tb = 0; tb < nb_all; ++tb) {
    {
      const int kb = u0 / 32 + (tid >> 6);  // fragment (kb, tb); thread = lane of wave tid / 64
      const i32x4 v = kb < nkb_out ? *(const i32x4*)(pout + ((int64_t)(kb * nb_all + tb) * 64 + lane) * 16)
                                   : i32x4{0, 0, 0, 0};
      *(i32x4*)(po_lds + tid * 16) = v;
    }
    __syncthreads();
    // element (row w of the block, column tb*16 + n): fragment w / 32, lane
    // 16 ((w % 32) / 8) + n, bf16 slot w % 8
    float po[2][4];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int w = r_wave + rt * 16 + 4 * g + i;
        const uint16_t h = *(const uint16_t*)(po_lds + (w / 32) * kFragBytes + (16 * ((w % 32) / 8) + m16) * 16 +
                                              (w % 8) * 2);
        po[rt][i] = bf16_bits_to_f32(h);
      }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if (t < na_all) {
        f32x4 ps = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int i = 0; i < 4; ++i) ps = mfma_f32_4(H[rt][t][i], po[rt][i], ps);
#pragma unroll
        for (int i = 0; i < 4; ++i) red[(wave * NT + t) * 256 + (4 * g + i) * 16 + m16] = ps[i];
      }
    }
    __syncthreads();
    for (int idx = tid; idx < na_all * 256; idx += 256) {
      const int t = idx >> 8, w = idx & 255;
      const float s = ((red[t * 256 + w] + red[(NT + t) * 256 + w]) + red[(2 * NT + t) * 256 + w]) +
                      red[(3 * NT + t) * 256 + w];
      dst[(t * 16 + (w >> 4)) * ldp + tb * 16 + (w & 15)] = s;
    }
    __syncthreads();
  }
}

int gfused_tiles_in(int k_in) {
  const int na = (k_in + 15) / 16;
  return na <= 1 ? 1 : na <= 2 ? 2 : na <= 4 ? 4 : 8;
}

hipError_t launch_gfused(const GFusedArgs& a, hipStream_t s) {
  if (a.ex_count <= 0) return hipSuccess;
  const int64_t n_vt = (a.d_in + kGFusedCols - 1) / kGFusedCols;
  if (a.n_ublocks <= 0 || a.n_tchunks <= 0 || a.tok_chunk <= 0 || a.n_vsplit <= 0 || a.vt_per_split <= 0 ||
      a.ex_count > 65535 || (int64_t)a.n_ublocks * a.n_vsplit * a.n_tchunks > INT32_MAX ||
      (int64_t)a.n_tchunks * a.tok_chunk < a.T || (a.tok_chunk % kTrTokens) != 0 ||
      (int64_t)a.n_vsplit * a.vt_per_split < n_vt || (int64_t)(a.n_vsplit - 1) * a.vt_per_split >= n_vt)
    return hipErrorInvalidValue;
  const dim3 grid(a.n_ublocks * a.n_vsplit * a.n_tchunks, a.ex_count);
  switch (gfused_tiles_in(a.k_in)) {
    case 1: hipLaunchKernelGGL(gfused_kernel<1>, grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL(gfused_kernel<2>, grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL(gfused_kernel<4>, grid, dim3(256), 0, s, a); break;
    default:
      if ((a.k_in + 15) / 16 > kGFusedMaxTilesIn) return hipErrorInvalidValue;
      hipLaunchKernelGGL(gfused_kernel<8>, grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace dattri
