// Materialized route in one pass for bf16 factor blocks with 16-byte aligned
// rows: per example, the weight gradient G = B^T A (Eq. (1)) is formed tile by
// tile and projected while the tile is in registers,
//   Psi = (P_out^T G P_in)^T = H^T P_out,   H = G P_in   (Eq. (2), right side),
// so G never goes to memory.
//
// Workgroup: 128 rows of G (output features u0 .. u0 + 127) of one example,
// over one chunk of its tokens and one range of its 128-column tiles (G is a
// sum over tokens and Psi a sum over the columns of G, so chunks and ranges
// give partial blocks that add up).  For each tile of 128 input features v0 ..
// v0 + 127, g_tile_dma (gtile.h) forms the transposed tile G^T[v][u] with bf16
// 32x32x16 MFMA.  In that C layout lane l holds one output feature u (l % 32)
// and 16 input features: element x is v = 8 (x / 4) + 4 (l / 32) + x % 4.
// Eight of them are exactly the K slots a 32x32x16 A operand takes from lane
// l, in the order
//   K slot s  <->  v = pi(s) = 8 ((s % 8) / 4) + 4 (s / 8) + s % 4,
// so the accumulators feed H[u][k] += sum_v G[u][v] P_in[v][k] directly, with
// the B operand (P_in) read from the packed map in the same permuted order:
// lane l takes rows 4 (l / 32) .. + 3 and 8 + 4 (l / 32) .. + 3 of a 16-row
// slice of column l % 32, two 8-byte pieces of one packed fragment.  No G
// values pass through LDS.  G is float32 and the MFMA takes bf16, so each G
// value is split exactly into three bf16 terms, hi + mid + lo (hi = v
// truncated to bf16, mid = (v - hi) truncated, lo = v - hi - mid: the
// differences are exact and lo has at most 8 significant bits); the map is
// exactly bf16, so every product is exact in the float32 accumulation.
//
// After the last tile, Psi_part[k][c] = sum_u H[u][k] P_out[u][c] in the same
// way: H's C layout gives lane l one k and 16 u's, split into three bf16
// terms, against permuted P_out slices.  The four waves' parts (each wave
// holds half the tile's v range for half its u range) are added in LDS in
// wave order and the workgroup writes one partial block, which the reduce
// kernel adds to the others in index order.
#include "device_common.h"
#include "gtile.h"
#include "internal.h"

namespace dattri {
using namespace dev;

static_assert(kGFusedRows == 128 && kGFusedCols == 128, "tile of g_tile_dma");

// Operand of K slots pi(0 .. 15) + 16 hx of the 32-row k-block kb of a packed
// bf16 map (k-blocks of 32 rows, 16-column tiles, lane (g, n) of a fragment
// holding rows 8 g .. 8 g + 7 of column n), column tile kt of 32 columns:
// lane l takes rows 16 hx + 4 (l / 32) + 0..3 from fragment lane (2 hx, n)
// and 16 hx + 8 + 4 (l / 32) + 0..3 from lane (2 hx + 1, n), n = l % 16, of
// tile 2 kt + (l % 32) / 16.  Zero past the map's k-blocks or column tiles.
__device__ inline i32x4 perm_operand(rsrc_t r, int kb, int nkb, int nt16, int kt, int hx, int lane) {
  const int t = 2 * kt + ((lane & 31) >> 4), n = lane & 15, h = lane >> 5;
  const bool ok = kb < nkb && t < nt16;
  const uint32_t off = (uint32_t)((((kb * nt16 + t) * 64 + 32 * hx + n) * 16) + 8 * h);
  const i32x2 lo = load8(r, ok ? off : kOOB);
  const i32x2 hi = load8(r, ok ? off + 16 * 16 : kOOB);  // fragment lane + 16
  return i32x4{lo[0], lo[1], hi[0], hi[1]};
}

// Elements 8 hx .. 8 hx + 7 of a 32x32 accumulator as three bf16x8 operands
// whose sum is exact (hi, mid, lo by truncation).
__device__ inline void split_terms(const f32x16& c, int hx, i32x4 (&term)[3]) {
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const float x = c[8 * hx + 2 * p], y = c[8 * hx + 2 * p + 1];
    const uint32_t ux = __builtin_bit_cast(uint32_t, x), uy = __builtin_bit_cast(uint32_t, y);
    const float rx = x - __builtin_bit_cast(float, ux & 0xFFFF0000u);
    const float ry = y - __builtin_bit_cast(float, uy & 0xFFFF0000u);
    const uint32_t urx = __builtin_bit_cast(uint32_t, rx), ury = __builtin_bit_cast(uint32_t, ry);
    const uint32_t lx = __builtin_bit_cast(uint32_t, rx - __builtin_bit_cast(float, urx & 0xFFFF0000u));
    const uint32_t ly = __builtin_bit_cast(uint32_t, ry - __builtin_bit_cast(float, ury & 0xFFFF0000u));
    // high halves of two words into one (v_perm_b32: bytes 2, 3 of the second
    // source, then bytes 2, 3 of the first)
    term[0][p] = (int)__builtin_amdgcn_perm(uy, ux, 0x07060302u);
    term[1][p] = (int)__builtin_amdgcn_perm(ury, urx, 0x07060302u);
    term[2][p] = (int)__builtin_amdgcn_perm(ly, lx, 0x07060302u);
  }
}

__device__ inline f32x16 mma32(i32x4 a, i32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                 0, 0);
}

// NK: 32-column tiles of k_in the instance holds (1, 2 or 4).
template <int NK>
__global__ __launch_bounds__(256, NK <= 2 ? 2 : 1) void gfused_kernel(GFusedArgs a) {
  static_assert(kWaves * 32 * 32 * 4 <= GDma::kBytes, "wave parts reuse the token staging ring");
  __shared__ __align__(16) uint8_t stage[GDma::kBytes];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // g_tile_dma's wave grid: wave (wr, wc) holds G^T rows (input features)
  // 64 wr .. 64 wr + 63 and columns (output features) 64 wc .. 64 wc + 63
  const int wr = wave >> 1, wc = wave & 1;
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
  const int na16 = (a.k_in + 15) >> 4, nb16 = (a.k_out + 15) >> 4;
  const int nkb_in = (a.d_in + 31) / 32, nkb_out = (a.d_out + 31) / 32;
  const rsrc_t rpin = make_rsrc(a.P_in, (uint32_t)((int64_t)nkb_in * na16 * kFragBytes));
  const rsrc_t rpout = make_rsrc(a.P_out, (uint32_t)((int64_t)nkb_out * nb16 * kFragBytes));

  // H[j][kt]: rows u0 + 64 wc + 32 j + (C layout), columns 32 kt + l % 32,
  // summed over this wave's half of every tile's input features
  f32x16 H[2][NK];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int kt = 0; kt < NK; ++kt)
#pragma unroll
      for (int x = 0; x < 16; ++x) H[j][kt][x] = 0.f;

  // G^T tiles: rows from the A blocks (d_in side), columns from the B blocks
  const GRows gr = g_rows(a_rows, b_rows, rows, a.d_in, a.d_out);
  for (int v0 = v_begin; v0 < v_end; v0 += kGFusedCols) {
    // P_in operands of this wave's input features, in flight during the
    // tile's token stages: k-block (v0 + 64 wr + 32 i) / 32, slice hx
    i32x4 pin[2][2][NK];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int hx = 0; hx < 2; ++hx)
#pragma unroll
        for (int kt = 0; kt < NK; ++kt)
          pin[i][hx][kt] = perm_operand(rpin, (v0 + 64 * wr + 32 * i) / 32, nkb_in, na16, kt, hx, lane);
    f32x16 acc[2][2];
    g_tile_dma(gr, rows, v0, u0, stage, acc);
    // acc[i][j]: G^T rows v0 + 64 wr + 32 i + (x-dependent), column
    // u0 + 64 wc + 32 j + l % 32
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int hx = 0; hx < 2; ++hx)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          i32x4 term[3];
          split_terms(acc[i][j], hx, term);
#pragma unroll
          for (int q = 0; q < 3; ++q)
#pragma unroll
            for (int kt = 0; kt < NK; ++kt) H[j][kt] = mma32(term[q], pin[i][hx][kt], H[j][kt]);
        }
  }

  // Psi_part[k][c] = sum over this wave's u of H[u][k] P_out[u][c], one
  // 32 x 32 tile (kt, ct) at a time; the four waves' tiles are added in LDS
  // in wave order.  H's C layout: lane l holds k = 32 kt + l % 32 and
  // u = 8 (x / 4) + 4 (l / 32) + x % 4 of block j, the A operand order.
  float* red = (float*)stage;
  const int ldp = nb16 * 16, kin_pad = na16 * 16;
  const int part_floats = kin_pad * ldp;
  float* dst =
      a.partials + ((int64_t)e_local * a.n_ublocks * a.n_vsplit * a.n_tchunks + blockIdx.x) * part_floats;
  const int nct = (a.k_out + 31) / 32;
#pragma unroll
  for (int kt = 0; kt < NK; ++kt) {
    if (32 * kt >= a.k_in) break;  // uniform
    for (int ct = 0; ct < nct; ++ct) {
      f32x16 d;
#pragma unroll
      for (int x = 0; x < 16; ++x) d[x] = 0.f;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int hx = 0; hx < 2; ++hx) {
          const i32x4 po = perm_operand(rpout, (u0 + 64 * wc + 32 * j) / 32, nkb_out, nb16, ct, hx, lane);
          i32x4 term[3];
          split_terms(H[j][kt], hx, term);
#pragma unroll
          for (int q = 0; q < 3; ++q) d = mma32(term[q], po, d);
        }
      // d's C layout: lane l, element x holds row k = 32 kt + 8 (x / 4) +
      // 4 (l / 32) + x % 4, column c = 32 ct + l % 32
#pragma unroll
      for (int x = 0; x < 16; ++x) red[(wave * 16 + x) * 64 + lane] = d[x];
      __syncthreads();
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const int idx = tid + 256 * m, x = idx >> 6, l = idx & 63;
        const float s = ((red[idx] + red[1024 + idx]) + red[2048 + idx]) + red[3072 + idx];
        const int k = 32 * kt + 8 * (x >> 2) + 4 * (l >> 5) + (x & 3), c = 32 * ct + (l & 31);
        if (k < kin_pad && c < ldp) dst[k * ldp + c] = s;
      }
      __syncthreads();
    }
  }
}

int gfused_tiles_in(int k_in) {
  const int na = (k_in + 15) / 16;
  return na <= 2 ? 2 : na <= 4 ? 4 : 8;
}

int gfused_wgs_per_cu(int k_in) { return gfused_tiles_in(k_in) <= 4 ? 2 : 1; }

hipError_t launch_gfused(const GFusedArgs& a, hipStream_t s) {
  if (a.ex_count <= 0) return hipSuccess;
  const int64_t n_vt = (a.d_in + kGFusedCols - 1) / kGFusedCols;
  if (a.n_ublocks <= 0 || a.n_tchunks <= 0 || a.tok_chunk <= 0 || a.n_vsplit <= 0 || a.vt_per_split <= 0 ||
      a.ex_count > 65535 || (int64_t)a.n_ublocks * a.n_vsplit * a.n_tchunks > INT32_MAX ||
      (int64_t)a.n_tchunks * a.tok_chunk < a.T || (a.tok_chunk % kTrTokens) != 0 ||
      (int64_t)a.n_vsplit * a.vt_per_split < n_vt || (int64_t)(a.n_vsplit - 1) * a.vt_per_split >= n_vt ||
      a.k_in < 1 || a.k_out < 1 || (a.k_in + 15) / 16 > kGFusedMaxTilesIn)
    return hipErrorInvalidValue;
  const dim3 grid(a.n_ublocks * a.n_vsplit * a.n_tchunks, a.ex_count);
  switch (gfused_tiles_in(a.k_in)) {
    case 2: hipLaunchKernelGGL(gfused_kernel<1>, grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL(gfused_kernel<2>, grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL(gfused_kernel<4>, grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace dattri
