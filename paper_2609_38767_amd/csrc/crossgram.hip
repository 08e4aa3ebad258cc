// Cross-Gram matrices of unprojected per-example weight gradients (Sec. 3.2
// "Factorized inner product", Eq. (4); App. A.4 routing table).
//
// Factorized route (ghost_kernel).  Each example's token rows are padded to
// Tp = T rounded up to 16, and the n1 (resp. n2) examples of a batch are laid
// end to end, giving a flattened token axis of n1*Tp1 rows on one side and
// n2*Tp2 on the other.  For a 128 x 128 tile of that token-pair space the
// kernel forms the input Gram A A'^T (contraction over d_in) and the output-
// gradient Gram B B'^T (contraction over d_out) in registers with the same
// MFMA C layout, multiplies them element by element and sums each 16 x 16 block
// (every block lies inside one example pair because Tp is a multiple of 16;
// padding rows and tokens past an example's length read zero).  Block sums go
// to a partial array; ghost_reduce_kernel adds, for each example pair, the
// blocks of its segment over all layers in a fixed order (deterministic).
//
// Materialized route.  DW = B^T A is built per example by gradient_kernel
// (float32, staged in the workspace); gdot_kernel takes Frobenius products of
// 16 x 16 blocks of example pairs over chunks of the flattened DW with float32
// MFMA, and kacc_kernel sums the chunks in a fixed pairwise order into K.
#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

// --------------------------------------------------------------- factorized
constexpr int kGhRows = 128;  // tile rows and columns (flattened tokens)

// 16-byte chunk `col`..`col`+EPL-1 of global row `grow` of a [rows, d] block
// (zero when the row is invalid or the columns fall past d).
template <int ELT>
__device__ inline i32x4 ghost_chunk(const uint8_t* base, int64_t grow, bool valid, int col, int d,
                                    bool aligned) {
  constexpr int EPL = 16 / ELT;
  i32x4 v = {0, 0, 0, 0};
  if (!valid || col >= d) return v;
  const uint8_t* p = base + (grow * d + col) * ELT;
  if (aligned && col + EPL <= d) return *(const i32x4*)p;
  uint32_t w[EPL];
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    w[j] = 0;
    if (col + j < d) w[j] = ELT == 2 ? (uint32_t)((const uint16_t*)p)[j] : ((const uint32_t*)p)[j];
  }
  if (ELT == 2) {
    v[0] = (int)(w[0] | (w[1] << 16));
    v[1] = (int)(w[2] | (w[3] << 16));
    v[2] = (int)(w[4] | (w[5] << 16));
    v[3] = (int)(w[6] | (w[7] << 16));
  } else {
    v[0] = (int)w[0]; v[1] = (int)w[1]; v[2] = (int)w[2]; v[3] = (int)w[3];
  }
  return v;
}

// Direct-load form of a tile's two Grams (bf16 entries with E.dma set):
// stages of 32 features (64 bytes per token row, one 16x16x32 K step) of both
// sides go straight from memory to LDS (buffer_load ... lds; one load moves
// 1 KiB = 16 rows, each wave issues 2 per side and stage) through a ring of 4
// stages, 3 in flight, over d_in's stages and then d_out's in one stream.
// The 16-byte chunk c of local row r sits at c XOR gswz16(r), so the 16-byte
// fragment reads (8 lanes served together, 8 rows x 16 bytes) fall in 8
// distinct 16-byte bank groups: measured 0 bank-conflict cycles, against 3.7
// per read unswizzled (a swizzle that also spread 16-lane groups measured the
// same as none, so the hardware serves 8 lanes of a 16-byte read at a time).
// Waits count direct
// loads as in the weight-gradient tile (gtile.h): stage k has landed when at
// most 4 x min(2, stages after k) of the wave's loads are in flight; the
// fragment reads are inline assembly tied to hand lgkmcnt waits, so the
// compiler does not drain the ring before them.
constexpr int kGhDmaStage = 2 * kGhRows * 64;  // both sides, 16 KiB
__device__ constexpr int gswz16(int r) { return (r >> 1) & 3; }

__device__ inline void ghost_tile_dma(const GhostEntry& E, const GhostTile& tl, uint8_t* lds,
                                      f32x4 (&acc)[2][4][4]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, m16 = lane & 15, wm = wave >> 1, wn = wave & 1;
  auto stage_barrier = [] { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };

  // this lane's rows of the direct loads: local rows 16 (2 wave + t) + lane / 4
  // of each side, physical chunk lane % 4; row index relative to the first
  // example of the tile's range (descriptors start there, so 32-bit offsets
  // reach every row of the tile)
  int rel[2][2], cl[2];
  bool ok[2][2];
  rsrc_t rA[2], rB[2];
#pragma unroll
  for (int side = 0; side < 2; ++side) {
    const int R0 = (side ? tl.ct : tl.rt) * kGhRows;
    const int Tp = side ? E.Tp2 : E.Tp1, T = side ? E.T2 : E.T1, n = side ? E.n2 : E.n1;
    const int32_t* len = side ? E.len2 : E.len1;
    const int e0 = R0 / Tp;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int row = 16 * (2 * wave + t) + (lane >> 2);
      const int R = R0 + row, e = R / Tp, tt = R - e * Tp;
      int t_eff = T;
      if (e < n && len) t_eff = min(max(len[e], 0), T);
      ok[side][t] = e < n && tt < t_eff;
      rel[side][t] = (e - e0) * T + tt;
      if (side == 0) cl[t] = (lane & 3) ^ gswz16(row);
    }
    const uint8_t* a = (const uint8_t*)(side ? E.A2 : E.A1);
    const uint8_t* b = (const uint8_t*)(side ? E.B2 : E.B1);
    const int64_t ra = (int64_t)(n - e0) * T * E.d_in * 2, rb = (int64_t)(n - e0) * T * E.d_out * 2;
    rA[side] = make_rsrc(a + (int64_t)e0 * T * E.d_in * 2, (uint32_t)min<int64_t>(ra, kOOB));
    rB[side] = make_rsrc(b + (int64_t)e0 * T * E.d_out * 2, (uint32_t)min<int64_t>(rb, kOOB));
  }
  const int nk0 = (E.d_in + 31) / 32, nk1 = (E.d_out + 31) / 32, ns = nk0 + nk1;
  auto issue = [&](int st) {
    const bool p = st >= nk0;
    const int kk = p ? st - nk0 : st, d = p ? E.d_out : E.d_in;
    uint8_t* sb = lds + (st & 3) * kGhDmaStage;
#pragma unroll
    for (int side = 0; side < 2; ++side) {
      const rsrc_t r = p ? rB[side] : rA[side];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int col = kk * 32 + cl[t] * 8;
        const uint32_t off = ok[side][t] && col < d ? (uint32_t)(((int64_t)rel[side][t] * d + col) * 2) : kOOB;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(r, DATTRI_LDS_PTR(sb + side * kGhRows * 64 + (2 * wave + t) * 1024),
                                                 16, off, 0, 0, 0);
      }
    }
  };

  // fragment reads: A operand rows wm 64 + 16 i + m16 of side 0, B operand
  // rows wn 64 + 16 j + m16 of side 1, logical chunk g (features 8 g .. 8 g + 7)
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)lds;
  uint32_t ao[4], bo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ra = wm * 64 + 16 * i + m16, rb = wn * 64 + 16 * i + m16;
    ao[i] = lds0 + (uint32_t)(ra * 64 + ((g ^ gswz16(ra)) << 4));
    bo[i] = lds0 + (uint32_t)(kGhRows * 64 + rb * 64 + ((g ^ gswz16(rb)) << 4));
  }
  auto rd = [](uint32_t addr) {
    i32x4 x;
    asm volatile("ds_read_b128 %0, %1" : "=v"(x) : "v"(addr));
    return x;
  };
  // one stage: the 4 B fragments, then the A fragments one at a time, each
  // row of 4 MFMA starting once its A fragment has landed (LDS returns in order)
  auto stage = [&](uint32_t so, f32x4 (&c)[4][4]) {
    i32x4 bf[4], af[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) bf[j] = rd(bo[j] + so);
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = rd(ao[i] + so);
    asm volatile("s_waitcnt lgkmcnt(3)" : "+v"(bf[0]), "+v"(bf[1]), "+v"(bf[2]), "+v"(bf[3]), "+v"(af[0]));
#pragma unroll
    for (int j = 0; j < 4; ++j) c[0][j] = frag_mma<2>(af[0], bf[j], c[0][j]);
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt lgkmcnt(2)" : "+v"(af[1]));
#pragma unroll
    for (int j = 0; j < 4; ++j) c[1][j] = frag_mma<2>(af[1], bf[j], c[1][j]);
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt lgkmcnt(1)" : "+v"(af[2]));
#pragma unroll
    for (int j = 0; j < 4; ++j) c[2][j] = frag_mma<2>(af[2], bf[j], c[2][j]);
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(af[3]));
#pragma unroll
    for (int j = 0; j < 4; ++j) c[3][j] = frag_mma<2>(af[3], bf[j], c[3][j]);
  };
  auto wait_for = [&](int k) {
    const int ahead = ns - 1 - k;
    if (ahead >= 2)
      wait_vmcnt_dma<8>();
    else if (ahead == 1)
      wait_vmcnt_dma<4>();
    else
      wait_vmcnt_dma<0>();
    stage_barrier();
    if (k + 3 < ns) issue(k + 3);
  };
#pragma unroll
  for (int p = 0; p < 3; ++p)
    if (p < ns) issue(p);
  for (int k = 0; k < nk0; ++k) {
    wait_for(k);
    stage((uint32_t)((k & 3) * kGhDmaStage), acc[0]);
  }
  for (int k = nk0; k < ns; ++k) {
    wait_for(k);
    stage((uint32_t)((k & 3) * kGhDmaStage), acc[1]);
  }
  stage_barrier();
}

// Register-staged form (float32 entries, unaligned rows): stages of 128 bytes
// of features per row are double-buffered in LDS (rows XOR-swizzled by
// 16-byte chunk) and the next stage is prefetched into registers while the
// current one is multiplied.  smem: 2 x 2 x 128 x 128 bytes.
template <int ELT>
__device__ inline void ghost_tile_reg(const GhostEntry& E, const GhostTile& tl, uint8_t (*smem)[2][kGhRows * 128],
                                      f32x4 (&acc)[2][4][4]) {
  constexpr int EPL = 16 / ELT;
  constexpr int BK = 128 / ELT;  // features per stage
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, m16 = lane & 15, wm = wave >> 1, wn = wave & 1;
  const bool aligned = E.aligned != 0;

  // rows handled by this thread's 4 load chunks (row = c >> 3 of c = tid + 256 i)
  int64_t grow[2][4];
  bool valid[2][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = (tid + 256 * i) >> 3;
#pragma unroll
    for (int side = 0; side < 2; ++side) {
      const int R = (side ? tl.ct : tl.rt) * kGhRows + row;
      const int Tp = side ? E.Tp2 : E.Tp1, T = side ? E.T2 : E.T1, n = side ? E.n2 : E.n1;
      const int32_t* len = side ? E.len2 : E.len1;
      const int e = R / Tp, t = R - e * Tp;
      int t_eff = T;
      if (e < n && len) t_eff = min(max(len[e], 0), T);
      valid[side][i] = e < n && t < t_eff;
      grow[side][i] = (int64_t)e * T + t;
    }
  }

#pragma unroll
  for (int p = 0; p < 2; ++p) {  // p = 0: input Gram over d_in; 1: output-gradient Gram over d_out
    const uint8_t* b1 = (const uint8_t*)(p ? E.B1 : E.A1);
    const uint8_t* b2 = (const uint8_t*)(p ? E.B2 : E.A2);
    const int d = p ? E.d_out : E.d_in;
    const int nk = (d + BK - 1) / BK;
    i32x4 r1[4], r2[4];
    auto gload = [&](int kk) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int col = kk * BK + ((tid + 256 * i) & 7) * EPL;
        r1[i] = ghost_chunk<ELT>(b1, grow[0][i], valid[0][i], col, d, aligned);
        r2[i] = ghost_chunk<ELT>(b2, grow[1][i], valid[1][i], col, d, aligned);
      }
    };
    auto swrite = [&](int st) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = tid + 256 * i, row = c >> 3, ch = c & 7;
        const int off = row * 128 + ((ch ^ (row & 7)) << 4);
        *(i32x4*)(smem[st][0] + off) = r1[i];
        *(i32x4*)(smem[st][1] + off) = r2[i];
      }
    };
    gload(0);
    swrite(0);
    __syncthreads();
    for (int kk = 0; kk < nk; ++kk) {
      const int st = kk & 1;
      if (kk + 1 < nk) gload(kk + 1);
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        i32x4 af[4], bf[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = wm * 64 + i * 16 + m16, ch = s * 4 + g;
          af[i] = *(const i32x4*)(smem[st][0] + row * 128 + ((ch ^ (row & 7)) << 4));
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int row = wn * 64 + j * 16 + m16, ch = s * 4 + g;
          bf[j] = *(const i32x4*)(smem[st][1] + row * 128 + ((ch ^ (row & 7)) << 4));
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[p][i][j] = frag_mma<ELT>(af[i], bf[j], acc[p][i][j]);
      }
      if (kk + 1 < nk) swrite(st ^ 1);
      __syncthreads();
    }
  }
}

// Workgroup: one 128 x 128 tile, 4 waves in a 2 x 2 grid of 64 x 64 (4 x 4
// blocks of 16 x 16 per Gram); entries with E.dma take the direct-load form.
template <int ELT>
__global__ __launch_bounds__(256, 2) void ghost_kernel(const GhostEntry* __restrict__ entries,
                                                       const GhostTile* __restrict__ tiles,
                                                       float* __restrict__ parts) {
  static_assert(4 * kGhDmaStage == 2 * 2 * kGhRows * 128, "one LDS block for both forms");
  __shared__ __align__(16) uint8_t smem[2][2][kGhRows * 128];  // [stage][row side, col side]
  const GhostTile tl = tiles[blockIdx.x];
  const GhostEntry E = entries[tl.entry];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  f32x4 acc[2][4][4];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[p][i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (ELT == 2 && E.dma)  // uniform
    ghost_tile_dma(E, tl, &smem[0][0][0], acc);
  else
    ghost_tile_reg<ELT>(E, tl, smem, acc);

  // Hadamard product of the two Grams, summed per 16 x 16 block (lanes hold
  // the same (row, column) of both accumulators)
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float v = 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) v += acc[0][i][j][r] * acc[1][i][j][r];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
      const int br = tl.rt * (kGhRows / 16) + wm * 4 + i;
      const int bc = tl.ct * (kGhRows / 16) + wn * 4 + j;
      if (lane == 0 && br < E.nbr && bc < E.nbc) parts[E.part_off + (int64_t)br * E.nbc + bc] = v;
    }
}

// K[I][J] (diag: out[I]) = sum over entries, in order, of the block sums of
// segment (i, j) = (I - out0, J) (diag: (I - out0, I - out0)) of every entry
// holding that pair: blocks [i*Tp1/16, (i+1)*Tp1/16) x [j*Tp2/16, ...).  One
// workgroup per output; thread t sums blocks t, t+256, ... of each entry in
// order, then a fixed tree.
__global__ __launch_bounds__(256) void ghost_reduce_kernel(const GhostEntry* __restrict__ entries,
                                                           int n_entries, const float* __restrict__ parts,
                                                           int n_cols, float* __restrict__ K, int64_t ld,
                                                           int diag, int accumulate) {
  __shared__ float red[256];
  const int cell = blockIdx.x;
  const int I = diag ? cell : cell / n_cols, J = diag ? cell : cell % n_cols;
  float s = 0.f;
  for (int e = 0; e < n_entries; ++e) {
    const GhostEntry& E = entries[e];
    const int i = I - E.out0, j = diag ? i : J;
    if (i < 0 || i >= E.n1 || j < 0 || j >= E.n2) continue;
    const int rb = E.Tp1 / 16, cb = E.Tp2 / 16;
    const int nblk = rb * cb;
    for (int b = threadIdx.x; b < nblk; b += 256) {
      const int br = i * rb + b / cb, bc = j * cb + b % cb;
      s += parts[E.part_off + (int64_t)br * E.nbc + bc];
    }
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    float* dst = diag ? &K[I] : &K[(int64_t)I * ld + J];
    *dst = accumulate ? *dst + red[0] : red[0];
  }
}

hipError_t launch_ghost(int elt, const GhostEntry* entries, const GhostTile* tiles, int n_tiles,
                        float* parts, hipStream_t s) {
  if (n_tiles <= 0) return hipSuccess;
  if (elt == 2)
    hipLaunchKernelGGL(ghost_kernel<2>, dim3(n_tiles), dim3(256), 0, s, entries, tiles, parts);
  else
    hipLaunchKernelGGL(ghost_kernel<4>, dim3(n_tiles), dim3(256), 0, s, entries, tiles, parts);
  return hipGetLastError();
}

hipError_t launch_ghost_reduce(const GhostEntry* entries, int n_entries, const float* parts,
                               int n_rows, int n_cols, float* K, int64_t ld, int diag, int accumulate,
                               hipStream_t s) {
  const int cells = diag ? n_rows : n_rows * n_cols;
  if (cells <= 0) return hipSuccess;
  hipLaunchKernelGGL(ghost_reduce_kernel, dim3(cells), dim3(256), 0, s, entries, n_entries, parts, n_cols,
                     K, ld, diag, accumulate);
  return hipGetLastError();
}

// ------------------------------------------------------------- materialized
// parts[c][i][j] = sum over chunk c of the flattened DW (D floats) of
// G1[i] * G2[j], for a 16 x 16 block of example pairs (grid y, z).  Each of the
// 4 waves takes a quarter of the chunk; 16x16x4 float32 MFMAs with A = rows of
// G1, B = rows of G2 (lane (g, m) holds 4 consecutive floats of row m at
// offset 4g of each 16-float step); the waves' results are summed in LDS in
// wave order.  diag: only pairs (i, i) are wanted (G2 == G1, grid z = 1, the
// block's columns are its rows) and parts[c][i] is written.
__global__ __launch_bounds__(256) void gdot_kernel(const float* __restrict__ G1, int n1,
                                                   const float* __restrict__ G2, int n2, int64_t D,
                                                   int64_t chunk, int diag, float* __restrict__ parts) {
  __shared__ f32x4 red[4][64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, m16 = lane & 15;
  const int c = blockIdx.x, i0 = blockIdx.y * 16, j0 = diag ? i0 : blockIdx.z * 16;
  const int64_t q = chunk / 4;
  const int64_t k_begin = c * chunk + wave * q;
  const int64_t k_end = min(D, k_begin + q);
  const int ia = i0 + m16, jb = j0 + m16;
  const float* ra = G1 + (int64_t)min(ia, n1 - 1) * D;
  const float* rb = G2 + (int64_t)min(jb, n2 - 1) * D;
  const bool va = ia < n1, vb = jb < n2;
  const bool vec = (D & 3) == 0;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int64_t k = k_begin; k < k_end; k += 16) {
    const int64_t kk = k + 4 * g;
    f32x4 a = {0.f, 0.f, 0.f, 0.f}, b = {0.f, 0.f, 0.f, 0.f};
    if (vec && kk + 4 <= k_end) {
      if (va) a = *(const f32x4*)(ra + kk);
      if (vb) b = *(const f32x4*)(rb + kk);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (kk + e < k_end) {
          if (va) a[e] = ra[kk + e];
          if (vb) b[e] = rb[kk + e];
        }
    }
    acc = mfma_f32_4(a[0], b[0], acc);
    acc = mfma_f32_4(a[1], b[1], acc);
    acc = mfma_f32_4(a[2], b[2], acc);
    acc = mfma_f32_4(a[3], b[3], acc);
  }
  red[wave][lane] = acc;
  __syncthreads();
  if (wave == 0) {
    f32x4 v = red[0][lane];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const f32x4 u = red[w][lane];
      v[0] += u[0]; v[1] += u[1]; v[2] += u[2]; v[3] += u[3];
    }
    // C layout: lane (g, m) holds rows 4g + r (pairs' i), column m (pairs' j)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = i0 + 4 * g + r, j = j0 + m16;
      if (diag) {
        if (i == j && i < n1) parts[(int64_t)c * n1 + i] = v[r];
      } else if (i < n1 && j < n2) {
        parts[((int64_t)c * n1 + i) * n2 + j] = v[r];
      }
    }
  }
}

// K[r0 + i][c0 + j] (+)= sum over chunks of parts[c][i][j]: per-thread sums of
// chunks t, t+256, ..., then a fixed tree.  diag: out[r0 + i] (+)= the sum of
// parts[c][i].
__global__ __launch_bounds__(256) void kacc_kernel(const float* __restrict__ parts, int nchunks, int n1,
                                                   int n2, float* __restrict__ K, int64_t ld, int r0,
                                                   int c0, int diag, int accumulate) {
  __shared__ float red[256];
  const int cell = blockIdx.x;
  const int i = diag ? cell : cell / n2, j = diag ? cell : cell % n2;
  float s = 0.f;
  for (int c = threadIdx.x; c < nchunks; c += 256)
    s += diag ? parts[(int64_t)c * n1 + i] : parts[((int64_t)c * n1 + i) * n2 + j];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    float* dst = diag ? &K[r0 + i] : &K[(int64_t)(r0 + i) * ld + c0 + j];
    *dst = accumulate ? *dst + red[0] : red[0];
  }
}

__global__ __launch_bounds__(256) void fill_rows_kernel(float* __restrict__ K, int rows, int cols,
                                                        int64_t ld) {
  const int64_t n = (int64_t)rows * cols;
  for (int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x; x < n; x += (int64_t)gridDim.x * 256)
    K[(x / cols) * ld + x % cols] = 0.f;
}

hipError_t launch_gdot(const float* G1, int n1, const float* G2, int n2, int64_t D, int64_t chunk,
                       int diag, float* parts, hipStream_t s) {
  const int64_t nchunks = (D + chunk - 1) / chunk;
  if (nchunks <= 0 || n1 <= 0 || n2 <= 0) return hipSuccess;
  if (chunk % 64 != 0) return hipErrorInvalidValue;  // 4 waves x 16-float steps
  hipLaunchKernelGGL(gdot_kernel, dim3((unsigned)nchunks, (n1 + 15) / 16, diag ? 1 : (n2 + 15) / 16), dim3(256),
                     0, s, G1, n1, G2, n2, D, chunk, diag, parts);
  return hipGetLastError();
}

hipError_t launch_kacc(const float* parts, int nchunks, int n1, int n2, float* K, int64_t ld, int r0,
                       int c0, int diag, int accumulate, hipStream_t s) {
  const int cells = diag ? n1 : n1 * n2;
  if (cells <= 0) return hipSuccess;
  hipLaunchKernelGGL(kacc_kernel, dim3(cells), dim3(256), 0, s, parts, nchunks, n1, n2, K, ld, r0, c0, diag,
                     accumulate);
  return hipGetLastError();
}

hipError_t launch_fill_rows(float* K, int rows, int cols, int64_t ld, hipStream_t s) {
  const int64_t n = (int64_t)rows * cols;
  if (n <= 0) return hipSuccess;
  const int blocks = (int)std::min<int64_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(fill_rows_kernel, dim3(blocks), dim3(256), 0, s, K, rows, cols, ld);
  return hipGetLastError();
}

}  // namespace dattri
