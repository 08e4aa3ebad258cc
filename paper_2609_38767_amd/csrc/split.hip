// Factored route (Eq. (2), left side) in two stages, for captures with few
// examples or short sequences.
//
// The fused kernel's work items are (input group, example, token chunk); with
// few layers, examples or tokens there are too few of them, each streaming
// whole rows of width d_in + d_out, and most of the chip idles.  Here the
// projections themselves are split over the feature dimension:
//
//   stage 1  for every factor block X (a group's A, each member's B) viewed as
//            n*T token rows: out[s][row][:] = X[row, slab s] P[slab s, :],
//            float32, one workgroup per (block, 256-row block, slab; 128 rows at 8 tiles);
//   stage 2  per (layer, example, token chunk): Psi[c][r] = sum_t a~_t[c] g~_t[r]
//            with a~_t = sum_s outA[s][t] and g~_t = sum_s outB[s][t], over
//            the example's first T_i tokens (Eq. (4) allows T_i < T), written
//            into the layer block of phi, or as partial blocks summed by the
//            reduce kernel when an example's tokens span several chunks.
//
// Every sum runs in a fixed order, so results are bitwise reproducible.
#include "device_common.h"
#include "internal.h"
#include "project_rows.h"

namespace dattri {
using namespace dev;


template <int ELT, bool AL, int NT>
__global__ __launch_bounds__(256, 2) void split_project_kernel(const SplitItem* __restrict__ items,
                                                               const SplitOp* __restrict__ ops,
                                                               float* __restrict__ out) {
  constexpr int KR = 4 * (16 / ELT);  // rows of a packed k-block
  constexpr int RT = split_rt_of(NT), ROWS = split_rows_of(NT);
  static_assert(kWaves * RT * 16 == ROWS, "row block");
  constexpr int PD = 2;  // measured: deeper prefetch does not pay with 4 row tiles
  __shared__ __align__(16) uint8_t pan[2][kPanel][NT][kFragBytes];
  const SplitItem it = items[blockIdx.x];
  if (it.op < 0) return;  // padding item of the XCD-interleaved order
  const SplitOp& O = ops[it.op];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, m16 = lane & 15;
  const int row0 = it.row_block * ROWS;
  const int nrows = min(ROWS, O.rows - row0);
  const int col0 = it.slab * O.slab_cols;
  const int d = min(O.slab_cols, O.ld - col0);
  // descriptor over this row block, starting at the slab's first column
  const uint8_t* base = (const uint8_t*)O.X + ((int64_t)row0 * O.ld + col0) * ELT;
  const rsrc_t r = make_rsrc(base, (uint32_t)(((int64_t)nrows * O.ld - col0) * ELT));
  FragSrc<NT> P;
  P.nt = O.nt;
  const int kb0 = col0 / KR;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int tt = t < O.nt ? t : 0;
    P.stride[t] = (int64_t)O.ptile_nt[tt] * kFragBytes;
    P.base[t] = (const uint8_t*)O.ptile[tt] + (int64_t)O.ptile_local[tt] * kFragBytes + kb0 * P.stride[t];
  }
  f32x4 acc[RT][NT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[rt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int r_wave = wave * RT * 16;
  project_rows<ELT, AL, RT, NT, NT, PD>(r, r_wave, nrows, d, O.ld, P, acc, pan);

  const int ldo = O.nt * 16;
  float* dst = out + O.out_base + ((int64_t)it.slab * O.rows + row0) * ldo;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if (t < O.nt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = r_wave + rt * 16 + 4 * g + i;
          if (row < nrows) dst[(int64_t)row * ldo + t * 16 + m16] = acc[rt][t][i];
        }
      }
    }
}

// ---------------------------------------------------------------- stage 2
// Workgroup: one (layer, example, chunk of tok_chunk tokens).  Tokens are
// staged kCT at a time in LDS with the slab sums already taken (slabs summed in
// index order); the (up to 128 x 64) output block is register-blocked: thread
// (c_lane = tid / 8, r_lane = tid % 8) owns rows c_lane + 32 i and columns
// r_lane + 8 j, so each staged token costs 12 LDS reads for 32 FMAs.  A task
// with one chunk per example writes phi; otherwise each chunk writes a padded
// partial block that the reduce kernel sums in chunk order.
constexpr int kCT = 32;  // tokens staged in LDS per step
constexpr int kCI = 4;   // output rows per thread   (32 * 4 = 128 = 16 * kMaxGroupTiles)
constexpr int kCJ = 8;   // output columns per thread (8 * 8 = 64 = 16 * kMaxMemberBTiles)

__global__ __launch_bounds__(256) void split_contract_kernel(const ContractTask* __restrict__ tasks,
                                                             const float* __restrict__ proj,
                                                             float* __restrict__ partials,
                                                             void* __restrict__ phi, int phi_bf16,
                                                             int64_t ld_phi) {
  __shared__ float sa[kCT][16 * kMaxGroupTiles];
  __shared__ float sb[kCT][16 * kMaxMemberBTiles];
  const ContractTask t = tasks[blockIdx.z];
  const int chunk = blockIdx.x, ex = blockIdx.y, tid = threadIdx.x;
  if (chunk >= t.n_tchunks) return;
  int t_eff = t.T;
  if (t.lengths) t_eff = min(max(t.lengths[ex], 0), t.T);
  const int tok0 = chunk * t.tok_chunk, tok1 = min(t_eff, tok0 + t.tok_chunk);
  const int ki16 = (t.k_in + 15) & ~15, ko16 = (t.k_out + 15) & ~15;
  const int c_lane = tid >> 3, r_lane = tid & 7;
  float acc[kCI][kCJ];
#pragma unroll
  for (int i = 0; i < kCI; ++i)
#pragma unroll
    for (int j = 0; j < kCJ; ++j) acc[i][j] = 0.f;
  const int64_t row_ex = (int64_t)ex * t.T;
  for (int t0 = tok0; t0 < tok1; t0 += kCT) {
    const int nt = min(kCT, tok1 - t0);
    for (int idx = tid; idx < kCT * ki16; idx += 256) {
      const int tt = idx / ki16, c = idx - tt * ki16;
      float s = 0.f;
      if (tt < nt && c < t.k_in) {
        const float* p = proj + t.a_base + (row_ex + t0 + tt) * t.a_ld + t.a_col0 + c;
        for (int sl = 0; sl < t.a_slabs; ++sl) s += p[(int64_t)sl * t.rows * t.a_ld];
      }
      sa[tt][c] = s;
    }
    for (int idx = tid; idx < kCT * ko16; idx += 256) {
      const int tt = idx / ko16, r = idx - tt * ko16;
      float s = 0.f;
      if (tt < nt && r < t.k_out) {
        const float* p = proj + t.b_base + (row_ex + t0 + tt) * t.b_ld + r;
        for (int sl = 0; sl < t.b_slabs; ++sl) s += p[(int64_t)sl * t.rows * t.b_ld];
      }
      sb[tt][r] = s;
    }
    __syncthreads();
    if (c_lane < ki16) {
      for (int tt = 0; tt < nt; ++tt) {
        float av[kCI], bv[kCJ];
#pragma unroll
        for (int i = 0; i < kCI; ++i) av[i] = (c_lane + 32 * i < ki16) ? sa[tt][c_lane + 32 * i] : 0.f;
#pragma unroll
        for (int j = 0; j < kCJ; ++j) bv[j] = (r_lane + 8 * j < ko16) ? sb[tt][r_lane + 8 * j] : 0.f;
#pragma unroll
        for (int i = 0; i < kCI; ++i)
#pragma unroll
          for (int j = 0; j < kCJ; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
      }
    }
    __syncthreads();
  }
  if (t.n_tchunks == 1) {
#pragma unroll
    for (int i = 0; i < kCI; ++i)
#pragma unroll
      for (int j = 0; j < kCJ; ++j) {
        const int c = c_lane + 32 * i, r = r_lane + 8 * j;
        if (c < t.k_in && r < t.k_out) {
          const int64_t o = (int64_t)ex * ld_phi + t.phi_offset + (int64_t)c * t.k_out + r;
          if (phi_bf16)
            ((uint16_t*)phi)[o] = f32_to_bf16_bits(acc[i][j]);
          else
            ((float*)phi)[o] = acc[i][j];
        }
      }
  } else {
    float* dst = partials + t.partial_base + ((int64_t)ex * t.n_tchunks + chunk) * ki16 * ko16;
#pragma unroll
    for (int i = 0; i < kCI; ++i)
#pragma unroll
      for (int j = 0; j < kCJ; ++j) {
        const int c = c_lane + 32 * i, r = r_lane + 8 * j;
        if (c < ki16 && r < ko16) dst[c * ko16 + r] = acc[i][j];
      }
  }
}

// ---------------------------------------------------------------- launch
int split_nt_instance(int nt_req) { return nt_req <= 1 ? 1 : nt_req <= 2 ? 2 : nt_req <= 4 ? 4 : 8; }

template <int ELT, bool AL>
static hipError_t launch_split_al(int nt, const SplitItem* items, int n_items, const SplitOp* ops,
                                  float* out, hipStream_t s) {
  const dim3 grid((unsigned)n_items), block(256);
  switch (nt) {
    case 1: hipLaunchKernelGGL((split_project_kernel<ELT, AL, 1>), grid, block, 0, s, items, ops, out); break;
    case 2: hipLaunchKernelGGL((split_project_kernel<ELT, AL, 2>), grid, block, 0, s, items, ops, out); break;
    case 4: hipLaunchKernelGGL((split_project_kernel<ELT, AL, 4>), grid, block, 0, s, items, ops, out); break;
    case 8: hipLaunchKernelGGL((split_project_kernel<ELT, AL, 8>), grid, block, 0, s, items, ops, out); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_split_project(int elt_bytes, int aligned, int nt, const SplitItem* items,
                                int n_items, const SplitOp* ops, float* out, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  if (elt_bytes == 2)
    return aligned ? launch_split_al<2, true>(nt, items, n_items, ops, out, s)
                   : launch_split_al<2, false>(nt, items, n_items, ops, out, s);
  return aligned ? launch_split_al<4, true>(nt, items, n_items, ops, out, s)
                 : launch_split_al<4, false>(nt, items, n_items, ops, out, s);
}

hipError_t launch_split_contract(const ContractTask* tasks, int n_tasks, int n_examples,
                                 int max_tchunks, const float* proj, float* partials, void* phi,
                                 int phi_bf16, int64_t ld_phi, hipStream_t s) {
  if (n_tasks <= 0 || n_examples <= 0 || max_tchunks <= 0) return hipSuccess;
  if (n_examples > 65535 || n_tasks > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(split_contract_kernel, dim3(max_tchunks, n_examples, n_tasks), dim3(256), 0, s,
                     tasks, proj, partials, phi, phi_bf16, ld_phi);
  return hipGetLastError();
}

}  // namespace dattri
