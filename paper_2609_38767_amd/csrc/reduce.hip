// Deterministic reductions of float32 partial results.
//
// reduce_kernel: the factored and materialized kernels write partial Psi
// blocks (padded na*16 x nb*16, row-major) per (layer, example); their sum is
// the layer block of phi, element (c, r) at column phi_offset + c*k_out + r
// (the ordering of Eq. (2)).  A workgroup owns 64 outputs of one (example,
// task); its four waves each sum every fourth partial (parts w, w+4, ...) in
// index order, with loads issued four at a time, and wave 0 adds the four
// sums in wave order.  No float atomics: results are bitwise reproducible.
//
// slab_sum_kernel: the split form's stage 1 writes one projected copy of each
// token row per feature slab; this adds slabs 1.. into slab 0 in slab order.
#include "device_common.h"
#include "internal.h"

namespace dattri {
using namespace dev;

__global__ __launch_bounds__(256) void reduce_kernel(const ReduceTask* __restrict__ tasks,
                                                     const float* __restrict__ partials,
                                                     void* __restrict__ phi, int phi_bf16,
                                                     int64_t ld_phi) {
  __shared__ float red[4][64];
  const ReduceTask t = tasks[blockIdx.y];
  const int ex_local = blockIdx.x;
  const int64_t ex = (int64_t)t.ex_begin + ex_local;
  const float* base = partials + t.partial_base + (int64_t)ex_local * t.n_parts * t.part_floats;
  const int n_out = t.k_in * t.k_out;
  const int el = threadIdx.x & 63, pl = threadIdx.x >> 6;
  for (int e0 = blockIdx.z * 64; e0 < n_out; e0 += gridDim.z * 64) {  // uniform trip count
    const int e = e0 + el;
    float s = 0.f;
    if (e < n_out) {
      const int c = e / t.k_out, r = e - c * t.k_out;
      const float* p = base + c * t.ldp + r;
      const int64_t step = (int64_t)t.part_floats;
      int q = pl;
      for (; q + 12 < t.n_parts; q += 16) {
        const float v0 = p[q * step], v1 = p[(q + 4) * step], v2 = p[(q + 8) * step],
                    v3 = p[(q + 12) * step];
        s = (((s + v0) + v1) + v2) + v3;
      }
      for (; q < t.n_parts; q += 4) s += p[q * step];
    }
    red[pl][el] = s;
    __syncthreads();
    if (pl == 0 && e < n_out) {
      const float v = ((red[0][el] + red[1][el]) + red[2][el]) + red[3][el];
      const int64_t o = ex * ld_phi + t.phi_offset + e;
      if (phi_bf16)
        ((uint16_t*)phi)[o] = f32_to_bf16_bits(v);
      else
        ((float*)phi)[o] = v;
    }
    __syncthreads();
  }
}

hipError_t launch_reduce(const ReduceTask* tasks, int n_tasks, int n_examples, int max_out,
                         const float* partials, void* phi, int phi_bf16, int64_t ld_phi,
                         hipStream_t s) {
  if (n_tasks <= 0 || n_examples <= 0 || max_out <= 0) return hipSuccess;
  if (n_tasks > 65535) return hipErrorInvalidValue;
  const int zb = (max_out + 63) / 64;
  const int z = zb < 64 ? zb : 64;
  hipLaunchKernelGGL(reduce_kernel, dim3(n_examples, n_tasks, z), dim3(256), 0, s, tasks, partials,
                     phi, phi_bf16, ld_phi);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void slab_sum_kernel(const SlabSumTask* __restrict__ tasks,
                                                       float* __restrict__ out) {
  const SlabSumTask t = tasks[blockIdx.y];
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;  // float4 index inside a slab
  if (i >= t.n4) return;
  f32x4* p = (f32x4*)(out + t.base) + i;
  f32x4 s = p[0];
  int sl = 1;
  for (; sl + 3 < t.n_slabs; sl += 4) {
    const f32x4 v0 = p[sl * t.stride4], v1 = p[(sl + 1) * t.stride4], v2 = p[(sl + 2) * t.stride4],
                v3 = p[(sl + 3) * t.stride4];
    s = (((s + v0) + v1) + v2) + v3;
  }
  for (; sl < t.n_slabs; ++sl) s += p[sl * t.stride4];
  p[0] = s;
}

hipError_t launch_slab_sum(const SlabSumTask* tasks, int n_tasks, int64_t max_n4, float* out,
                           hipStream_t s) {
  if (n_tasks <= 0 || max_n4 <= 0) return hipSuccess;
  if (n_tasks > 65535 || (max_n4 + 255) / 256 > INT32_MAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(slab_sum_kernel, dim3((unsigned)((max_n4 + 255) / 256), n_tasks), dim3(256), 0, s,
                     tasks, out);
  return hipGetLastError();
}

}  // namespace dattri
