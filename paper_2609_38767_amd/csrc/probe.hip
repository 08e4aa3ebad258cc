// Measurement probes: the denominators the rooflines are also reported
// against, measured on the device itself.
//
// probe_read_kernel streams a buffer once with non-temporal 16-byte loads
// (grid-stride, four loads in flight per lane per step) and folds what it read
// into one word per lane, so no load can be dropped: the achievable rate of a
// pure HBM read stream.
//
// probe_mfma_kernel issues bf16 32x32x16 MFMAs back to back on eight
// independent accumulators per wave, each with its own pseudo-random operands
// held in registers, and no memory traffic in the loop: the achievable dense
// bf16 matrix rate with data-like operands, including whatever clock the chip
// holds under that load.
#include <stddef.h>
#include <stdint.h>

#include "api_common.h"
#include "device_common.h"

namespace dattri {
using namespace dev;

constexpr int kProbeChains = 8;  // independent accumulators per wave

__global__ __launch_bounds__(256) void probe_read_kernel(const i32x4* __restrict__ p, int64_t n16,
                                                         int32_t* __restrict__ sink) {
  const int64_t step = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  i32x4 a = {0, 0, 0, 0};
  for (; i + 3 * step < n16; i += 4 * step) {
    const i32x4 v0 = __builtin_nontemporal_load(p + i);
    const i32x4 v1 = __builtin_nontemporal_load(p + i + step);
    const i32x4 v2 = __builtin_nontemporal_load(p + i + 2 * step);
    const i32x4 v3 = __builtin_nontemporal_load(p + i + 3 * step);
    a ^= v0 ^ v1 ^ v2 ^ v3;
  }
  for (; i < n16; i += step) a ^= __builtin_nontemporal_load(p + i);
  sink[(int64_t)blockIdx.x * 256 + threadIdx.x] = a.x ^ a.y ^ a.z ^ a.w;
}

// Operand bits of the MFMA probe: a bf16 with a pseudo-random sign and 7-bit
// mantissa and an exponent in [-2, 1], from a 32-bit hash of (lane, element,
// chain, side), so the multipliers see data-like switching.
__host__ __device__ inline uint16_t probe_operand_bits(uint32_t lane, uint32_t e, uint32_t c, uint32_t side) {
  uint32_t h = lane * 0x9E3779B1u + e * 0x85EBCA77u + c * 0xC2B2AE3Du + side * 0x27D4EB2Fu + 0x165667B1u;
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  h ^= h >> 12;
  const uint32_t sign = (h >> 31) & 1u, expo = 125u + ((h >> 8) & 3u), mant = h & 0x7Fu;
  return (uint16_t)((sign << 15) | (expo << 7) | mant);
}

__global__ __launch_bounds__(256) void probe_mfma_kernel(int iters, float* __restrict__ sink) {
  const int tid = threadIdx.x, lane = tid & 63;
  // each chain has its own operands, so consecutive MFMAs switch inputs
  bf16x8 a[kProbeChains], b[kProbeChains];
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      a[c][e] = __builtin_bit_cast(__bf16, probe_operand_bits(lane, e, c, 0));
      b[c][e] = __builtin_bit_cast(__bf16, probe_operand_bits(lane, e, c, 1));
    }
  f32x16 acc[kProbeChains];
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[c][v] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kProbeChains; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[c], b[c], acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[c][v];
  sink[(int64_t)blockIdx.x * 256 + tid] = s;
}

}  // namespace dattri

using namespace dattri;

extern "C" dattri_status dattri_probe_read(const void* buf, size_t bytes, int32_t* sink, int32_t workgroups,
                                           void* stream) {
  reset_error();
  if (!buf || !sink) return fail(DATTRI_E_INVALID_ARG, "buf and sink must be non-NULL");
  if ((uintptr_t)buf % 16 != 0 || bytes == 0 || bytes % 16 != 0)
    return fail(DATTRI_E_INVALID_ARG, "buf must be 16-byte aligned and bytes a positive multiple of 16");
  if (workgroups < 1 || workgroups > (1 << 20))
    return fail(DATTRI_E_INVALID_ARG, "workgroups must be in [1, 2^20] (got %d)", workgroups);
  hipLaunchKernelGGL(probe_read_kernel, dim3((unsigned)workgroups), dim3(256), 0, (hipStream_t)stream,
                     (const i32x4*)buf, (int64_t)(bytes / 16), sink);
  HIP_TRY(hipGetLastError());
  return DATTRI_OK;
}

extern "C" dattri_status dattri_probe_mfma(float* sink, int32_t workgroups, int32_t iters, double* flops,
                                           void* stream) {
  reset_error();
  if (!sink || !flops) return fail(DATTRI_E_INVALID_ARG, "sink and flops must be non-NULL");
  if (workgroups < 1 || workgroups > (1 << 20))
    return fail(DATTRI_E_INVALID_ARG, "workgroups must be in [1, 2^20] (got %d)", workgroups);
  if (iters < 1) return fail(DATTRI_E_INVALID_ARG, "iters must be >= 1 (got %d)", iters);
  // 4 waves per workgroup, kProbeChains MFMAs of 2 * 32 * 32 * 16 FLOP per iteration
  *flops = (double)workgroups * 4.0 * iters * kProbeChains * (2.0 * 32 * 32 * 16);
  hipLaunchKernelGGL(probe_mfma_kernel, dim3((unsigned)workgroups), dim3(256), 0, (hipStream_t)stream, iters,
                     sink);
  HIP_TRY(hipGetLastError());
  return DATTRI_OK;
}
