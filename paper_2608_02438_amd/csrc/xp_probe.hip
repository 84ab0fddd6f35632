// Measured peaks of the two resources the path is bound by, so that a kernel's
// roofline fraction can be stated against what this GPU delivers as well as
// against its published figures:
//   - HBM read bandwidth: each workgroup streams a contiguous range of a
//     buffer with 16-byte non-temporal loads, reduced to a 32-bit checksum so
//     that nothing is elided;
//   - bf16 matrix throughput: independent chains of v_mfma_f32_32x32x16_bf16
//     on register operands supplied by the caller (random operands draw more
//     power than constant ones, and the rate follows).
// Neither is part of the refine + verify path.
#include "xp_internal.h"

namespace xp {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 8;     // independent loads in flight per thread
constexpr int kProbeChains = 8;     // independent accumulators per wave

// Workgroup g streams the contiguous 16-byte units [g n16 / G, (g + 1) n16 / G),
// kProbeUnroll x 4 KB per iteration (each wave instruction reads 1 KB).
__global__ __launch_bounds__(kProbeThreads) void k_probe_read(const u32x4* __restrict__ buf,
                                                              size_t n16, uint32_t* __restrict__ out) {
  const size_t lo = n16 * blockIdx.x / gridDim.x, hi = n16 * (blockIdx.x + 1) / gridDim.x;
  constexpr int kStep = kProbeThreads * kProbeUnroll;
  size_t i = lo + threadIdx.x;
  uint32_t s = 0;
  for (; i + (kProbeUnroll - 1) * kProbeThreads < hi; i += kStep) {
    u32x4 v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) v[u] = ld16_nt(buf + i + u * kProbeThreads);
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) s += (v[u].x + v[u].y) + (v[u].z + v[u].w);
  }
  for (; i < hi; i += kProbeThreads) {
    const u32x4 v = ld16_nt(buf + i);
    s += (v.x + v.y) + (v.z + v.w);
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, kWave);
  if ((threadIdx.x & 63) == 0) atomicAdd(out, s);
}

__global__ __launch_bounds__(kProbeThreads) __attribute__((amdgpu_waves_per_eu(2))) void k_probe_mfma(const u32x4* __restrict__ ops,
                                                              int iters, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  u32x4 a[kProbeChains], b[kProbeChains];
#pragma unroll
  for (int j = 0; j < kProbeChains; ++j) {
    a[j] = ops[(j * 64 + lane) * 2];
    b[j] = ops[(j * 64 + lane) * 2 + 1];
  }
  floatx16 acc[kProbeChains];
#pragma unroll
  for (int j = 0; j < kProbeChains; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < kProbeChains; ++j)
      acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[j]),
                                                       __builtin_bit_cast(bf16x8, b[j]), acc[j], 0,
                                                       0, 0);
  }
#pragma unroll
  for (int j = 1; j < kProbeChains; ++j) acc[0] += acc[j];
  const floatx16 t = acc[0];
  const size_t gw = (size_t)blockIdx.x * (kProbeThreads / 64) + (threadIdx.x >> 6);
  float* o = out + (gw * 64 + lane) * 16;
#pragma unroll
  for (int e = 0; e < 16; e += 4)
    *reinterpret_cast<float4*>(o + e) = make_float4(t[e], t[e + 1], t[e + 2], t[e + 3]);
}

}  // namespace xp

using namespace xp;

extern "C" xp_status xp_probe_hbm_read(const void* buf, size_t bytes, uint32_t* out_sum,
                                       int32_t workgroups, void* stream) {
  if (buf == nullptr || out_sum == nullptr || bytes == 0 || bytes % 16 != 0 ||
      reinterpret_cast<uintptr_t>(buf) % 16 != 0 || workgroups < 1 || workgroups > (1 << 20))
    return XP_EINVAL;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (hipMemsetAsync(out_sum, 0, sizeof(uint32_t), st) != hipSuccess) return XP_EHIP;
  hipLaunchKernelGGL(k_probe_read, dim3(workgroups), dim3(kProbeThreads), 0, st,
                     reinterpret_cast<const u32x4*>(buf), bytes / 16, out_sum);
  return hipGetLastError() == hipSuccess ? XP_OK : XP_EHIP;
}

extern "C" xp_status xp_probe_mfma_bf16(const void* operands, int32_t workgroups, int32_t iters,
                                        float* out, void* stream) {
  if (operands == nullptr || out == nullptr || workgroups < 1 || workgroups > (1 << 16) ||
      iters < 0 || reinterpret_cast<uintptr_t>(operands) % 16 != 0 ||
      reinterpret_cast<uintptr_t>(out) % 16 != 0)
    return XP_EINVAL;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(k_probe_mfma, dim3(workgroups), dim3(kProbeThreads), 0, st,
                     reinterpret_cast<const u32x4*>(operands), iters, out);
  return hipGetLastError() == hipSuccess ? XP_OK : XP_EHIP;
}
