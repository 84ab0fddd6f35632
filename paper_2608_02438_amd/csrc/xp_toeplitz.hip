// The Toeplitz form of Mix (remark after Proposition 1, section 3): when the
// per-channel mixer depends only on the offset k - j, L^(d)_{k,j} = kappa_d[k - j],
// and Mix is a causal depthwise conv1d of kernel size B.  The handle folds any
// mixer into its per-pass operators once (the packed strictly-lower L), so the
// Toeplitz form needs no kernel of its own per pass: this entry point writes
// the full [r][B][B] mixer from the r x B kernel taps, on the device, for
// xp_weights.L.
#include "xp_internal.h"

namespace xp {

constexpr int kToepThreads = 256;

// one thread per entry (d, k, j) of L; lag 0 (the identity of eq. mix) and the
// upper triangle are written as zeros
template <typename T>
__global__ __launch_bounds__(kToepThreads) void k_toeplitz(const T* __restrict__ kappa, int B,
                                                          size_t n, T* __restrict__ L) {
  const size_t e = (size_t)blockIdx.x * kToepThreads + threadIdx.x;
  if (e >= n) return;
  const size_t d = e / ((size_t)B * B);
  const int kj = (int)(e - d * B * B), k = kj / B, j = kj - k * B;
  L[e] = j < k ? kappa[d * B + (k - j)] : T(0);
}

}  // namespace xp

using namespace xp;

extern "C" xp_status xp_toeplitz_mixer(const void* kappa, int32_t r, int32_t B, int32_t dtype,
                                       void* L_out, void* stream) {
  if (kappa == nullptr || L_out == nullptr || r < 1 || r > 65536 || B < 1 || B > 32 ||
      (dtype != XP_F32 && dtype != XP_BF16))
    return XP_EINVAL;
  const size_t n = (size_t)r * B * B;
  const int grid = (int)((n + kToepThreads - 1) / kToepThreads);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (dtype == XP_F32)
    hipLaunchKernelGGL(k_toeplitz<float>, dim3(grid), dim3(kToepThreads), 0, st,
                       static_cast<const float*>(kappa), (int)B, n, static_cast<float*>(L_out));
  else
    hipLaunchKernelGGL(k_toeplitz<uint16_t>, dim3(grid), dim3(kToepThreads), 0, st,
                       static_cast<const uint16_t*>(kappa), (int)B, n,
                       static_cast<uint16_t*>(L_out));
  return hipGetLastError() == hipSuccess ? XP_OK : XP_EHIP;
}
