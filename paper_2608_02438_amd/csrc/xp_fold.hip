// Weight-only precompute at handle creation.
//
// Fuse (eq. fuse) is linear in each of its three inputs, so the parts of it
// that touch only weights are folded once, in fp32 (section 4.1 notes that the
// linear Fuse-Mix path can be folded and precomputed):
//   T  [V][r] = W_e W_in[:, 2r:3r]^T   token part: a_k gets row T[x_{k-1}]
//   Fh [r][H] = W_in[:, 0:r]  W_h      applied to h_k
//   Fg [r][H] = W_in[:, r:2r] W_g      applied to g
// and L is repacked to its strictly lower part, Lp[k(k-1)/2 + i][d] = L[d][k][i].
#include "xp_internal.h"

namespace xp {

// T[v][d] = sum_e W_in[d][2r + e] * W_e[v][e]; 32 tokens per workgroup, thread d.
template <typename T>
__global__ __launch_bounds__(256) void k_fold_T(const T* __restrict__ We, const T* __restrict__ Win,
                                                int V, float* __restrict__ Ttab) {
  constexpr int r = 256, VB = 32;
  __shared__ float we[VB][r];
  const int v0 = blockIdx.x * VB, d = threadIdx.x;
  for (int i = threadIdx.x; i < VB * r; i += blockDim.x) {
    const int v = v0 + i / r;
    we[i / r][i % r] = v < V ? to_f32(We[(size_t)v * r + i % r]) : 0.f;
  }
  __syncthreads();
  float acc[VB];
#pragma unroll
  for (int i = 0; i < VB; ++i) acc[i] = 0.f;
  const T* w = Win + (size_t)d * (3 * r) + 2 * r;
  for (int e = 0; e < r; ++e) {
    const float wv = to_f32(w[e]);
#pragma unroll
    for (int i = 0; i < VB; ++i) acc[i] += wv * we[i][e];
  }
#pragma unroll
  for (int i = 0; i < VB; ++i)
    if (v0 + i < V) Ttab[(size_t)(v0 + i) * r + d] = acc[i];
}

// F[d][k] = sum_e W_in[d][cb*r + e] * Wx[e][k]; 16 rows d per workgroup, thread k.
template <typename T>
__global__ __launch_bounds__(256) void k_fold_F(const T* __restrict__ Win, int cb,
                                                const T* __restrict__ Wx, int H,
                                                float* __restrict__ F) {
  constexpr int r = 256, DB = 16;
  __shared__ float win[DB][r];
  const int d0 = blockIdx.y * DB, k = blockIdx.x * 256 + threadIdx.x;
  for (int i = threadIdx.x; i < DB * r; i += blockDim.x)
    win[i / r][i % r] = to_f32(Win[(size_t)(d0 + i / r) * (3 * r) + cb * r + i % r]);
  __syncthreads();
  if (k >= H) return;
  float acc[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) acc[i] = 0.f;
  for (int e = 0; e < r; ++e) {
    const float x = to_f32(Wx[(size_t)e * H + k]);
#pragma unroll
    for (int i = 0; i < DB; ++i) acc[i] += win[i][e] * x;
  }
#pragma unroll
  for (int i = 0; i < DB; ++i) F[(size_t)(d0 + i) * H + k] = acc[i];
}

template <typename T>
__global__ void k_pack_L(const T* __restrict__ L, int B, T* __restrict__ Lp) {
  constexpr int r = 256;
  const int pair = blockIdx.x, d = threadIdx.x;
  int k = 1;
  while ((k + 1) * k / 2 <= pair) ++k;          // pair = k(k-1)/2 + i, 0 <= i < k
  const int i = pair - k * (k - 1) / 2;
  Lp[(size_t)pair * r + d] = L[((size_t)d * B + k) * B + i];
}

template <typename T>
static hipError_t fold_t(xp_handle* h, hipStream_t st) {
  hipLaunchKernelGGL((k_fold_T<T>), dim3((h->V + 31) / 32), dim3(256), 0, st, (const T*)h->W_e,
                     (const T*)h->W_in, h->V, h->ws.T);
  hipLaunchKernelGGL((k_fold_F<T>), dim3((h->H + 255) / 256, h->r / 16), dim3(256), 0, st,
                     (const T*)h->W_in, 0, (const T*)h->W_h, h->H, h->ws.Fh);
  hipLaunchKernelGGL((k_fold_F<T>), dim3((h->H + 255) / 256, h->r / 16), dim3(256), 0, st,
                     (const T*)h->W_in, 1, (const T*)h->W_g, h->H, h->ws.Fg);
  const int npairs = h->B * (h->B - 1) / 2;
  if (npairs > 0)
    hipLaunchKernelGGL((k_pack_L<T>), dim3(npairs), dim3(256), 0, st, (const T*)h->L, h->B,
                       (T*)h->ws.Lp);
  return hipGetLastError();
}

hipError_t launch_fold(xp_handle* h, hipStream_t st) {
  return h->dtype == XP_BF16 ? fold_t<uint16_t>(h, st) : fold_t<float>(h, st);
}

}  // namespace xp
