// r-space stages of the refiner (section 4.1): Fuse, Mix, Trans.
//
// Fuse is linear, so its iteration-invariant part is computed once per call
// (h and g are fixed across Jacobi passes, section 4.2):
//     P_k = (W_in[:, 0:r] W_h) h_k + (W_in[:, r:2r] W_g) g ,   g = mean_j h_j
// and its token part is a row of the precomputed table T = W_e W_in[:, 2r:3r]^T,
// so a pass's Fuse is a gather:  a_k = P_k + T[x_{k-1}]  (eq. fuse).
// Mix (eq. mix) and the first Trans product run in one kernel per
// (sequence, slice of W_1 rows); W_2, the residual and the bf16 rounding of z
// in a second kernel (eq. mlp).
#include "xp_internal.h"

namespace xp {

// g[b][k] = (1/B) sum_j h[b][j][k]
template <typename T>
__global__ __launch_bounds__(256) void k_gmean(const T* __restrict__ hid, int B, int H,
                                               float* __restrict__ g) {
  const int b = blockIdx.x, k = blockIdx.y * 256 + threadIdx.x;
  if (k >= H) return;
  float acc = 0.f;
  for (int j = 0; j < B; ++j) acc += to_f32(hid[((size_t)b * B + j) * H + k]);
  g[(size_t)b * H + k] = acc / (float)B;
}

// out[n][o] = sum_k F[o][k] x_n[k] for n < N, o < O, F fp32 [O][Kd].
// One wave per output row, 16 input rows per workgroup column.
template <typename TX>
__global__ __launch_bounds__(256) void k_rowdot(const float* __restrict__ F, int O, int Kd,
                                                const TX* __restrict__ X, int N,
                                                float* __restrict__ out) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int o = blockIdx.x * 4 + wave, n0 = blockIdx.y * 16;
  if (o >= O) return;
  float acc[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) acc[j] = 0.f;
  for (int k = lane * 4; k < Kd; k += 256) {
    const float4 f = *reinterpret_cast<const float4*>(F + (size_t)o * Kd + k);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int n = n0 + j;
      if (n < N) {
        const TX* x = X + (size_t)n * Kd + k;
        acc[j] += f.x * to_f32(x[0]) + f.y * to_f32(x[1]) + f.z * to_f32(x[2]) + f.w * to_f32(x[3]);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < 16; ++j) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) acc[j] += __shfl_xor(acc[j], m, kWave);
  }
#pragma unroll
  for (int j = 0; j < 16; ++j)
    if (lane == j && n0 + j < N) out[(size_t)(n0 + j) * O + o] = acc[j];
}

// Fuse (gather form) + Mix + h1 = silu(W_1 c) for rows [j0, j0 + R1) of W_1.
// Thread d owns channel d (r = 256 threads).  Workgroup y == 0 also stores c.
template <typename T>
__global__ __launch_bounds__(256) void k_fuse_mix_w1(
    int B, int V, int R1, const float* __restrict__ uh, const float* __restrict__ ug,
    const float* __restrict__ Ttab, const T* __restrict__ Lp, const int32_t* __restrict__ anchor,
    const int32_t* __restrict__ Y, const T* __restrict__ W1, float* __restrict__ c_out,
    float* __restrict__ h1, uint32_t* __restrict__ err, const int32_t* __restrict__ ctrl,
    int skip_when_done) {
  if (skip_when_done && ctrl[1]) return;
  constexpr int r = 256;
  __shared__ float cs[32][r + 1];
  const int b = blockIdx.x, d = threadIdx.x;
  const float gpart = ug[(size_t)b * r + d];
  for (int k = 0; k < B; ++k) {
    int x = (k == 0) ? anchor[b] : Y[b * B + k - 1];
    if (x < 0 || x >= V) {
      atomicOr(err, XP_DEVERR_TOKEN);
      x = 0;
    }
    cs[k][d] = uh[((size_t)b * B + k) * r + d] + gpart + Ttab[(size_t)x * r + d];
  }
  // c_k = a_k + sum_{i<k} L[d][k][i] a_i, in place from the last position down
  for (int k = B - 1; k >= 1; --k) {
    float acc = cs[k][d];
    const T* lk = Lp + (size_t)(k * (k - 1) / 2) * r + d;
    for (int i = 0; i < k; ++i) acc += to_f32(lk[(size_t)i * r]) * cs[i][d];
    cs[k][d] = acc;
  }
  if (blockIdx.y == 0)
    for (int k = 0; k < B; ++k) c_out[((size_t)b * B + k) * r + d] = cs[k][d];
  __syncthreads();
  const int j0 = blockIdx.y * R1;
  for (int o = threadIdx.x; o < R1 * B; o += blockDim.x) {
    const int j = j0 + o / B, k = o % B;
    const T* w = W1 + (size_t)j * r;
    float acc = 0.f;
    for (int e = 0; e < r; ++e) acc += to_f32(w[e]) * cs[k][e];
    h1[((size_t)b * B + k) * (2 * r) + j] = acc / (1.f + expf(-acc));
  }
}

// z = c + W_2 h1 for rows [d0, d0 + R2); rounded to bf16 for bf16 weights.
template <typename T>
__global__ __launch_bounds__(256) void k_w2(int B, int R2, const float* __restrict__ c,
                                            const float* __restrict__ h1, const T* __restrict__ W2,
                                            T* __restrict__ z, const int32_t* __restrict__ ctrl,
                                            int skip_when_done) {
  if (skip_when_done && ctrl[1]) return;
  constexpr int r = 256, r2 = 512;
  __shared__ float hs[16][r2 + 1];
  const int b = blockIdx.x, d0 = blockIdx.y * R2;
  for (int kg = 0; kg < B; kg += 16) {
    const int nk = min(16, B - kg);
    __syncthreads();
    for (int i = threadIdx.x; i < nk * r2; i += blockDim.x)
      hs[i / r2][i % r2] = h1[((size_t)b * B + kg + i / r2) * r2 + i % r2];
    __syncthreads();
    for (int o = threadIdx.x; o < R2 * nk; o += blockDim.x) {
      const int dd = d0 + o / nk, k = o % nk;
      const T* w = W2 + (size_t)dd * r2;
      float acc = 0.f;
      for (int j = 0; j < r2; ++j) acc += to_f32(w[j]) * hs[k][j];
      const size_t m = (size_t)b * B + kg + k;
      const float zv = c[m * r + dd] + acc;
      if constexpr (sizeof(T) == 2)
        z[m * r + dd] = f32_to_bf16_rne(zv);
      else
        z[m * r + dd] = zv;
    }
  }
}

// ---------------------------------------------------------------------------
hipError_t launch_prep(xp_handle* h, int batch, const void* hidden, hipStream_t st) {
  const int M = batch * h->B;
  dim3 gg(batch, (h->H + 255) / 256);
  if (h->dtype == XP_BF16) {
    hipLaunchKernelGGL((k_gmean<uint16_t>), gg, dim3(256), 0, st, (const uint16_t*)hidden, h->B,
                       h->H, h->ws.g);
    hipLaunchKernelGGL((k_rowdot<uint16_t>), dim3(h->r / 4, (M + 15) / 16), dim3(256), 0, st,
                       h->ws.Fh, h->r, h->H, (const uint16_t*)hidden, M, h->ws.uh);
  } else {
    hipLaunchKernelGGL((k_gmean<float>), gg, dim3(256), 0, st, (const float*)hidden, h->B, h->H,
                       h->ws.g);
    hipLaunchKernelGGL((k_rowdot<float>), dim3(h->r / 4, (M + 15) / 16), dim3(256), 0, st,
                       h->ws.Fh, h->r, h->H, (const float*)hidden, M, h->ws.uh);
  }
  hipLaunchKernelGGL((k_rowdot<float>), dim3(h->r / 4, (batch + 15) / 16), dim3(256), 0, st,
                     h->ws.Fg, h->r, h->H, (const float*)h->ws.g, batch, h->ws.ug);
  return hipGetLastError();
}

static constexpr int kR1 = 16;   // W_1 rows per workgroup
static constexpr int kR2 = 16;   // W_2 rows per workgroup

hipError_t launch_fuse_mix_w1(xp_handle* h, int batch, int pass, uint32_t flags,
                              const int32_t* anchor, hipStream_t st) {
  const int skip = (flags & XP_EARLY_EXIT) ? 1 : 0;
  dim3 grid(batch, 2 * h->r / kR1);
  if (h->dtype == XP_BF16)
    hipLaunchKernelGGL((k_fuse_mix_w1<uint16_t>), grid, dim3(256), 0, st, h->B, h->V, kR1,
                       h->ws.uh, h->ws.ug, h->ws.T, (const uint16_t*)h->ws.Lp, anchor,
                       h->ws.Y[pass % 2], (const uint16_t*)h->W_1, h->ws.c, h->ws.h1, h->ws.err,
                       h->ws.ctrl, skip);
  else
    hipLaunchKernelGGL((k_fuse_mix_w1<float>), grid, dim3(256), 0, st, h->B, h->V, kR1, h->ws.uh,
                       h->ws.ug, h->ws.T, (const float*)h->ws.Lp, anchor, h->ws.Y[pass % 2],
                       (const float*)h->W_1, h->ws.c, h->ws.h1, h->ws.err, h->ws.ctrl, skip);
  return hipGetLastError();
}

hipError_t launch_w2(xp_handle* h, int batch, int pass, uint32_t flags, hipStream_t st) {
  (void)pass;
  const int skip = (flags & XP_EARLY_EXIT) ? 1 : 0;
  dim3 grid(batch, h->r / kR2);
  if (h->dtype == XP_BF16)
    hipLaunchKernelGGL((k_w2<uint16_t>), grid, dim3(256), 0, st, h->B, kR2, h->ws.c, h->ws.h1,
                       (const uint16_t*)h->W_2, (uint16_t*)h->ws.z, h->ws.ctrl, skip);
  else
    hipLaunchKernelGGL((k_w2<float>), grid, dim3(256), 0, st, h->B, kR2, h->ws.c, h->ws.h1,
                       (const float*)h->W_2, (float*)h->ws.z, h->ws.ctrl, skip);
  return hipGetLastError();
}

}  // namespace xp
