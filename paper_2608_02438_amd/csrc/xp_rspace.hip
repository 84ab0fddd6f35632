// r-space stages of the refiner (section 4.1): Fuse, Mix, Trans.
//
// Fuse is linear, so its iteration-invariant part is computed once per call
// (h and g are fixed across Jacobi passes, section 4.2):
//     P_k = (W_in[:, 0:r] W_h) h_k + (W_in[:, r:2r] W_g) g ,   g = mean_j h_j
// by k_prep, and its token part is a row of the precomputed table
// T = W_e W_in[:, 2r:3r]^T, so a pass's Fuse is a gather:  a_k = P_k + T[x_{k-1}].
// A pass then runs Mix (eq. mix) and Trans (eq. mlp).  With bf16 weights the
// r-space products run on the bf16 matrix cores with the fp32 operand split
// into three exact bf16 terms (products exact, sums in fp32); with fp32
// weights they use v_mfma_f32_16x16x4_f32.  z is rounded to the weight dtype.
#include "xp_internal.h"
#include "xp_split.h"

namespace xp {

__device__ __forceinline__ float4 load4f(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 load4f(const uint16_t* p) {
  const uint2 v = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u),
                     __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xFFFF0000u));
}
__device__ __forceinline__ floatx4 mma4(float4 a, float4 b, floatx4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, c, 0, 0, 0);
  return c;
}

// ---------------------------------------------------------------------------
// k_prep: part[mat][ks][m][o] = F_mat[o][slice ks] . h[m][slice ks] for
// F_0 = W_in[:,0:r] W_h and F_1 = W_in[:,r:2r] W_g (fp32 [r][H]); the KSP
// slice partials are added (in slice order) by their consumer.  Grid (16 row
// tiles, KSP k-slices, 2 * groups of pbg position blocks); 4 waves split a
// slice and sum their 16x16 tiles in LDS in wave order.  F is split into
// three bf16 terms (exact), so the products run on the bf16 matrix cores;
// with bf16 h and slices of at most kPrepSteps steps a wave loads and splits
// its F fragments once for all its position blocks, and takes the blocks
// four at a time (their h loads issued together, one LDS reduction per four,
// wave w summing block w).  Workgroup (0,0,0) also clears the per-call
// Jacobi state.
// ---------------------------------------------------------------------------
constexpr int kPrepPBG = 8;            // position blocks per workgroup, at least
constexpr int kMaxKsp = 8;             // most k-slices of the prep product
constexpr int kPrepSteps = 4;          // 32-wide steps per wave loaded at once

// k-slices of the prep product: the most (up to 8) that leave every wave a
// whole number of 32-element (bf16) or 16-element (fp32) MFMA steps.
int prep_ksp(int H) {
  for (int k = 8; k > 1; k >>= 1)
    if (H % (k * 4 * 32) == 0) return k;
  return 1;
}

template <typename T>
__global__ __launch_bounds__(256) void k_prep(const float* __restrict__ Fh,
                                              const float* __restrict__ Fg,
                                              const T* __restrict__ hid, int H, int M,
                                              int ksp, int pbg, float* __restrict__ part,
                                              int batch,
                                              int32_t* __restrict__ iters,
                                              int32_t* __restrict__ ctrl,
                                              const uint8_t* __restrict__ temp,
                                              const float* __restrict__ temperature,
                                              float* __restrict__ invT,
                                              uint32_t* __restrict__ err) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rt = blockIdx.x, ks = blockIdx.y, mat = blockIdx.z & 1, pgi = blockIdx.z >> 1;
  if (blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0) {
    for (int i = threadIdx.x; i < batch; i += blockDim.x) {
      iters[i] = 0;
      // 1 / T of the sequence, the factor its sampled logits are scaled by
      // (softmax(l / T)); T must be finite and positive
      const float tau = temperature != nullptr ? temperature[i] : 1.f;
      const bool ok = tau > 0.f && tau <= 3.4e38f;             // false for NaN too
      if (!ok && temp != nullptr && temp[i] != 0) atomicOr(err, XP_DEVERR_TEMPERATURE);
      invT[i] = ok ? 1.f / tau : 1.f;
    }
    if (threadIdx.x < 2) ctrl[threadIdx.x] = 0;
  }
  const float* F = mat ? Fg : Fh;
  const int kw = H / ksp / 4;                                 // k per wave
  const int g = lane >> 4, li = lane & 15;
  const int k0 = ks * (H / ksp) + wave * kw;
  const float* arow = F + (size_t)(rt * 16 + li) * H + k0;
  __shared__ floatx4 red[4][4][64];
  const int npb = (M + 15) / 16;
  const int pb0 = pgi * pbg, pb1 = min(npb, (pgi + 1) * pbg);
  if constexpr (sizeof(T) == 2) {
    if (kw / 32 <= kPrepSteps) {
      const int ns = kw / 32;
      u32x4 fh[kPrepSteps], fm[kPrepSteps], fl[kPrepSteps];
#pragma unroll
      for (int u = 0; u < kPrepSteps; ++u) {
        const int uc = u < ns ? u : ns - 1;
        split3x8(*reinterpret_cast<const float4*>(arow + uc * 32 + 8 * g),
                 *reinterpret_cast<const float4*>(arow + uc * 32 + 8 * g + 4), fh[u], fm[u], fl[u]);
      }
      for (int pq = pb0; pq < pb1; pq += 4) {
        u32x4 bv[4][kPrepSteps];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int p = (pq + q) * 16 + li;
          const T* brow = hid + (size_t)(p < M ? p : M - 1) * H + k0 + 8 * g;
#pragma unroll
          for (int u = 0; u < kPrepSteps; ++u) {
            bv[q][u] = ld16(brow + (u < ns ? u : ns - 1) * 32);
            if (pq + q >= pb1 || p >= M) bv[q][u] = u32x4{0u, 0u, 0u, 0u};
          }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int u = 0; u < kPrepSteps; ++u)
            if (u < ns) {
              acc = Mfma<uint16_t>::mma(fh[u], bv[q][u], acc);
              acc = Mfma<uint16_t>::mma(fm[u], bv[q][u], acc);
              acc = Mfma<uint16_t>::mma(fl[u], bv[q][u], acc);
            }
          red[wave][q][lane] = acc;
        }
        __syncthreads();
        if (pq + wave < pb1) {                        // wave w sums block pq + w in wave order
          floatx4 s = red[0][wave][lane];
#pragma unroll
          for (int w = 1; w < 4; ++w) {
            const floatx4 o = red[w][wave][lane];
            s[0] += o[0]; s[1] += o[1]; s[2] += o[2]; s[3] += o[3];
          }
          const int p = (pq + wave) * 16 + li;
          if (p < M) {
            float* dst = part + (((size_t)mat * ksp + ks) * M + p) * 256 + rt * 16 + 4 * g;
            *reinterpret_cast<float4*>(dst) = make_float4(s[0], s[1], s[2], s[3]);
          }
        }
        __syncthreads();
      }
      return;
    }
  }
  for (int pb = pb0; pb < pb1; ++pb) {
    const int p = pb * 16 + li;
    const int pc = p < M ? p : M - 1;
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    if constexpr (sizeof(T) == 2) {
      // all (at most kPrepSteps) steps of the wave's slice are loaded at once
      const T* brow = hid + (size_t)pc * H + k0 + 8 * g;
      const int ns = kw / 32;
      float4 a0[kPrepSteps], a1[kPrepSteps];
      u32x4 bv[kPrepSteps];
#pragma unroll
      for (int u = 0; u < kPrepSteps; ++u) {
        const int uc = u < ns ? u : ns - 1;
        a0[u] = *reinterpret_cast<const float4*>(arow + uc * 32 + 8 * g);
        a1[u] = *reinterpret_cast<const float4*>(arow + uc * 32 + 8 * g + 4);
        bv[u] = ld16(brow + uc * 32);
      }
#pragma unroll
      for (int u = 0; u < kPrepSteps; ++u) {
        if (u < ns) acc = mma_split_a(a0[u], a1[u], p < M ? bv[u] : u32x4{0u, 0u, 0u, 0u}, acc);
      }
      for (int u = kPrepSteps; u < ns; ++u) {       // slices longer than kPrepSteps steps
        const float4 c0 = *reinterpret_cast<const float4*>(arow + u * 32 + 8 * g);
        const float4 c1 = *reinterpret_cast<const float4*>(arow + u * 32 + 8 * g + 4);
        u32x4 b1 = ld16(brow + u * 32);
        if (p >= M) b1 = u32x4{0u, 0u, 0u, 0u};
        acc = mma_split_a(c0, c1, b1, acc);
      }
    } else {
      const T* brow = hid + (size_t)pc * H + k0 + 4 * g;
      for (int u = 0; u < kw / 16; ++u) {
        const float4 a = load4f(arow + u * 16 + 4 * g);
        float4 bv = load4f(brow + u * 16);
        if (p >= M) bv = make_float4(0.f, 0.f, 0.f, 0.f);
        acc = mma4(a, bv, acc);
      }
    }
    red[wave][0][lane] = acc;
    __syncthreads();
    if (wave == 0) {
      floatx4 s = red[0][0][lane];
#pragma unroll
      for (int w = 1; w < 4; ++w) {
        const floatx4 o = red[w][0][lane];
        s[0] += o[0]; s[1] += o[1]; s[2] += o[2]; s[3] += o[3];
      }
      if (p < M) {
        float* dst = part + (((size_t)mat * ksp + ks) * M + p) * 256 + rt * 16 + 4 * g;
        *reinterpret_cast<float4*>(dst) = make_float4(s[0], s[1], s[2], s[3]);
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// One Jacobi pass in r-space runs as three short, wide kernels so that every
// workgroup reads only a few KB (a single CU streams from L2 at well under
// 100 GB/s, so per-workgroup bytes, not flops, set the time):
//   k_fusemix  (batch, 16 d-tiles):  a_k = P_k + T[x_{k-1}], c = (I + L) a
//   k_trans1   (batch, 32 row tiles): h1 = silu(W_1 c), 16 rows each
//   k_trans2   (batch, 16 row tiles): z = c + W_2 h1, rounded to the weight dtype
// Every load a workgroup needs is issued before its first use and none sits
// under a branch (indices are clamped, results masked), so the loads overlap.
// ---------------------------------------------------------------------------

// Pa_k = F_h h_k + (1/B) sum_j F_g h_j: the pass-invariant part of Fuse,
// from the prep k-slice partials (added in slice order), once per call.
template <int BP>
__global__ __launch_bounds__(256) void k_prep_sum(int B, int M, int ksp,
                                                  const float* __restrict__ part,
                                                  float* __restrict__ Pa) {
  constexpr int r = 256, EPT = BP / 16;
  __shared__ float G[BP][17];
  __shared__ float ug[16];
  const int b = blockIdx.x, dt = blockIdx.y, tid = threadIdx.x;
  const int dl = tid & 15, kg = tid >> 4, d = dt * 16 + dl;
  float phv[EPT][kMaxKsp], pgv[EPT][kMaxKsp];
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const int k = kg + 16 * j;
    const size_t m = (size_t)b * B + (k < B ? k : B - 1);
#pragma unroll
    for (int q = 0; q < kMaxKsp; ++q) {
      const int qc = q < ksp ? q : ksp - 1;
      phv[j][q] = part[((size_t)qc * M + m) * r + d];
      pgv[j][q] = part[((size_t)(ksp + qc) * M + m) * r + d];
    }
  }
  float ph[EPT];
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    float sh = 0.f, sg = 0.f;
#pragma unroll
    for (int q = 0; q < kMaxKsp; ++q) {
      sh += q < ksp ? phv[j][q] : 0.f;
      sg += q < ksp ? pgv[j][q] : 0.f;
    }
    ph[j] = sh;
    const int k = kg + 16 * j;
    if (k < B) G[k][dl] = sg;
  }
  __syncthreads();
  if (tid < 16) {                                    // (W_in[:,r:2r] W_g) g, g = mean_k h_k
    float t = 0.f;
    for (int k = 0; k < B; ++k) t += G[k][tid];
    ug[tid] = t / (float)B;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const int k = kg + 16 * j;
    if (k < B) Pa[((size_t)b * B + k) * r + d] = ph[j] + ug[dl];
  }
}

// Fuse (gather form) and Mix for 16 feature dims d of one sequence.  Mix is
// independent per d (eq. mix: c^(d) = (I + L^(d)) a^(d)), so the 16 dims of a
// workgroup need only their own 16 columns of every L^(d).
template <typename T, int BP>
__global__ __launch_bounds__(256) void k_fusemix(
    int B, int V, int M, const float* __restrict__ Pa, const float* __restrict__ Ttab,
    const T* __restrict__ Lp, const int32_t* __restrict__ anchor, const int32_t* __restrict__ Y,
    float* __restrict__ c, uint32_t* __restrict__ err, const int32_t* __restrict__ iters,
    int skip_when_done) {
  if (skip_when_done && iters[blockIdx.x]) return;    // the sequence is at its fixed point
  constexpr int r = 256;
  constexpr int EPT = BP / 16;                       // positions per thread
  constexpr int NPAIR = BP * (BP - 1) / 2;
  constexpr int CPP = (int)sizeof(T);                // 16-byte chunks per pair (16 dims)
  constexpr int LCH_T = (NPAIR * CPP + 255) / 256;   // chunks per thread
  __shared__ float A[BP][17];
  __shared__ u32x4 Ls[NPAIR * CPP > 0 ? NPAIR * CPP : 1];
  const int b = blockIdx.x, dt = blockIdx.y, tid = threadIdx.x;
  const int dl = tid & 15, kg = tid >> 4, d = dt * 16 + dl;
  const int npair = B * (B - 1) / 2, nch = npair * CPP;

  u32x4 lc[LCH_T];
#pragma unroll
  for (int j = 0; j < LCH_T; ++j) {                  // L columns [dt*16, dt*16+16) of every pair
    int q = tid + 256 * j;
    q = q < nch ? q : (nch > 0 ? nch - 1 : 0);
    const int pr = q / CPP, cc = q % CPP;
    lc[j] = *reinterpret_cast<const u32x4*>(Lp + (size_t)pr * r + dt * 16 + cc * (16 / CPP));
  }
  // the Fuse constant Pa_k and the previous tokens, issued together
  float pa[EPT], tv[EPT];
  int xv[EPT];
  const int ya = anchor[b];
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const int k = kg + 16 * j;
    const int kc = k < B ? k : B - 1;
    const size_t m = (size_t)b * B + kc;
    pa[j] = Pa[m * r + d];
    xv[j] = Y[kc == 0 ? m : m - 1];
    if (kc == 0) xv[j] = ya;
  }
  bool bad = false;
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const int x = xv[j];
    const bool ok = x >= 0 && x < V;
    bad |= !ok && kg + 16 * j < B;
    tv[j] = Ttab[(size_t)(ok ? x : 0) * r + d];
  }
#pragma unroll
  for (int j = 0; j < LCH_T; ++j) {
    const int q = tid + 256 * j;
    if (q < nch) Ls[q] = lc[j];
  }
#pragma unroll
  for (int j = 0; j < EPT; ++j) {                    // a_k = Pa_k + T[x_{k-1}]; rows >= B
    const int k = kg + 16 * j;                       // are zeroed without a branch
    A[k][dl] = (pa[j] + tv[j]) * (k < B ? 1.f : 0.f);
  }
  if (bad) atomicOr(err, XP_DEVERR_TOKEN);
  __syncthreads();
  const T* ls = reinterpret_cast<const T*>(Ls);      // [pair][16 dims]
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const int k = kg + 16 * j;
    if (k < B) {
      float acc = A[k][dl];
      const int p0 = k * (k - 1) / 2;
      for (int i = 0; i < k; ++i) acc += to_f32(ls[(p0 + i) * 16 + dl]) * A[i][dl];
      c[((size_t)b * B + k) * r + d] = acc;
    }
  }
}

// h1[m][16*rt .. 16*rt+16) = silu(W_1[rows] c_m) for the positions of one
// sequence; 4 waves split the 256-long contraction and add their tiles in
// wave order.
template <typename T, int BP>
__global__ __launch_bounds__(256) void k_trans1(int B, const T* __restrict__ W1,
                                                const float* __restrict__ c,
                                                float* __restrict__ h1,
                                                const int32_t* __restrict__ iters,
                                                int skip_when_done) {
  if (skip_when_done && iters[blockIdx.x]) return;    // the sequence is at its fixed point
  constexpr int r = 256, r2 = 512, NPB = BP / 16;
  constexpr bool kBf = sizeof(T) == 2;
  const int b = blockIdx.x, rt = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, li = lane & 15;
  const int k0 = wave * (r / 4);                     // this wave's 64-long k slice
  const T* arow = W1 + (size_t)(rt * 16 + li) * r + k0;
  __shared__ floatx4 red[4][NPB][64];
  floatx4 acc[NPB];
  if constexpr (kBf) {
    u32x4 w[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) w[u] = ld16(arow + u * 32 + 8 * g);
    float4 x[NPB][2][2];
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      const int k = pb * 16 + li;
      const float* crow = c + ((size_t)b * B + (k < B ? k : B - 1)) * r + k0 + 8 * g;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        x[pb][u][0] = *reinterpret_cast<const float4*>(crow + u * 32);
        x[pb][u][1] = *reinterpret_cast<const float4*>(crow + u * 32 + 4);
      }
    }
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      acc[pb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < 2; ++u) acc[pb] = mma_split_b(w[u], x[pb][u][0], x[pb][u][1], acc[pb]);
    }
  } else {
    float4 w[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) w[u] = load4f(arow + u * 16 + 4 * g);
    float4 x[NPB][4];
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      const int k = pb * 16 + li;
      const float* crow = c + ((size_t)b * B + (k < B ? k : B - 1)) * r + k0 + 4 * g;
#pragma unroll
      for (int u = 0; u < 4; ++u) x[pb][u] = *reinterpret_cast<const float4*>(crow + u * 16);
    }
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      acc[pb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[pb] = mma4(w[u], x[pb][u], acc[pb]);
    }
  }
#pragma unroll
  for (int pb = 0; pb < NPB; ++pb) red[wave][pb][lane] = acc[pb];
  __syncthreads();
  if (wave < NPB) {
    const int pb = wave;
    const floatx4 q0 = red[0][pb][lane], q1 = red[1][pb][lane];
    const floatx4 q2 = red[2][pb][lane], q3 = red[3][pb][lane];
    const int k = pb * 16 + li;
    if (k < B) {
      float o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = ((q0[i] + q1[i]) + q2[i]) + q3[i];
        o[i] = v / (1.f + expf(-v));
      }
      *reinterpret_cast<float4*>(h1 + ((size_t)b * B + k) * r2 + rt * 16 + 4 * g) =
          make_float4(o[0], o[1], o[2], o[3]);
    }
  }
}

// z[m][16*zt .. 16*zt+16) = c_m + W_2[rows] h1_m (eq. mlp), rounded to the
// weight dtype; 4 waves split the 512-long contraction.
template <typename T, int BP>
__global__ __launch_bounds__(256) void k_trans2(int B, const T* __restrict__ W2,
                                                const float* __restrict__ c,
                                                const float* __restrict__ h1, T* __restrict__ z,
                                                const int32_t* __restrict__ iters,
                                                int skip_when_done) {
  if (skip_when_done && iters[blockIdx.x]) return;    // the sequence is at its fixed point
  constexpr int r = 256, r2 = 512, NPB = BP / 16;
  constexpr bool kBf = sizeof(T) == 2;
  const int b = blockIdx.x, zt = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, li = lane & 15;
  const int k0 = wave * (r2 / 4);                    // this wave's 128-long k slice
  const T* arow = W2 + (size_t)(zt * 16 + li) * r2 + k0;
  __shared__ floatx4 red[4][NPB][64];
  floatx4 acc[NPB];
  float4 res[NPB];
  if constexpr (kBf) {
    u32x4 w[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) w[u] = ld16(arow + u * 32 + 8 * g);
    float4 x[NPB][4][2];
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      const int k = pb * 16 + li;
      const float* hrow = h1 + ((size_t)b * B + (k < B ? k : B - 1)) * r2 + k0 + 8 * g;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        x[pb][u][0] = *reinterpret_cast<const float4*>(hrow + u * 32);
        x[pb][u][1] = *reinterpret_cast<const float4*>(hrow + u * 32 + 4);
      }
      res[pb] = *reinterpret_cast<const float4*>(c + ((size_t)b * B + (k < B ? k : B - 1)) * r +
                                                 zt * 16 + 4 * g);
    }
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      acc[pb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[pb] = mma_split_b(w[u], x[pb][u][0], x[pb][u][1], acc[pb]);
    }
  } else {
    float4 w[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) w[u] = load4f(arow + u * 16 + 4 * g);
    float4 x[NPB][8];
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      const int k = pb * 16 + li;
      const float* hrow = h1 + ((size_t)b * B + (k < B ? k : B - 1)) * r2 + k0 + 4 * g;
#pragma unroll
      for (int u = 0; u < 8; ++u) x[pb][u] = *reinterpret_cast<const float4*>(hrow + u * 16);
      res[pb] = *reinterpret_cast<const float4*>(c + ((size_t)b * B + (k < B ? k : B - 1)) * r +
                                                 zt * 16 + 4 * g);
    }
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      acc[pb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < 8; ++u) acc[pb] = mma4(w[u], x[pb][u], acc[pb]);
    }
  }
#pragma unroll
  for (int pb = 0; pb < NPB; ++pb) red[wave][pb][lane] = acc[pb];
  __syncthreads();
  if (wave < NPB) {
    const int pb = wave;
    const floatx4 q0 = red[0][pb][lane], q1 = red[1][pb][lane];
    const floatx4 q2 = red[2][pb][lane], q3 = red[3][pb][lane];
    const int k = pb * 16 + li;
    float4 cr = res[0];                              // residual c of this block
#pragma unroll
    for (int q = 1; q < NPB; ++q)
      if (pb == q) cr = res[q];
    if (k < B) {
      const float cv[4] = {cr.x, cr.y, cr.z, cr.w};
      const size_t m = (size_t)b * B + k;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float zv = cv[i] + (((q0[i] + q1[i]) + q2[i]) + q3[i]);
        if constexpr (kBf)
          z[m * r + zt * 16 + 4 * g + i] = f32_to_bf16_rne(zv);
        else
          z[m * r + zt * 16 + 4 * g + i] = zv;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// The two Trans products for many positions (bf16 weights, M >= kTransTiled):
// MODE 0 h1 = silu(W_1 c) (K = r), MODE 1 z = bf16(c + W_2 h1) (K = 2r).  The
// per-sequence kernels above re-read a sequence's inputs once per 16-row
// tile; here a workgroup takes 64 output rows x 32 positions, stages the
// positions' fp32 inputs once in LDS (rows padded by 16 bytes, so the 16
// positions of a fragment read fall in different banks), and each wave holds
// its 16 weight rows for the whole contraction in registers.  Products are
// the same exact split-term products, summed in fp32 in k order.  The
// results of sequences already at their fixed point are recomputed from
// unchanged inputs, so they do not change; a launch after the whole batch
// converged returns at once.
// ---------------------------------------------------------------------------
constexpr int kTransTiled = 1024;      // positions from which the tiled kernels run
constexpr int kTransPT = 32;           // positions per workgroup

template <int K, int MODE>
__global__ __launch_bounds__(256) void k_trans_tiled(const uint16_t* __restrict__ W,
                                                     const float* __restrict__ x, int M,
                                                     const float* __restrict__ c,
                                                     float* __restrict__ h1,
                                                     uint16_t* __restrict__ z,
                                                     const int32_t* __restrict__ ctrl,
                                                     int skip_when_done) {
  if (skip_when_done && ctrl[1]) return;             // every sequence is at its fixed point
  constexpr int LDX = K + 4;                         // floats per staged row
  constexpr int r = 256, NO = MODE == 0 ? 2 * r : r; // output rows
  __shared__ float xs[kTransPT * LDX];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, li = lane & 15;
  const int m0 = blockIdx.y * kTransPT;
  const int ob = blockIdx.x * 64 + wave * 16;        // the wave's first output row
  // the wave's weight rows (A operand: row ob + li, k = 32 ks + 8 g ..)
  u32x4 w[K / 32];
#pragma unroll
  for (int ks = 0; ks < K / 32; ++ks) w[ks] = ld16(W + (size_t)(ob + li) * K + 32 * ks + 8 * g);
  // the positions' inputs (rows past M repeat row M - 1)
#pragma unroll
  for (int j = 0; j < kTransPT * K / 4 / 256; ++j) {
    const int i = threadIdx.x + 256 * j;
    const int row = i / (K / 4), col = 4 * (i - row * (K / 4));
    const int m = m0 + row < M ? m0 + row : M - 1;
    *reinterpret_cast<float4*>(&xs[row * LDX + col]) =
        *reinterpret_cast<const float4*>(x + (size_t)m * K + col);
  }
  __syncthreads();
  floatx4 acc[kTransPT / 16];
#pragma unroll
  for (int pb = 0; pb < kTransPT / 16; ++pb) acc[pb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < K / 32; ++ks)
#pragma unroll
    for (int pb = 0; pb < kTransPT / 16; ++pb) {
      const float* xr = &xs[(pb * 16 + li) * LDX + 32 * ks + 8 * g];
      acc[pb] = mma_split_b(w[ks], *reinterpret_cast<const float4*>(xr),
                            *reinterpret_cast<const float4*>(xr + 4), acc[pb]);
    }
  // lane holds output rows ob + 4 g + i of position pb * 16 + li
#pragma unroll
  for (int pb = 0; pb < kTransPT / 16; ++pb) {
    const int m = m0 + pb * 16 + li;
    if (m >= M) continue;
    if constexpr (MODE == 0) {
      float o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = acc[pb][i];
        o[i] = v / (1.f + expf(-v));
      }
      *reinterpret_cast<float4*>(h1 + (size_t)m * NO + ob + 4 * g) = make_float4(o[0], o[1], o[2], o[3]);
    } else {
      const float4 cr = *reinterpret_cast<const float4*>(c + (size_t)m * r + ob + 4 * g);
      const float cv[4] = {cr.x, cr.y, cr.z, cr.w};
      uint16_t o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = f32_to_bf16_rne(cv[i] + acc[pb][i]);
      *reinterpret_cast<uint2*>(z + (size_t)m * r + ob + 4 * g) =
          make_uint2(o[0] | ((uint32_t)o[1] << 16), o[2] | ((uint32_t)o[3] << 16));
    }
  }
}

// ---------------------------------------------------------------------------
hipError_t launch_prep(xp_handle* h, int batch, const void* hidden, const uint8_t* temp,
                       const float* temperature, hipStream_t st) {
  const int M = batch * h->B;
  const int npb = (M + 15) / 16;
  const int ksp = prep_ksp(h->H);
  // position blocks per workgroup: kPrepPBG, more for large calls (about
  // four groups, so a launch has 2 * 16 * ksp * 4 workgroups)
  const int pbg = std::max(kPrepPBG, (npb + 3) / 4);
  dim3 grid(h->r / 16, ksp, 2 * ((npb + pbg - 1) / pbg));
  if (h->dtype == XP_BF16)
    hipLaunchKernelGGL((k_prep<uint16_t>), grid, dim3(256), 0, st, h->ws.Fh, h->ws.Fg,
                       (const uint16_t*)hidden, h->H, M, ksp, pbg, h->ws.ppart, batch,
                       h->ws.iters, h->ws.ctrl, temp, temperature, h->ws.invT, h->ws.err);
  else
    hipLaunchKernelGGL((k_prep<float>), grid, dim3(256), 0, st, h->ws.Fh, h->ws.Fg,
                       (const float*)hidden, h->H, M, ksp, pbg, h->ws.ppart, batch,
                       h->ws.iters, h->ws.ctrl, temp, temperature, h->ws.invT, h->ws.err);
  if (h->B <= 16)
    hipLaunchKernelGGL((k_prep_sum<16>), dim3(batch, 16), dim3(256), 0, st, h->B, M, ksp,
                       h->ws.ppart, h->ws.Pa);
  else
    hipLaunchKernelGGL((k_prep_sum<32>), dim3(batch, 16), dim3(256), 0, st, h->B, M, ksp,
                       h->ws.ppart, h->ws.Pa);
  return hipGetLastError();
}

// front = false launches only the second Trans product (the fused pass kernel
// has already produced c and h1).
template <typename T, int BP>
static void rspace_t(xp_handle* h, int batch, int pass, int skip, const int32_t* anchor,
                     bool front, hipStream_t st) {
  const int M = batch * h->B;
  const bool tiled = sizeof(T) == 2 && M >= kTransTiled;
  const dim3 tgrid1(512 / 64, (M + kTransPT - 1) / kTransPT), tgrid2(256 / 64, tgrid1.y);
  if (front) {
    hipLaunchKernelGGL((k_fusemix<T, BP>), dim3(batch, 16), dim3(256), 0, st, h->B, h->V, M,
                       h->ws.Pa, h->ws.T, (const T*)h->ws.Lp, anchor, h->ws.Y[pass % 2], h->ws.c,
                       h->ws.err, h->ws.iters, skip);
    if (tiled)
      hipLaunchKernelGGL((k_trans_tiled<256, 0>), tgrid1, dim3(256), 0, st,
                         (const uint16_t*)h->W_1, h->ws.c, M, h->ws.c, h->ws.h1,
                         (uint16_t*)nullptr, h->ws.ctrl, skip);
    else
      hipLaunchKernelGGL((k_trans1<T, BP>), dim3(batch, 32), dim3(256), 0, st, h->B,
                         (const T*)h->W_1, h->ws.c, h->ws.h1, h->ws.iters, skip);
  }
  if (tiled)
    hipLaunchKernelGGL((k_trans_tiled<512, 1>), tgrid2, dim3(256), 0, st,
                       (const uint16_t*)h->W_2, h->ws.h1, M, h->ws.c, (float*)nullptr,
                       (uint16_t*)h->ws.z, h->ws.ctrl, skip);
  else
    hipLaunchKernelGGL((k_trans2<T, BP>), dim3(batch, 16), dim3(256), 0, st, h->B,
                       (const T*)h->W_2, h->ws.c, h->ws.h1, (T*)h->ws.z, h->ws.iters, skip);
}

hipError_t launch_rspace(xp_handle* h, int batch, int pass, uint32_t flags, const int32_t* anchor,
                         bool front, hipStream_t st) {
  const int skip = (flags & XP_EARLY_EXIT) ? 1 : 0;
  if (h->dtype == XP_BF16) {
    if (h->B <= 16)
      rspace_t<uint16_t, 16>(h, batch, pass, skip, anchor, front, st);
    else
      rspace_t<uint16_t, 32>(h, batch, pass, skip, anchor, front, st);
  } else {
    if (h->B <= 16)
      rspace_t<float, 16>(h, batch, pass, skip, anchor, front, st);
    else
      rspace_t<float, 32>(h, batch, pass, skip, anchor, front, st);
  }
  return hipGetLastError();
}

}  // namespace xp
