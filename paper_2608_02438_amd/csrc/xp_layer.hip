// The context layer: one Qwen3-8B-shaped decoder layer over the positions of
// a drafted block, attending to each sequence's context KV (the layer whose
// output h the base readout s_k = W_lm h_k of section 4.1 consumes; the
// refiner itself never reads the context, Proposition 1).
//
// Kernels, in launch order:
//   k_rmsnorm     RMSNorm of x (bf16 in, fp32 copy out) and of x1, to bf16 u;
//                 x1 = the output projection's split-K slabs + x where that
//                 projection was split
//   k_gemv_sk     (one block of up to 16 positions, K <= 4096) y = u W^T
//                 (+ residual) in the LM-head stream kernel's manner: x in
//                 LDS, stream-K items with line-complete loads, per-wave LDS
//                 transpose; gate and up side by side, then k_swiglu
//   k_linear      (otherwise up to 64 positions) y = u W^T (+ residual), or the SwiGLU
//                 product of the gate and up projections: W streamed from HBM,
//                 split over the 8 waves of a workgroup along k, 16 or 32
//                 output rows per workgroup, 16 P positions per pass of the
//                 weight, the waves' partial sums added in fixed order in LDS;
//                 above 64 positions the tiled GEMM of xp_lgemm.hip takes
//                 the projections (SwiGLU in its epilogue; split-K where its
//                 tiles are fewer than the CUs)
//   k_qkrope      QK-norm and RoPE of every q and k head, v to bf16 (adding
//                 the q/k/v projection's split-K slabs)
//   k_attn        split-KV block attention: a workgroup takes a chunk of
//                 64-key sub-chunks of one KV head for 16 block positions, one
//                 wave per query head of the group, with an online softmax;
//                 each sub-chunk's K and V (transposed) staged in LDS while the
//                 next one loads; S = K Q^T and O = P V on the matrix cores
//   k_attn_comb   merges the chunks of every query row in chunk order
//   k_splitk_sum  the down projection's split-K slabs + x1, to h
// Every reduction runs in a fixed order, so two runs give identical bits.
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <mutex>

#include "xp_internal.h"

namespace xp {

constexpr int kLinWaves = 8;        // k-split of k_linear
constexpr int kLinMaxStream = 64;   // positions up to which the projections stream
constexpr int kAttnWgs = 1024;      // attention workgroups aimed at per call
constexpr int kHd = 128;            // head_dim (the only one built)

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

// ---------------------------------------------------------------------------
// RMSNorm of one row per workgroup: u = bf16(x / sqrt(mean(x^2) + eps) * g).
// The input is bf16 or fp32 (a template parameter: a select between two
// pointers per element would put every load under a branch); with S > 0
// (fp32 only) the row is (P_0 + ... + P_{S-1}) + x, P_s = P + s slab, added in
// that order; x32, if given, receives the fp32 row.
// ---------------------------------------------------------------------------
template <typename TI>
__global__ __launch_bounds__(256) void k_rmsnorm(const TI* __restrict__ x,
                                                 const float* __restrict__ P, int S, size_t slab,
                                                 int H, const uint16_t* __restrict__ g, float eps,
                                                 float* __restrict__ x32,
                                                 uint16_t* __restrict__ u) {
  // chunks of 8 consecutive elements (16-byte bf16 loads and stores); H is a
  // multiple of 256 up to 8192, so a thread takes at most 4 chunks
  constexpr int kPer = 8192 / 8 / 256;
  __shared__ float part[4];
  const size_t row = blockIdx.x;
  const int tid = threadIdx.x, nch = H / 8;
  float v[kPer][8];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {               // clamped loads: none under a branch
    const int c = tid + 256 * j, cc = c < nch ? c : nch - 1;
    if constexpr (sizeof(TI) == 2) {
      const u32x4 q = ld16(x + row * H + 8 * (size_t)cc);
      const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[j][2 * e] = bf16_to_f32((uint16_t)(w[e] & 0xFFFFu));
        v[j][2 * e + 1] = bf16_to_f32((uint16_t)(w[e] >> 16));
      }
    } else {
      const size_t off = row * H + 8 * (size_t)cc;
      float4 a = *reinterpret_cast<const float4*>(x + off);
      float4 b = *reinterpret_cast<const float4*>(x + off + 4);
      if (S > 0) {
        float4 pa = *reinterpret_cast<const float4*>(P + off);
        float4 pb = *reinterpret_cast<const float4*>(P + off + 4);
        for (int q = 1; q < S; ++q) {
          const float4 ta = *reinterpret_cast<const float4*>(P + q * slab + off);
          const float4 tb = *reinterpret_cast<const float4*>(P + q * slab + off + 4);
          pa.x += ta.x; pa.y += ta.y; pa.z += ta.z; pa.w += ta.w;
          pb.x += tb.x; pb.y += tb.y; pb.z += tb.z; pb.w += tb.w;
        }
        a = make_float4(pa.x + a.x, pa.y + a.y, pa.z + a.z, pa.w + a.w);
        b = make_float4(pb.x + b.x, pb.y + b.y, pb.z + b.z, pb.w + b.w);
      }
      v[j][0] = a.x; v[j][1] = a.y; v[j][2] = a.z; v[j][3] = a.w;
      v[j][4] = b.x; v[j][5] = b.y; v[j][6] = b.z; v[j][7] = b.w;
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kPer; ++j)
    if (tid + 256 * j < nch)
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += v[j][e] * v[j][e];
  ss = wave_sum(ss);
  if ((tid & 63) == 0) part[tid >> 6] = ss;
  __syncthreads();
  const float tot = (part[0] + part[1]) + (part[2] + part[3]);
  const float r = 1.f / sqrtf(tot / (float)H + eps);
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int c = tid + 256 * j;
    if (c < nch) {
      const u32x4 gq = ld16(g + 8 * (size_t)c);
      const uint32_t gw[4] = {gq.x, gq.y, gq.z, gq.w};
      uint32_t o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float g0 = bf16_to_f32((uint16_t)(gw[e] & 0xFFFFu));
        const float g1 = bf16_to_f32((uint16_t)(gw[e] >> 16));
        o[e] = f32_to_bf16_rne(v[j][2 * e] * r * g0) |
               ((uint32_t)f32_to_bf16_rne(v[j][2 * e + 1] * r * g1) << 16);
      }
      *reinterpret_cast<u32x4*>(u + row * H + 8 * (size_t)c) = u32x4{o[0], o[1], o[2], o[3]};
      if (x32) {
        *reinterpret_cast<float4*>(x32 + row * H + 8 * (size_t)c) =
            make_float4(v[j][0], v[j][1], v[j][2], v[j][3]);
        *reinterpret_cast<float4*>(x32 + row * H + 8 * (size_t)c + 4) =
            make_float4(v[j][4], v[j][5], v[j][6], v[j][7]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// y[p][n] = sum_k X[p][k] W[n][k] (+ R[p][n]) for 16 rows n per workgroup
// (blockIdx.x; 32 in MODE 2) and 16 P positions (blockIdx.y).  Up to three
// weights stacked by rows share a launch (rows [0, n0) of W0, [n0, n0 + n1)
// of W1, the rest of W2: the q, k and v projections of one input).  MODE 1
// (GLU): a workgroup takes the same 16 rows of W0 (gate) and W1 (up) and
// writes bf16(silu(gate) * up).  MODE 2: two consecutive 16-row tiles share
// every X fragment (used from two position blocks on).
// Wave w multiplies the k range [w K/8, (w+1) K/8): 16-row x 32-k W
// fragments (A) against the positions' X fragments (B) on
// v_mfma_f32_16x16x32_bf16, 8 / P k steps of loads issued before their
// products; at most 128 VGPRs, so that two workgroups share a CU and one
// streams while the other reduces.  Lane l's
// accumulator element i is row 4 (l / 16) + i of the tile for position
// l % 16, so one 16-byte store (or an 8-byte bf16 store) per lane writes four
// consecutive outputs.  The waves' partial sums are added in wave order.
// ---------------------------------------------------------------------------
template <int P, int MODE>
__global__ __launch_bounds__(kLinWaves * kWave, 2) void k_linear(
    const uint16_t* __restrict__ W0, const uint16_t* __restrict__ W1,
    const uint16_t* __restrict__ W2, int n0, int n1, int K, const uint16_t* __restrict__ X,
    int M, const float* __restrict__ R, int ldr, float* __restrict__ Y,
    uint16_t* __restrict__ Yb, int ldy) {
  constexpr bool GLU = MODE == 1, TWO = MODE == 2, DUAL = MODE != 0;
  constexpr int NW = DUAL ? 2 : 1;
  constexpr int RPW = TWO ? 2 * kTile : kTile;   // rows per workgroup
  constexpr int CH = 8 / P;                      // k steps per round of loads
  __shared__ floatx4 red[kLinWaves][NW * P][kWave];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, li = lane & 15;
  const int r0 = blockIdx.x * RPW, p0 = blockIdx.y * kTile * P;
  const int kw = K / kLinWaves, nks = kw / 32;
  const uint16_t* Wa = W0;
  int ra = r0;
  if (!GLU && r0 >= n0) {                        // workgroup-uniform
    if (r0 < n0 + n1) {
      Wa = W1;
      ra = r0 - n0;
    } else {
      Wa = W2;
      ra = r0 - n0 - n1;
    }
  }
  const uint16_t* wp0 = Wa + (size_t)(ra + li) * K + wave * kw + 8 * g;
  const uint16_t* wp1 = GLU   ? W1 + (size_t)(r0 + li) * K + wave * kw + 8 * g
                        : TWO ? wp0 + (size_t)kTile * K
                              : wp0;
  const uint16_t* xp[P];
  bool pv[P];
#pragma unroll
  for (int pb = 0; pb < P; ++pb) {
    const int p = p0 + kTile * pb + li;
    pv[pb] = p < M;
    xp[pb] = X + (size_t)(pv[pb] ? p : 0) * K + wave * kw + 8 * g;
  }
  floatx4 acc0[P], acc1[P];
#pragma unroll
  for (int pb = 0; pb < P; ++pb) acc0[pb] = acc1[pb] = floatx4{0.f, 0.f, 0.f, 0.f};
  const u32x4 zero{0u, 0u, 0u, 0u};
  for (int c = 0; c < nks; c += CH) {
    u32x4 a0[CH], a1[CH], b[CH][P];
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      const int ks = c + j < nks ? c + j : nks - 1;   // past the end: re-read, not used
      a0[j] = ld16(wp0 + 32 * ks);
      if constexpr (DUAL) a1[j] = ld16(wp1 + 32 * ks);
#pragma unroll
      for (int pb = 0; pb < P; ++pb) b[j][pb] = ld16(xp[pb] + 32 * ks);
    }
#pragma unroll
    for (int j = 0; j < CH; ++j)
      if (c + j < nks)
#pragma unroll
        for (int pb = 0; pb < P; ++pb) {
          const u32x4 bx = pv[pb] ? b[j][pb] : zero;
          acc0[pb] = Mfma<uint16_t>::mma(a0[j], bx, acc0[pb]);
          if constexpr (DUAL) acc1[pb] = Mfma<uint16_t>::mma(a1[j], bx, acc1[pb]);
        }
  }
#pragma unroll
  for (int pb = 0; pb < P; ++pb) {
    red[wave][pb][lane] = acc0[pb];
    if constexpr (DUAL) red[wave][P + pb][lane] = acc1[pb];
  }
  __syncthreads();
  if (wave < P) {                                // wave pb adds the 8 partials of block pb
    const int pb = wave;
    floatx4 s0 = red[0][pb][lane], s1{0.f, 0.f, 0.f, 0.f};
    if constexpr (DUAL) s1 = red[0][P + pb][lane];
#pragma unroll
    for (int w = 1; w < kLinWaves; ++w) {
      s0 += red[w][pb][lane];
      if constexpr (DUAL) s1 += red[w][P + pb][lane];
    }
    const int p = p0 + kTile * pb + li;
    if (p < M) {
      const int n = r0 + 4 * g;
      auto put = [&](floatx4 v, int nn) {
        if (R) v += *reinterpret_cast<const floatx4*>(R + (size_t)p * ldr + nn);
        if (Y) *reinterpret_cast<floatx4*>(Y + (size_t)p * ldy + nn) = v;
        if (Yb) {
          const uint32_t lo = f32_to_bf16_rne(v[0]) | ((uint32_t)f32_to_bf16_rne(v[1]) << 16);
          const uint32_t hi = f32_to_bf16_rne(v[2]) | ((uint32_t)f32_to_bf16_rne(v[3]) << 16);
          *reinterpret_cast<uint2*>(Yb + (size_t)p * ldy + nn) = make_uint2(lo, hi);
        }
      };
      if constexpr (GLU) {
#pragma unroll
        for (int e = 0; e < 4; ++e) s0[e] = s0[e] / (1.f + __expf(-s0[e])) * s1[e];
        put(s0, n);
      } else {
        put(s0, n);
        if constexpr (TWO) put(s1, n + kTile);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// The same projections for one block of up to 16 positions and K <= 4096, in
// the manner of the LM-head stream kernel (A1): x (16 positions x K) sits in
// LDS for the whole kernel; every wave takes a contiguous share of its
// workgroup's (16-row tile, 64-k group) items, loads each item with two
// line-complete instructions (8 rows x 128 B), transposes it through a 2 KB
// per-wave LDS tile into operand order and keeps PF items in flight.  A tile
// whose items straddle waves is finished at the end, its partial tiles added
// in wave order (= k order).  Rows of up to three stacked weights (boundaries
// multiples of 16).  Output: y[p][n] (+ R) row-major, fp32 and / or bf16.
// ---------------------------------------------------------------------------
constexpr int kGsWaves = 16;
constexpr int kGsPF = 5;                // items in flight per wave
constexpr int kGsXChunks = 512;         // 16-byte chunks of x per position (K <= 4096)

__device__ __forceinline__ int gs_slot(int row, int c) { return row * 8 + (c ^ ((row & 7) ^ (row >> 3))); }

__global__ __launch_bounds__(kGsWaves * kWave) void k_gemv_sk(
    const uint16_t* __restrict__ W0, const uint16_t* __restrict__ W1,
    const uint16_t* __restrict__ W2, int n0, int n1, int N, int K,
    const uint16_t* __restrict__ X, int M, int U, const float* __restrict__ R, int ldr,
    float* __restrict__ Y, uint16_t* __restrict__ Yb, int ldy) {
  __shared__ u32x4 lds[16 * kGsXChunks + kGsWaves * 128];     // x (128 KB) + transpose tiles
  u32x4* xl = lds;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  u32x4* tb = lds + 16 * kGsXChunks + wave * 128;
  const int u = blockIdx.x, ntiles = N / kTile;
  const int tlo = unit_tile_lo(u, ntiles, U), thi = unit_tile_lo(u + 1, ntiles, U);
  const int nch = K / 8, G = K / 64;                          // chunks per row, items per tile
  const int NI = (thi - tlo) * G;
  auto wlo = [&](int w) { return (int)(((long)w * NI) / kGsWaves); };
  const int i0 = wlo(wave), i1 = wlo(wave + 1);

  // x: every thread issues its (at most 8) chunk loads at once; positions
  // past M are loaded from position M - 1 and zeroed
  constexpr int kXPer = 16 * kGsXChunks / (kGsWaves * kWave);
  u32x4 xv[kXPer];
#pragma unroll
  for (int j = 0; j < kXPer; ++j) {
    int e = threadIdx.x + kGsWaves * kWave * j;
    e = e < 16 * nch ? e : 0;
    const int pr = e / nch;
    xv[j] = ld16(X + (size_t)(pr < M ? pr : M - 1) * K + (size_t)(e % nch) * 8);
  }
  // load role: 8 lanes per row, lane -> (row ri of 8, chunk lc of 8)
  const int ri = lane >> 3, lc = lane & 7;
  // MFMA role: row / position li, k-group g
  const int li = lane & 15, g = lane >> 4;
  const bool pact = li < M;
  // item counters of the next load: tile (relative) and k-group; frozen at the
  // wave's last item, so loads past the end re-read it
  int lt = G > 0 ? i0 / G : 0, lq = i0 - lt * G, ln = i0;
  auto load_item = [&](u32x4 (&r)[2]) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int row = (tlo + lt) * kTile + 8 * j + ri;
      const uint16_t* w = row < n0 ? W0 + (size_t)row * K
                        : row < n0 + n1 ? W1 + (size_t)(row - n0) * K
                                        : W2 + (size_t)(row - n0 - n1) * K;
      r[j] = ld16_nt(w + (size_t)(8 * lq + lc) * 8);
    }
    const int adv = ln + 1 < i1 ? 1 : 0;                  // scalar, branch-free
    ln += adv;
    lq += adv;
    const int wrap = lq == G ? 1 : 0;
    lq = wrap ? 0 : lq;
    lt += wrap;
  };
  auto finalize = [&](floatx4 acc, int t) {
    const int n = t * kTile + 4 * g;
    if (pact) {
      if (R) acc += *reinterpret_cast<const floatx4*>(R + (size_t)li * ldr + n);
      if (Y) *reinterpret_cast<floatx4*>(Y + (size_t)li * ldy + n) = acc;
      if (Yb) {
        const uint32_t lo = f32_to_bf16_rne(acc[0]) | ((uint32_t)f32_to_bf16_rne(acc[1]) << 16);
        const uint32_t hi = f32_to_bf16_rne(acc[2]) | ((uint32_t)f32_to_bf16_rne(acc[3]) << 16);
        *reinterpret_cast<uint2*>(Yb + (size_t)li * ldy + n) = make_uint2(lo, hi);
      }
    }
  };
  const int tf = G > 0 ? i0 / G : 0;                      // first (relative) tile of the wave
  floatx4 acc = {0.f, 0.f, 0.f, 0.f}, part0 = acc, part1 = acc;
  int ct = tf, cq = i0 - tf * G;                          // item being computed
  auto step = [&](const u32x4 (&r)[2], int i) {
#pragma unroll
    for (int j = 0; j < 2; ++j) tb[gs_slot(8 * j + ri, lc)] = r[j];
    wave_lds_order();
#pragma unroll
    for (int uu = 0; uu < 2; ++uu) {
      const int c = 4 * uu + g;
      const u32x4 a = tb[gs_slot(li, c)];
      const int cc = 8 * cq + c;
      const u32x4 b = xl[li * kGsXChunks + ((cc & ~15) | ((cc & 15) ^ li))];
      acc = Mfma<uint16_t>::mma(a, b, acc);
    }
    wave_lds_order();
    if (cq == G - 1 || i == i1 - 1) {                     // end of a tile segment
      if (cq == G - 1 && ct * G >= i0)
        finalize(acc, tlo + ct);
      else if (ct == tf)
        part0 = acc;
      else
        part1 = acc;
      acc = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    if (++cq == G) {
      cq = 0;
      ++ct;
    }
  };

  asm volatile("" ::: "memory");
  u32x4 ring[kGsPF][2];
  if (i0 < i1) {
#pragma unroll
    for (int q = 0; q < kGsPF; ++q) load_item(ring[q]);
  }
  asm volatile("" ::: "memory");
  // no guard on the stores (a guarded store would sink its load): chunks past
  // 16 * nch were loaded from chunk 0 and rewrite chunk 0's slot with its value
#pragma unroll
  for (int j = 0; j < kXPer; ++j) {
    int e = threadIdx.x + kGsWaves * kWave * j;
    e = e < 16 * nch ? e : 0;
    const int pp = e / nch, c = e % nch;
    xl[pp * kGsXChunks + ((c & ~15) | ((c & 15) ^ pp))] = pp < M ? xv[j] : u32x4{0u, 0u, 0u, 0u};
  }
  lds_barrier();                                          // x is in LDS; items stay in flight
  if (i0 < i1) {
    int i = i0;
    for (; i + kGsPF <= i1; i += kGsPF) {
#pragma unroll
      for (int q = 0; q < kGsPF; ++q) {
        step(ring[q], i + q);
        load_item(ring[q]);
      }
    }
#pragma unroll
    for (int q = 0; q < kGsPF; ++q)
      if (i + q < i1) step(ring[q], i + q);
  }
  // tiles split between waves: partial tiles through LDS (the x area is free)
  __syncthreads();
  floatx4* fx = reinterpret_cast<floatx4*>(lds);          // [wave][2][64]
  fx[(wave * 2 + 0) * 64 + lane] = part0;
  fx[(wave * 2 + 1) * 64 + lane] = part1;
  __syncthreads();
  if (i0 < i1) {
    const int tl = (i1 - 1) / G;
    int tfin = -1;
    floatx4 a = part0;
    if (i0 % G == 0 && i1 < (tf + 1) * G) {               // starts a tile it does not finish
      tfin = tf;
    } else if (tl > tf && i1 % G != 0) {                  // last tile started here, unfinished
      tfin = tl;
      a = part1;
    }
    if (tfin >= 0) {
      for (int w = wave + 1; w < kGsWaves && wlo(w) < (tfin + 1) * G; ++w) {
        if (wlo(w + 1) > wlo(w)) {
          const floatx4 o = fx[(w * 2 + 0) * 64 + lane];
          a[0] += o[0]; a[1] += o[1]; a[2] += o[2]; a[3] += o[3];
        }
      }
      finalize(a, tlo + tfin);
    }
  }
  __builtin_amdgcn_s_waitcnt(0x0070);                     // the re-read loads past the end
}

// ---------------------------------------------------------------------------
// QK-norm + RoPE: one workgroup per position m; wave w takes the head slots
// w, w + 4, ...: slots [0, nh) are the q heads, [nh, nh + nkv) the k heads,
// [nh + nkv, nh + 2 nkv) the v heads (converted only).  Lane l holds elements
// l and l + 64, the rotate-half pair of frequency l; the angle (taken in
// double) depends on the position and l only, so each wave forms its cosine
// and sine once for all its slots.  The row is P_0 + ... + P_{S-1}
// (P_s = qkv + s slab, added in that order; S = 1: the projection itself).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_qkrope(
    const float* __restrict__ qkv, int S, size_t slab, int ldq, int B, int nh, int nkv,
    const int32_t* __restrict__ ctx_len, int Cmax, const uint16_t* __restrict__ gq,
    const uint16_t* __restrict__ gk, float eps, float theta, uint16_t* __restrict__ qn,
    uint16_t* __restrict__ kb, uint16_t* __restrict__ vb) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m = blockIdx.x;
  const int nslots = nh + 2 * nkv;
  int C = ctx_len[m / B];
  C = C < 0 ? 0 : (C > Cmax ? Cmax : C);
  const double pos = (double)(C + m % B);
  const double ang = pos * pow((double)theta, -2.0 * (double)lane / (double)kHd);
  const float cs = (float)cos(ang), sn = (float)sin(ang);
  const float gq0 = bf16_to_f32(gq[lane]), gq1 = bf16_to_f32(gq[lane + 64]);
  const float gk0 = bf16_to_f32(gk[lane]), gk1 = bf16_to_f32(gk[lane + 64]);
  for (int hs = wave; hs < nslots; hs += 4) {
    const float* src = qkv + (size_t)m * ldq + (size_t)hs * kHd;
    float a = src[lane], b = src[lane + 64];
    for (int q = 1; q < S; ++q) {
      a += src[q * slab + lane];
      b += src[q * slab + lane + 64];
    }
    if (hs >= nh + nkv) {                        // wave-uniform
      uint16_t* dst = vb + ((size_t)m * nkv + (hs - nh - nkv)) * kHd;
      dst[lane] = f32_to_bf16_rne(a);
      dst[lane + 64] = f32_to_bf16_rne(b);
      continue;
    }
    const bool isq = hs < nh;
    const float ss = wave_sum(a * a + b * b);
    const float r = 1.f / sqrtf(ss / (float)kHd + eps);
    a = a * r * (isq ? gq0 : gk0);
    b = b * r * (isq ? gq1 : gk1);
    uint16_t* dst =
        isq ? qn + ((size_t)m * nh + hs) * kHd : kb + ((size_t)m * nkv + (hs - nh)) * kHd;
    dst[lane] = f32_to_bf16_rne(a * cs - b * sn);
    dst[lane + 64] = f32_to_bf16_rne(b * cs + a * sn);
  }
}

// ---------------------------------------------------------------------------
// Split-KV block attention, flash-decoding style.  Grid (chunk s, KV head,
// sequence b); wave w is query head kvh * GRP + w % GRP for the block
// positions 16 pb .. 16 pb + 15, pb = w / GRP (NPB position blocks), so the
// group's query heads and the block's positions share every K and V byte
// read.  A chunk is nsub sub-chunks of 64 keys, walked with an online softmax.
// Key kk of sequence b is context key kk (kk < C) or block key kk - C
// (C <= kk < C + B); keys from C + B on do not exist (their rows are loaded
// as the last key's and masked).
//
// K and V go from HBM straight into an NS-stage LDS ring (global_load_lds,
// 1 KB per instruction, no staging registers); a stage is the sub-chunk's 64
// K rows then its 64 V rows, 256 B each, the 16-byte chunk c of row r stored
// at position c ^ (r & 15), so that both reads below are free of bank
// conflicts.  S^T = K Q^T per 16-key tile (A: key rows, B: the wave's q):
// lane l holds keys 16 t + 4 (l / 16) + i for query l % 16.  With the
// running maximum m (per query) the numerators e = exp(s - m) enter O = P V
// as two bf16 parts: the A operand's eight k slots of lane l are its own e of
// tiles 2u and 2u + 1 (keys 32 u + 4 (l/16) + 0..3 and 32 u + 16 + 4 (l/16) +
// 0..3); the B operand takes V of the same keys with two transposing reads
// (ds_read_b64_tr_b16: in each 16-lane group, output lane i receives element
// i % 4 of the 8-byte reads of lanes 4 j + i / 4, j = 0..3, so when lane s
// reads 4 columns of key row k0 + s / 4, lane i receives keys k0 .. k0 + 3 of
// one column); the output lane holds queries 4 (l / 16) + i for
// d = 16 dt + l % 16.  The reference m of a query moves only when a score
// exceeds it by more than 2^8 (scores in base-2 units), and then O and l are
// rescaled by 2^(m_old - m_new).  Written per (chunk, query): O and l
// relative to the chunk's final reference m, and m.
// ---------------------------------------------------------------------------
constexpr int kSub = 64;                       // keys per sub-chunk (one LDS stage)
constexpr int kAttnSlots = 2 * kSub * kHd / 8; // 16-byte slots of a stage: K rows, then V rows

typedef short v4i16 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 lds_read_tr16(const uint16_t* p) {   // p: an LDS address
  const v4i16 r =
      __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)p);
  return __builtin_bit_cast(uint2, r);
}

// Waves of a workgroup: one per (query head of the group, position block),
// times KH = 2 key halves where that leaves at most eight (the two waves of a
// pair take keys 0..31 and 32..63 of every sub-chunk with their own running
// maximum, sum and O, merged at the end), so that a CU holds enough waves to
// hide each one's latency (with eight pairs the halves' extra registers cost
// more than they hide: measured).  The LDS ring has NS = 2 stages (64 KB, two
// workgroups per CU), 3 for 16 waves (96 KB, one workgroup per CU).
__host__ __device__ constexpr int attn_halves(int grp, int npb) { return grp * npb <= 4 ? 2 : 1; }
__host__ __device__ constexpr int attn_waves(int grp, int npb) {
  return grp * npb * attn_halves(grp, npb);
}
template <int GRP, int NPB>
struct AttnShape {
  static constexpr int KH = attn_halves(GRP, NPB);
  static constexpr int W = attn_waves(GRP, NPB);
  static constexpr int NS = W >= 16 ? 3 : 2;
};

// The PER loads of one wave for the sub-chunk starting at key k0 into the
// stage at `stage`: load e is instruction ins = wave PER + e of the stage,
// slots 64 ins .. + 63: K rows (ins < 16) or V rows 4 (ins % 16) + lane / 16,
// lane l bringing logical chunk (l % 16) ^ (row & 15) of its row (rows past
// the last key repeat it).
template <int PER>
__device__ __forceinline__ void attn_issue(u32x4* stage, int wave, int lane, int k0, int nkeys,
                                           int C, int B, int Cmax, int nkv, int kvh, int b,
                                           const uint16_t* kcache, const uint16_t* vcache,
                                           const uint16_t* kb, const uint16_t* vb) {
  const int lrow = lane >> 4, lpc = lane & 15;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int ins = wave * PER + e;
    const bool isv = ins >= 16;
    const int row = 4 * (ins & 15) + lrow;
    int kk = k0 + row;
    kk = kk < nkeys ? kk : nkeys - 1;
    const uint16_t* src =
        kk < C ? (isv ? vcache : kcache) + (((size_t)b * Cmax + kk) * nkv + kvh) * kHd
               : (isv ? vb : kb) + (((size_t)b * B + (kk - C)) * nkv + kvh) * kHd;
    lds_dma16(src + 8 * (lpc ^ (row & 15)), stage + 64 * ins);
  }
}

// One sub-chunk of the wave's keys (tiles t0 .. t0 + NT - 1 of the stage at
// Ks / Vs): S, the online softmax and O += P V.  Scores are kept in base-2
// units (q.k / sqrt(hd) times log2 e), so every exponential is one exp2.
template <int NT>
__device__ __forceinline__ void attn_step(const u32x4* Ks, const uint16_t* Vs,
                                          const u32x4 (&qf)[kHd / 32], int t0, int g, int li,
                                          bool qv, bool interior, int kb0, int nkeys, int C,
                                          int causal, int p, floatx4 (&o)[kHd / 16],
                                          float& m_run, float& l_run) {
  constexpr float kScale2 = 0.12751743082459868f;   // log2(e) / sqrt(128)
  floatx4 sc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int kr = kTile * (t0 + t) + li;         // A operand: key kr, d 32 ks + 8 g ..
    floatx4 acc{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < kHd / 32; ++ks)
      acc = Mfma<uint16_t>::mma(Ks[kr * 16 + ((4 * ks + g) ^ li)], qf[ks], acc);
    if (interior) {                               // workgroup-uniform
#pragma unroll
      for (int i = 0; i < 4; ++i) sc[t][i] = qv ? acc[i] * kScale2 : -INFINITY;
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = kb0 + kTile * (t0 + t) + 4 * g + i;
        const bool vis = qv && key < nkeys && (key < C || !causal || key - C <= p);
        sc[t][i] = vis ? acc[i] * kScale2 : -INFINITY;
      }
    }
  }
  // The reference maximum m_run of a query moves only when one of its
  // scores exceeds it by more than kLazy (base-2 units), so most sub-chunks
  // skip the rescale of O and l; the numerators are then at most 2^kLazy,
  // well inside fp32, and their bf16 parts keep the same relative precision.
  constexpr float kLazy = 8.f;
  float mt = -INFINITY;                           // the sub-chunk's row maximum
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) mt = fmaxf(mt, sc[t][i]);
  mt = fmax_xor32(fmax_xor16(mt));
  const bool grow = __ballot(mt > m_run + kLazy) != 0;   // wave-uniform
  const float mref = grow ? fmaxf(m_run, mt) : m_run;
  // with no visible key yet (mref = -inf) every exponent below is -inf: 0
  const float mxs = mref == -INFINITY ? 0.f : mref;
  // numerators as two bf16 parts (hi = bf16(e), lo = bf16(e - hi)); the
  // sum is taken over the same parts
  uint32_t eh[NT][2], el[NT][2];
  float lsum = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int i = 0; i < 4; i += 2) {
      const float e0 = __builtin_amdgcn_exp2f(sc[t][i] - mxs);
      const float e1 = __builtin_amdgcn_exp2f(sc[t][i + 1] - mxs);
      const uint32_t h = pk_bf16(e0, e1);
      const float h0 = __uint_as_float(h << 16), h1 = __uint_as_float(h & 0xFFFF0000u);
      const uint32_t lo = pk_bf16(e0 - h0, e1 - h1);
      const float l0 = __uint_as_float(lo << 16), l1 = __uint_as_float(lo & 0xFFFF0000u);
      lsum += h0 + l0;
      lsum += h1 + l1;
      eh[t][i / 2] = h;
      el[t][i / 2] = lo;
    }
  lsum = fadd_xor32(fadd_xor16(lsum));
  if (grow) {                                     // wave-uniform
    const float alpha = __builtin_amdgcn_exp2f(m_run - mxs);
    l_run = l_run * alpha + lsum;
    // O rows are queries 4 (l / 16) + i: their factors come from lanes 4 g + i
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float ai = __shfl(alpha, 4 * g + i, kWave);
#pragma unroll
      for (int dt = 0; dt < kHd / 16; ++dt) o[dt][i] *= ai;
    }
  } else {
    l_run += lsum;
  }
  m_run = mref;
  // V reads: lane (g, li) supplies key row k0 + li / 4 (k0 = 32 u + 4 g,
  // then + 16), columns 16 dt + 4 (li % 4) .. + 3: chunk 2 dt + (li % 4) / 2,
  // half (li % 4) & 1
  const int vr = li >> 2, vc = (li & 3) >> 1, vh = 4 * (li & 1);
#pragma unroll
  for (int u = 0; u < NT / 2; ++u) {
    const u32x4 ph{eh[2 * u][0], eh[2 * u][1], eh[2 * u + 1][0], eh[2 * u + 1][1]};
    const u32x4 pl{el[2 * u][0], el[2 * u][1], el[2 * u + 1][0], el[2 * u + 1][1]};
    const int r0 = kTile * t0 + 32 * u + 4 * g + vr, r1 = r0 + 16;
#pragma unroll
    for (int dt = 0; dt < kHd / 16; ++dt) {
      const int c = 2 * dt + vc;
      const uint2 v0 = lds_read_tr16(Vs + 8 * (r0 * 16 + (c ^ (r0 & 15))) + vh);
      const uint2 v1 = lds_read_tr16(Vs + 8 * (r1 * 16 + (c ^ (r1 & 15))) + vh);
      const u32x4 vvv{v0.x, v0.y, v1.x, v1.y};
      o[dt] = Mfma<uint16_t>::mma(pl, vvv, o[dt]);
      o[dt] = Mfma<uint16_t>::mma(ph, vvv, o[dt]);
    }
  }
}

template <int GRP, int NPB>
__global__ __launch_bounds__(attn_waves(GRP, NPB) * kWave) void k_attn(
    const uint16_t* __restrict__ qn, const uint16_t* __restrict__ kcache,
    const uint16_t* __restrict__ vcache, const uint16_t* __restrict__ kb,
    const uint16_t* __restrict__ vb, const int32_t* __restrict__ ctx_len, int Cmax, int B,
    int nh, int nkv, int causal, int ns, int nsub, float* __restrict__ opart,
    float* __restrict__ mlpart) {
  using SH = AttnShape<GRP, NPB>;
  constexpr int W = SH::W, NS = SH::NS, KH = SH::KH;
  constexpr int PER = kAttnSlots / 64 / W;       // 1 KB loads per wave per stage
  static_assert(PER * W * 64 == kAttnSlots && 16 % PER == 0, "loads per stage, K or V per wave");
  static_assert((NS - 2) * PER < 64, "vmcnt field");
  constexpr int NT = kSub / kTile / KH;          // 16-key tiles per wave per sub-chunk
  static_assert(NT % 2 == 0, "tiles come in pairs");
  constexpr int kMerge = kTile * kHd + 2 * kTile;                // floats per pair
  static_assert(KH == 1 || GRP * NPB * kMerge * 4 <= NS * kAttnSlots * 16, "merge in LDS");
  __shared__ u32x4 lds[NS * kAttnSlots];
  const int s = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int pair = wave % (GRP * NPB), kh = wave / (GRP * NPB);
  const int hw = pair % GRP, pb = pair / GRP;
  const int t0 = kh * NT;                        // first tile of the wave's keys
  const int g = lane >> 4, li = lane & 15;
  int C = ctx_len[b];
  C = C < 0 ? 0 : (C > Cmax ? Cmax : C);
  const int nkeys = C + B, kbase = s * kSub * nsub;
  const size_t pidx = ((((size_t)b * NPB + pb) * nkv + kvh) * ns + s) * GRP + hw;
  float* op = opart + pidx * (kTile * kHd);
  float* ml = mlpart + pidx * (2 * kTile);
  if (kbase >= nkeys) {                          // whole workgroup: no key in this chunk
    if (kh == 0 && lane < kTile) {
      ml[2 * lane] = -INFINITY;
      ml[2 * lane + 1] = 0.f;
    }
    return;
  }
  const int left = (nkeys - kbase + kSub - 1) / kSub;
  const int nj = left < nsub ? left : nsub;      // sub-chunks holding keys (>= 1)

  // the wave's q (B operand): query li of block pb, head kvh * GRP + hw
  const int p = pb * kTile + li;
  const bool qv = p < B;
  const uint16_t* qs =
      qn + (((size_t)b * B + (qv ? p : 0)) * nh + (size_t)kvh * GRP + hw) * kHd + 8 * g;
  u32x4 qf[kHd / 32];
#pragma unroll
  for (int ks = 0; ks < kHd / 32; ++ks) qf[ks] = qv ? ld16(qs + 32 * ks) : u32x4{0u, 0u, 0u, 0u};

  // Loads of sub-chunks inside the context: the wave's rows (K or V, one
  // kind per wave) at a per-lane address plus the sub-chunk's first key
  // times the key stride; other sub-chunks take attn_issue's general path.
  const size_t kst = (size_t)nkv * kHd;           // elements per key row
  const uint16_t* lp[PER];
  {
    const bool isv = wave * PER >= 16;
    const uint16_t* cb = (isv ? vcache : kcache) + ((size_t)b * Cmax * nkv + kvh) * kHd;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int row = 4 * ((wave * PER + e) & 15) + (lane >> 4);
      lp[e] = cb + (size_t)row * kst + 8 * ((lane & 15) ^ (row & 15));
    }
  }
  __builtin_amdgcn_s_waitcnt(0x0070);            // q landed: from here vmcnt counts the ring

  float m_run = -INFINITY, l_run = 0.f;          // per query li, base-2 units
  floatx4 o[kHd / 16];
#pragma unroll
  for (int dt = 0; dt < kHd / 16; ++dt) o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};

  // sub-chunk j (clamped to the last) into ring slot `slot` (0 <= slot < NS);
  // both arguments are evaluated once, before the macro's own loop
#define XP_ATTN_ISSUE(j, slot)                                                                \
  do {                                                                                        \
    const int j_ = (j), slot_ = (slot);                                                       \
    const int k0_ = kbase + (j_ < nj ? j_ : nj - 1) * kSub;                                   \
    u32x4* st_ = lds + slot_ * kAttnSlots;                                                    \
    if (k0_ + kSub <= C) {                                                                    \
      _Pragma("unroll") for (int e_ = 0; e_ < PER; ++e_)                                      \
        lds_dma16(lp[e_] + (size_t)k0_ * kst, st_ + 64 * (wave * PER + e_));                  \
    } else {                                                                                  \
      attn_issue<PER>(st_, wave, lane, k0_, nkeys, C, B, Cmax, nkv, kvh, b, kcache, vcache,   \
                      kb, vb);                                                                \
    }                                                                                         \
  } while (0)
#pragma unroll
  for (int jp = 0; jp < NS - 1; ++jp) XP_ATTN_ISSUE(jp, jp);
  constexpr int kWait = (NS - 2) * PER;          // this wave's loads of the NS - 2 later stages
  for (int j0 = 0; j0 < nj; j0 += NS) {
#pragma unroll
    for (int sl = 0; sl < NS; ++sl) {            // ring slot sl holds sub-chunk j0 + sl
      const int j = j0 + sl;
      if (j < nj) {                              // workgroup-uniform
        // sub-chunk j landed (every wave's loads) and every wave is done
        // with j - 1, whose slot then takes sub-chunk j + NS - 1
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0x0070 | (kWait & 15) | ((kWait >> 4) << 14));
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        XP_ATTN_ISSUE(j + NS - 1, (sl + NS - 1) % NS);
        const u32x4* Ks = lds + sl * kAttnSlots;
        const int kb0 = kbase + j * kSub;
        attn_step<NT>(Ks, reinterpret_cast<const uint16_t*>(Ks + kAttnSlots / 2), qf, t0, g, li,
                      qv, kb0 + kSub <= C, kb0, nkeys, C, causal, p, o, m_run, l_run);
      }
    }
  }
#undef XP_ATTN_ISSUE
  __builtin_amdgcn_s_waitcnt(0x0070);            // the clamped loads past the last sub-chunk
  if constexpr (KH == 2) {
    // the second key half hands (m, l, O) to the first through the ring's
    // LDS: O' = 2^(m0 - M) O0 + 2^(m1 - M) O1, l likewise, M = max(m0, m1)
    __syncthreads();                             // every wave's loads landed and reads done
    float* mg = reinterpret_cast<float*>(lds) + pair * kMerge;
    if (kh == 1) {
#pragma unroll
      for (int dt = 0; dt < kHd / 16; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) mg[(4 * g + i) * kHd + 16 * dt + li] = o[dt][i];
      if (lane < kTile) {
        mg[kTile * kHd + lane] = m_run;
        mg[kTile * kHd + kTile + lane] = l_run;
      }
    }
    __syncthreads();
    if (kh == 1) return;                         // whole wave; no barrier follows
    const float m1 = mg[kTile * kHd + li], l1 = mg[kTile * kHd + kTile + li];
    const float M = fmaxf(m_run, m1);
    const float Ms = M == -INFINITY ? 0.f : M;
    const float f0 = __builtin_amdgcn_exp2f(m_run - Ms), f1 = __builtin_amdgcn_exp2f(m1 - Ms);
    l_run = f0 * l_run + f1 * l1;
    m_run = M;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a0 = __shfl(f0, 4 * g + i, kWave), a1 = __shfl(f1, 4 * g + i, kWave);
#pragma unroll
      for (int dt = 0; dt < kHd / 16; ++dt)
        o[dt][i] = a0 * o[dt][i] + a1 * mg[(4 * g + i) * kHd + 16 * dt + li];
    }
  }
#pragma unroll
  for (int dt = 0; dt < kHd / 16; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) op[(4 * g + i) * kHd + 16 * dt + li] = o[dt][i];
  if (lane < kTile) {
    ml[2 * lane] = m_run;
    ml[2 * lane + 1] = l_run;
  }
}

// One wave per (position m, query head h): merge the chunks in order,
// attn = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s, to bf16 (m in the
// base-2 units of k_attn).  Lane j
// takes the (m, l) of chunk s0 + j; the O rows are then read eight chunks at a
// time and added in chunk order.  A chunk whose l is 0 (no visible key; its O
// may be unwritten) contributes nothing.
__global__ __launch_bounds__(256) void k_attn_comb(const float* __restrict__ opart,
                                                   const float* __restrict__ mlpart, int M, int B,
                                                   int npb, int nh, int nkv, int grp, int ns,
                                                   uint16_t* __restrict__ attn) {
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= M * nh) return;                       // whole wave
  const int m = w / nh, h = w - m * nh;
  const int b = m / B, p = m - b * B, pb = p / kTile, q = p - pb * kTile;
  const int kvh = h / grp, wv = h - kvh * grp, z = b * npb + pb;
  const size_t base = (((size_t)z * nkv + kvh) * ns) * grp + wv;
  auto mlv = [&](int s, float& ms, float& ls) {
    if (s < ns) {
      const size_t pi = base + (size_t)s * grp;
      ms = mlpart[pi * 2 * kTile + 2 * q];
      ls = mlpart[pi * 2 * kTile + 2 * q + 1];
    } else {
      ms = -INFINITY;
      ls = 0.f;
    }
  };
  float mm = -INFINITY;
  for (int s0 = 0; s0 < ns; s0 += kWave) {
    float ms, ls;
    mlv(s0 + lane, ms, ls);
    if (ls > 0.f) mm = fmaxf(mm, ms);
  }
#pragma unroll
  for (int k = 32; k >= 1; k >>= 1) mm = fmaxf(mm, __shfl_xor(mm, k, kWave));
  float Ll = 0.f, o0 = 0.f, o1 = 0.f;
  for (int s0 = 0; s0 < ns; s0 += kWave) {
    float ms, ls;
    mlv(s0 + lane, ms, ls);
    const float f = ls > 0.f ? __builtin_amdgcn_exp2f(ms - mm) : 0.f;
    Ll += f * ls;
    const int cnt = ns - s0 < kWave ? ns - s0 : kWave;
    for (int j0 = 0; j0 < cnt; j0 += 8) {
      float fj[8], v0[8], v1[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + u < cnt ? j0 + u : cnt - 1;
        fj[u] = __shfl(f, j, kWave);
        if (j0 + u >= cnt) fj[u] = 0.f;
        const size_t pi = base + (size_t)(s0 + j) * grp;
        v0[u] = opart[pi * (kTile * kHd) + q * kHd + lane];
        v1[u] = opart[pi * (kTile * kHd) + q * kHd + lane + 64];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        o0 += fj[u] != 0.f ? fj[u] * v0[u] : 0.f;
        o1 += fj[u] != 0.f ? fj[u] * v1[u] : 0.f;
      }
    }
  }
  const float L = wave_sum(Ll);
  const float inv = L > 0.f ? 1.f / L : 0.f;     // L > 0: every query sees its own key
  uint16_t* dst = attn + (size_t)m * nh * kHd + (size_t)h * kHd;
  dst[lane] = f32_to_bf16_rne(o0 * inv);
  dst[lane + 64] = f32_to_bf16_rne(o1 * inv);
}

// silu(gate) * up to bf16, gate and up side by side in one row of 2 F
// (the GEMM path computes both projections in one launch)
__global__ __launch_bounds__(256) void k_swiglu(const float* __restrict__ GU, int F, size_t n,
                                                uint16_t* __restrict__ act) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const size_t m = i / F, j = i - m * F;
  const float gv = GU[m * 2 * F + j], uv = GU[m * 2 * F + F + j];
  act[i] = f32_to_bf16_rne(silu_mul(gv, uv));
}

// y = (P_0 + ... + P_{S-1}) + R, added in that order, P_s = P + s n (the
// split-K slabs of a projection, rows of N); Y fp32 and Yb bf16 if given.
// Four consecutive elements per thread.
__global__ __launch_bounds__(256) void k_splitk_sum(const float* __restrict__ P, int S, size_t n,
                                                    const float* __restrict__ R,
                                                    float* __restrict__ Y,
                                                    uint16_t* __restrict__ Yb) {
  const size_t i = 4 * ((size_t)blockIdx.x * 256 + threadIdx.x);
  if (i >= n) return;
  floatx4 v = *reinterpret_cast<const floatx4*>(P + i);
  for (int q = 1; q < S; ++q) v += *reinterpret_cast<const floatx4*>(P + q * n + i);
  v += *reinterpret_cast<const floatx4*>(R + i);
  if (Y) *reinterpret_cast<floatx4*>(Y + i) = v;
  if (Yb)
    *reinterpret_cast<uint2*>(Yb + i) =
        make_uint2(f32_to_bf16_rne(v[0]) | ((uint32_t)f32_to_bf16_rne(v[1]) << 16),
                   f32_to_bf16_rne(v[2]) | ((uint32_t)f32_to_bf16_rne(v[3]) << 16));
}

}  // namespace xp

using namespace xp;

// Device buffers of one forward (a layer's workspace, or the static scratch
// of the allocation-free entry point).
struct LayerBufs {
  float* x32 = nullptr;              // [M][H]    x in fp32 (residual of Wo)
  uint16_t* u = nullptr;             // [M][H]    RMSNorm(x) g_attn, then RMSNorm(x1) g_mlp
  float* qkv = nullptr;              // [M][nhd + 2 kvd]
  uint16_t *qn = nullptr, *kb = nullptr, *vb = nullptr;   // normed, rotated q, k; v
  float *opart = nullptr, *mlpart = nullptr;              // attention chunk partials
  uint16_t* attn = nullptr;          // [M][nhd]
  float *x1 = nullptr, *h32 = nullptr, *GU = nullptr;     // GU: [gu_rows][2 F] gate | up
  uint16_t* act = nullptr;           // [M][F]    SwiGLU activation
  float* part = nullptr;             // split-K slabs of one projection (NULL: no split)
  size_t nparts = 0;                 // attention partials the buffers hold
  size_t gu_rows = 0;                // positions GU holds
  size_t part_floats = 0;            // floats `part` holds
};

struct xp_layer {
  int H, nh, nkv, ffn, grp;
  float eps, theta;
  const uint16_t *g_attn, *Wq, *Wk, *Wv, *g_q, *g_k, *Wo, *g_mlp, *Wg, *Wu, *Wd;
  int max_batch = 0, max_B = 0, max_ctx = 0;
  void* ws = nullptr;                // the workspace allocation (NULL: static scratch)
  LayerBufs b;
  std::string err;                   // message of the last failed call
};

// Message of the last failed xp_layer_create or xp_layer_forward_noalloc of
// this thread (calls without a layer to hold it).
static thread_local std::string g_layer_err;

static xp_status layer_fail(xp_layer* L, xp_status s, const char* fmt, ...)
    __attribute__((format(printf, 3, 4)));
static xp_status layer_fail(xp_layer* L, xp_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  (L ? L->err : g_layer_err) = buf;
  return s;
}

extern "C" const char* xp_layer_last_error(const xp_layer* L) {
  return L ? L->err.c_str() : g_layer_err.c_str();
}

static int attn_chunks(int C_max, int B, int keys) { return (C_max + B + keys - 1) / keys; }

// Checks the weight set and copies it into *L (shapes and pointers only).
// Errors are reported through layer_fail(nullptr, ...).
static xp_status layer_weights(const xp_layer_weights* w, xp_layer* L) {
  if (w == nullptr) return layer_fail(nullptr, XP_EINVAL, "weights is NULL");
  const void* ptrs[] = {w->g_attn, w->Wq, w->Wk, w->Wv, w->g_q, w->g_k,
                        w->Wo,     w->g_mlp, w->Wg, w->Wu, w->Wd};
  const char* names[] = {"g_attn", "Wq", "Wk", "Wv", "g_q", "g_k", "Wo", "g_mlp", "Wg", "Wu", "Wd"};
  for (int i = 0; i < 11; ++i)
    if (ptrs[i] == nullptr || reinterpret_cast<uintptr_t>(ptrs[i]) % 16 != 0)
      return layer_fail(nullptr, XP_EINVAL, "weight %s is NULL or not 16-byte aligned", names[i]);
  if (w->H < 1 || w->n_heads < 1 || w->n_kv < 1 || w->ffn < 1 || w->head_dim < 1 ||
      !(w->eps >= 0.f) || !(w->rope_theta > 0.f))
    return layer_fail(nullptr, XP_EINVAL,
                      "sizes must be positive, eps >= 0 and rope_theta > 0 (H=%d heads=%d kv=%d "
                      "head_dim=%d ffn=%d)", w->H, w->n_heads, w->n_kv, w->head_dim, w->ffn);
  const int grp = w->n_heads / w->n_kv;
  if (w->head_dim != kHd || w->n_heads % w->n_kv != 0 ||
      (grp != 1 && grp != 2 && grp != 4 && grp != 8) || w->H % 256 != 0 || w->H > 8192 ||
      (w->n_heads * kHd) % 256 != 0 || w->ffn % 256 != 0 || w->ffn > (1 << 16))
    return layer_fail(nullptr, XP_EUNSUPPORTED,
                      "shape not built: head_dim %d (128), heads/kv %d/%d (group 1, 2, 4 or 8), "
                      "H %d and heads*128 multiples of 256 with H <= 8192, ffn %d a multiple of 256 "
                      "up to 65536", w->head_dim, w->n_heads, w->n_kv, w->H, w->ffn);
  L->H = w->H;
  L->nh = w->n_heads;
  L->nkv = w->n_kv;
  L->ffn = w->ffn;
  L->grp = grp;
  L->eps = w->eps;
  L->theta = w->rope_theta;
  L->g_attn = (const uint16_t*)w->g_attn;
  L->Wq = (const uint16_t*)w->Wq;
  L->Wk = (const uint16_t*)w->Wk;
  L->Wv = (const uint16_t*)w->Wv;
  L->g_q = (const uint16_t*)w->g_q;
  L->g_k = (const uint16_t*)w->g_k;
  L->Wo = (const uint16_t*)w->Wo;
  L->g_mlp = (const uint16_t*)w->g_mlp;
  L->Wg = (const uint16_t*)w->Wg;
  L->Wu = (const uint16_t*)w->Wu;
  L->Wd = (const uint16_t*)w->Wd;
  return XP_OK;
}

// Every projection addresses rows of its input as (position * K) in 32 bits.
static bool rows_fit_int32(const xp_layer& L, int64_t positions) {
  const int64_t widest = std::max<int64_t>({(int64_t)L.H, (int64_t)L.nh * kHd, (int64_t)L.ffn});
  return positions * widest < ((int64_t)1 << 31);
}

// The gate/up projections write fp32 [M][2 F] to GU on the stream kernel's
// path only (calls of at most one 16-position block, H within its LDS copy of
// x); the tiled GEMM and k_linear form the SwiGLU product themselves.
static size_t gu_rows_for(const xp_layer& L, size_t Mx) {
  return (size_t)L.H <= 8 * (size_t)kGsXChunks ? std::min(Mx, (size_t)kTile) : 0;
}

// Split-K slabs are used by the tiled GEMM only (calls above kLinMaxStream
// positions); their size is bounded independently of M.
static size_t part_floats_for(size_t Mx) {
  return Mx > (size_t)kLinMaxStream ? kLayerPartFloats : 0;
}

// Lays out the buffers for up to Mx positions and nparts attention partials
// from `base` (256-byte aligned slices); returns the bytes used.  With
// base == nullptr only the size is computed.
static size_t carve(const xp_layer& L, size_t Mx, size_t nparts, size_t gu_rows,
                    size_t part_floats, char* base, LayerBufs* b) {
  const size_t H = L.H, nhd = (size_t)L.nh * kHd, kvd = (size_t)L.nkv * kHd, F = L.ffn;
  LayerBufs t;
  t.nparts = nparts;
  t.gu_rows = gu_rows;
  t.part_floats = part_floats;
  struct Slice {
    void** p;
    size_t bytes;
  } sl[] = {
      {(void**)&t.x32, Mx * H * 4},           {(void**)&t.u, Mx * H * 2},
      {(void**)&t.qkv, Mx * (nhd + 2 * kvd) * 4}, {(void**)&t.qn, Mx * nhd * 2},
      {(void**)&t.kb, Mx * kvd * 2},          {(void**)&t.vb, Mx * kvd * 2},
      {(void**)&t.opart, nparts * kTile * kHd * 4}, {(void**)&t.mlpart, nparts * 2 * kTile * 4},
      {(void**)&t.attn, Mx * nhd * 2},        {(void**)&t.x1, Mx * H * 4},
      {(void**)&t.act, Mx * F * 2},           {(void**)&t.h32, Mx * H * 4},
      {(void**)&t.GU, (gu_rows ? gu_rows : 1) * 2 * F * 4},
      {(void**)&t.part, (part_floats ? part_floats : 1) * 4},
  };
  size_t off = 0;
  for (auto& q : sl) {
    if (base) *q.p = base + off;
    off += (q.bytes + 255) / 256 * 256;
  }
  if (part_floats == 0) t.part = nullptr;
  if (base && b) *b = t;
  return off;
}

// Attention chunking of one call: chunks of nsub 64-key sub-chunks, about
// kAttnWgs workgroups (sequence, KV head, chunk) in all (one sub-chunk each
// at small calls), so that the partials stay few.  Returns the partial count
// batch * npb * nkv * ns * grp.
struct AttnPlan {
  int nsub, ns;
  size_t parts;
};
static AttnPlan attn_plan(const xp_layer& L, int batch, int B, int C_max, int nsub) {
  const int npb = (B + kTile - 1) / kTile;
  const int ns = attn_chunks(C_max, B, kSub * nsub);
  return {nsub, ns, (size_t)batch * npb * L.nkv * ns * L.grp};
}
static AttnPlan attn_plan_default(const xp_layer& L, int batch, int B, int C_max) {
  const size_t w64 = (size_t)batch * L.nkv * attn_chunks(C_max, B, kSub);
  int nsub = (int)(w64 / kAttnWgs);
  nsub = nsub < 1 ? 1 : (nsub > 256 ? 256 : nsub);
  return attn_plan(L, batch, B, C_max, nsub);
}

extern "C" xp_status xp_layer_create(const xp_layer_weights* w, int32_t max_batch, int32_t max_B,
                                     int32_t max_ctx, xp_layer** out) {
  g_layer_err.clear();
  if (out == nullptr) return layer_fail(nullptr, XP_EINVAL, "out is NULL");
  *out = nullptr;
  if (max_batch < 1 || max_batch > 4096 || max_B < 1 || max_B > 32 || max_ctx < 0 ||
      max_ctx > (1 << 20))
    return layer_fail(nullptr, XP_EINVAL,
                      "max_batch=%d (1..4096), max_B=%d (1..32) or max_ctx=%d (0..2^20) out of range",
                      max_batch, max_B, max_ctx);
  xp_layer tmp;
  const xp_status ws = layer_weights(w, &tmp);
  if (ws != XP_OK) return ws;
  if (!rows_fit_int32(tmp, (int64_t)max_batch * max_B))
    return layer_fail(nullptr, XP_EUNSUPPORTED,
                      "max_batch*max_B*max(H, heads*128, ffn) reaches 2^31 (max_batch=%d max_B=%d)",
                      max_batch, max_B);
  xp_layer* L = new (std::nothrow) xp_layer(tmp);
  if (L == nullptr) return layer_fail(nullptr, XP_ENOMEM, "host allocation failed");
  L->max_batch = max_batch;
  L->max_B = max_B;
  L->max_ctx = max_ctx;
  const size_t Mx = (size_t)max_batch * max_B;
  // attention partials: a call has at most max(2 kAttnWgs, w64 / 256) + one
  // per (sequence, KV head) chunks, w64 its (sequence, KV head, 64-key
  // sub-chunk) triples, and npb grp partials per chunk
  const size_t qmax = (size_t)max_batch * L->nkv, npbmax = (max_B + kTile - 1) / kTile;
  const size_t w64max = qmax * (size_t)attn_chunks(max_ctx, max_B, kSub);
  const size_t nparts =
      (std::max((size_t)2 * kAttnWgs, (w64max + 255) / 256) + qmax) * npbmax * L->grp;
  const size_t gu = gu_rows_for(*L, Mx), pf = part_floats_for(Mx);
  const size_t total = carve(*L, Mx, nparts, gu, pf, nullptr, nullptr);
  const hipError_t e = hipMalloc(&L->ws, total);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    delete L;
    return layer_fail(nullptr, XP_ENOMEM, "workspace of %zu bytes: %s", total,
                      hipGetErrorString(e));
  }
  carve(*L, Mx, nparts, gu, pf, static_cast<char*>(L->ws), &L->b);
  *out = L;
  return XP_OK;
}

extern "C" void xp_layer_destroy(xp_layer* L) {
  if (L == nullptr) return;
  (void)hipDeviceSynchronize();
  if (L->ws) (void)hipFree(L->ws);
  delete L;
}

// y [M][N] (row stride ldy) = X [M][K] W^T (+ R), W the rows of W0 | W1 | W2
// stacked (n0, n1 rows of the first two); glu: bf16(silu(X W0^T) * (X W1^T))
// to Yb.  With `splits` given the tiled GEMM may cut k into S > 1 parts: it
// then writes the fp32 partial products to the S slabs of b.part ([S][M][N],
// no residual, no Yb) and sets *splits = S, and the caller adds them (with R);
// else *splits = 1 and y is written.  Returns the first failed launch's
// error; hipErrorInvalidValue if GU is too small for the path taken.
static hipError_t linear(const LayerBufs& b, const uint16_t* W0, const uint16_t* W1,
                         const uint16_t* W2, int n0, int n1, int N, int K, const uint16_t* X,
                         int M, const float* R, int ldr, float* Y, uint16_t* Yb, int ldy,
                         bool glu, int* splits, hipStream_t st) {
  if (splits) *splits = 1;
  // one block of positions and x small enough for LDS: the stream-K kernel
  // (gate and up side by side, then SwiGLU)
  if (M <= kTile && K <= 8 * kGsXChunks && K % 64 == 0 && N % kTile == 0 && n0 % kTile == 0 &&
      n1 % kTile == 0) {
    const int rows = glu ? 2 * N : N, ntl = rows / kTile;
    const int U = ntl < 256 ? ntl : 256;
    if (glu) {
      if ((size_t)M > b.gu_rows) return hipErrorInvalidValue;
      hipLaunchKernelGGL(k_gemv_sk, dim3(U), dim3(kGsWaves * kWave), 0, st, W0, W1, W1, N, N,
                         2 * N, K, X, M, U, (const float*)nullptr, 0, b.GU, (uint16_t*)nullptr,
                         2 * N);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      const size_t na = (size_t)M * N;
      hipLaunchKernelGGL(k_swiglu, dim3((unsigned)((na + 255) / 256)), dim3(256), 0, st, b.GU, N,
                         na, Yb);
    } else {
      hipLaunchKernelGGL(k_gemv_sk, dim3(U), dim3(kGsWaves * kWave), 0, st, W0, W1, W2, n0, n1,
                         N, K, X, M, U, R, ldr, Y, Yb, ldy);
    }
    return hipGetLastError();
  }
  // above one 64-position pass of the stream: the tiled GEMM (weights read
  // once per 128 or 256 positions)
  if (M > kLinMaxStream) {
    const size_t pf = splits && b.part ? b.part_floats : 0;   // no slabs: S = 1
    const LayerPlan pl = glu ? layer_plan(N, N, 2 * N, K, M, true, 0)
                             : layer_plan(n0, n1, N, K, M, false, pf);
    if (pl.bn != 0) {
      if (glu) return launch_layer_glu(pl, W0, W1, N, K, X, M, Yb, ldy, st);
      if (pl.S > 1) {
        *splits = pl.S;
        return launch_layer_gemm(pl, W0, W1, W2, n0, n1, N, K, X, M, nullptr, 0, b.part, nullptr,
                                 N, st);
      }
      return launch_layer_gemm(pl, W0, W1, W2, n0, n1, N, K, X, M, R, ldr, Y, Yb, ldy, st);
    }
  }
  const int nb = (M + kTile - 1) / kTile;
  const int P = nb >= 4 ? 4 : (nb >= 2 ? 2 : 1);
  // two row tiles per workgroup (stacked row counts are multiples of 32) once
  // several position blocks reuse each X fragment; one at a single block,
  // where the workgroup count matters more
  const int mode = glu ? 1 : (P > 1 ? 2 : 0);
  const dim3 grid(N / (mode == 2 ? 2 * kTile : kTile), (M + kTile * P - 1) / (kTile * P)),
      block(kLinWaves * kWave);
#define XP_LIN(PP, MM)                                                                        \
  hipLaunchKernelGGL((k_linear<PP, MM>), grid, block, 0, st, W0, W1, W2, n0, n1, K, X, M, R, \
                     ldr, Y, Yb, ldy)
  if (glu) {
    if (P == 4) XP_LIN(4, 1);
    else if (P == 2) XP_LIN(2, 1);
    else XP_LIN(1, 1);
  } else {
    if (P == 4) XP_LIN(4, 2);
    else if (P == 2) XP_LIN(2, 2);
    else XP_LIN(1, 0);
  }
#undef XP_LIN
  return hipGetLastError();
}

// Argument checks of a forward call, shared by both entry points.
static xp_status check_call(xp_layer* Lerr, int32_t batch, int32_t B, int32_t causal,
                            const void* x, const void* k_cache, const void* v_cache,
                            int32_t C_max, const int32_t* ctx_len, const float* h_f32,
                            const void* h_bf16) {
  if (x == nullptr || k_cache == nullptr || v_cache == nullptr || ctx_len == nullptr)
    return layer_fail(Lerr, XP_EINVAL, "x, k_cache, v_cache and ctx_len are required");
  if (causal != 0 && causal != 1) return layer_fail(Lerr, XP_EINVAL, "causal=%d is not 0 or 1", causal);
  if (batch < 1 || B < 1 || B > 32 || C_max < 1 || C_max > (1 << 20))
    return layer_fail(Lerr, XP_EINVAL, "batch=%d, B=%d (1..32) or C_max=%d (1..2^20) out of range",
                      batch, B, C_max);
  const char* pn[] = {"x", "k_cache", "v_cache", "h_f32", "h_bf16"};
  const void* pv[] = {x, k_cache, v_cache, (const void*)h_f32, h_bf16};
  for (int i = 0; i < 5; ++i)
    if (reinterpret_cast<uintptr_t>(pv[i]) % 16 != 0)
      return layer_fail(Lerr, XP_EINVAL, "%s is not 16-byte aligned", pn[i]);
  return XP_OK;
}

// The launch sequence of one forward over `batch` blocks of B positions with
// the attention chunking `ap`, on the buffers `b` (which hold at least the
// call's positions and ap.parts partials).  Errors go to Lerr (NULL: the
// thread's message).
static xp_status forward(const xp_layer& L, const LayerBufs& b, const AttnPlan& ap,
                         xp_layer* Lerr, int32_t batch, int32_t B, int32_t causal, const void* x,
                         const void* k_cache, const void* v_cache, int32_t C_max,
                         const int32_t* ctx_len, float* h_f32, void* h_bf16, hipStream_t st) {
  const int M = batch * B, H = L.H, nh = L.nh, nkv = L.nkv, F = L.ffn, grp = L.grp;
  const int nhd = nh * kHd, kvd = nkv * kHd, ldq = nhd + 2 * kvd;
  const int npb = (B + kTile - 1) / kTile;
  const int ns = ap.ns, nsub = ap.nsub;
  if (ap.parts > b.nparts)
    return layer_fail(Lerr, XP_EINVAL, "attention partials exceed the buffers");   // not reached
  float* hout = h_f32 ? h_f32 : b.h32;
  hipError_t e;
#define XP_STEP(what, call)                                                                  \
  do {                                                                                       \
    call;                                                                                    \
    if ((e = hipGetLastError()) != hipSuccess)                                               \
      return layer_fail(Lerr, XP_EHIP, "%s launch failed: %s", what, hipGetErrorString(e));  \
  } while (0)
#define XP_LINEAR(what, ...)                                                                 \
  do {                                                                                       \
    if ((e = linear(__VA_ARGS__)) != hipSuccess)                                             \
      return layer_fail(Lerr, e == hipErrorInvalidValue ? XP_EINVAL : XP_EHIP,               \
                        "%s projection failed: %s", what, hipGetErrorString(e));             \
  } while (0)

  XP_STEP("rmsnorm", hipLaunchKernelGGL(k_rmsnorm<uint16_t>, dim3(M), dim3(256), 0, st,
                                        (const uint16_t*)x, (const float*)nullptr, 0, (size_t)0,
                                        H, L.g_attn, L.eps, b.x32, b.u));
  int sq = 1, so = 1, sd = 1;                    // k splits of q/k/v, output, down
  XP_LINEAR("q/k/v", b, L.Wq, L.Wk, L.Wv, nhd, kvd, ldq, H, b.u, M, nullptr, 0, b.qkv, nullptr,
            ldq, false, &sq, st);
  XP_STEP("qk-norm/rope",
          hipLaunchKernelGGL(k_qkrope, dim3(M), dim3(256), 0, st, sq > 1 ? b.part : b.qkv, sq,
                             (size_t)M * ldq, ldq, B, nh, nkv, ctx_len, C_max, L.g_q, L.g_k,
                             L.eps, L.theta, b.qn, b.kb, b.vb));
#define XP_ATTN(GG, PB)                                                                      \
  hipLaunchKernelGGL((k_attn<GG, PB>), dim3(ns, nkv, batch),                                  \
                     dim3(attn_waves(GG, PB) * kWave), 0, st,                                 \
                     b.qn, (const uint16_t*)k_cache, (const uint16_t*)v_cache, b.kb, b.vb,    \
                     ctx_len, C_max, B, nh, nkv, causal, ns, nsub, b.opart, b.mlpart)
  if (npb == 1) {
    if (grp == 1) XP_STEP("attention", XP_ATTN(1, 1));
    else if (grp == 2) XP_STEP("attention", XP_ATTN(2, 1));
    else if (grp == 4) XP_STEP("attention", XP_ATTN(4, 1));
    else XP_STEP("attention", XP_ATTN(8, 1));
  } else {
    if (grp == 1) XP_STEP("attention", XP_ATTN(1, 2));
    else if (grp == 2) XP_STEP("attention", XP_ATTN(2, 2));
    else if (grp == 4) XP_STEP("attention", XP_ATTN(4, 2));
    else XP_STEP("attention", XP_ATTN(8, 2));
  }
#undef XP_ATTN
  const int cw = M * nh;
  XP_STEP("attention combine",
          hipLaunchKernelGGL(k_attn_comb, dim3((cw + 3) / 4), dim3(256), 0, st, b.opart,
                             b.mlpart, M, B, npb, nh, nkv, grp, ns, b.attn));
  XP_LINEAR("output", b, L.Wo, nullptr, nullptr, H, 0, H, nhd, b.attn, M, b.x32, H, b.x1,
            nullptr, H, false, &so, st);
  // x1 = Wo attn + x: written by the projection, or here from its slabs
  if (so > 1)
    XP_STEP("rmsnorm", hipLaunchKernelGGL(k_rmsnorm<float>, dim3(M), dim3(256), 0, st,
                                          (const float*)b.x32, (const float*)b.part, so,
                                          (size_t)M * H, H, L.g_mlp, L.eps, b.x1, b.u));
  else
    XP_STEP("rmsnorm", hipLaunchKernelGGL(k_rmsnorm<float>, dim3(M), dim3(256), 0, st,
                                          (const float*)b.x1, (const float*)nullptr, 0, (size_t)0,
                                          H, L.g_mlp, L.eps, (float*)nullptr, b.u));
  XP_LINEAR("gate/up", b, L.Wg, L.Wu, nullptr, F, 0, F, H, b.u, M, nullptr, 0, nullptr, b.act, F,
            true, nullptr, st);
  XP_LINEAR("down", b, L.Wd, nullptr, nullptr, H, 0, H, F, b.act, M, b.x1, H, hout,
            (uint16_t*)h_bf16, H, false, &sd, st);
  if (sd > 1) {
    const size_t n = (size_t)M * H;
    XP_STEP("down split-K sum",
            hipLaunchKernelGGL(k_splitk_sum, dim3((unsigned)((n / 4 + 255) / 256)), dim3(256), 0,
                               st, (const float*)b.part, sd, n, (const float*)b.x1, hout,
                               (uint16_t*)h_bf16));
  }
#undef XP_STEP
#undef XP_LINEAR
  return XP_OK;
}

extern "C" xp_status xp_layer_forward(xp_layer* L, int32_t batch, int32_t B, int32_t causal,
                                      const void* x, const void* k_cache, const void* v_cache,
                                      int32_t C_max, const int32_t* ctx_len, float* h_f32,
                                      void* h_bf16, void* stream) {
  if (L == nullptr) return XP_EINVAL;
  const xp_status cs =
      check_call(L, batch, B, causal, x, k_cache, v_cache, C_max, ctx_len, h_f32, h_bf16);
  if (cs != XP_OK) return cs;
  if (batch > L->max_batch || B > L->max_B)
    return layer_fail(L, XP_EINVAL, "batch=%d (1..%d) or B=%d (1..%d) outside the created maxima",
                      batch, L->max_batch, B, L->max_B);
  if (C_max > (L->max_ctx > 0 ? L->max_ctx : 1))
    return layer_fail(L, XP_EINVAL, "C_max=%d out of range 1..%d", C_max,
                      L->max_ctx > 0 ? L->max_ctx : 1);
  return forward(*L, L->b, attn_plan_default(*L, batch, B, C_max), L, batch, B, causal, x,
                 k_cache, v_cache, C_max, ctx_len, h_f32, h_bf16, (hipStream_t)stream);
}

// ---------------------------------------------------------------------------
// The allocation-free forward.  Its buffers live in `scratch`, a static
// device array (every GPU the library runs on holds its own copy until the
// process ends).  Host code never uses the array's name as an address: the
// device address is looked up once per device with hipGetSymbolAddress and
// kept in g_scratch.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = (size_t)64 << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

static std::mutex g_scratch_mu;
static void* g_scratch[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up on the first
// call there.
static hipError_t scratch_ptr(char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = p;
  }
  *out = static_cast<char*>(g_scratch[dev]);
  return hipSuccess;
}

extern "C" xp_status xp_layer_forward_noalloc(const xp_layer_weights* w, int32_t batch, int32_t B,
                                              int32_t causal, const void* x, const void* k_cache,
                                              const void* v_cache, int32_t C_max,
                                              const int32_t* ctx_len, float* h_f32, void* h_bf16,
                                              void* stream) {
  g_layer_err.clear();
  xp_layer L;
  xp_status s = layer_weights(w, &L);
  if (s != XP_OK) return s;
  s = check_call(nullptr, batch, B, causal, x, k_cache, v_cache, C_max, ctx_len, h_f32, h_bf16);
  if (s != XP_OK) return s;
  const size_t M = (size_t)batch * B;
  if (!rows_fit_int32(L, (int64_t)M))
    return layer_fail(nullptr, XP_EINVAL, "batch*B*max(H, heads*128, ffn) reaches 2^31");
  // The buffers the call needs, its partials at the default chunking; if
  // those do not fit, chunks of more 64-key sub-chunks (fewer partials).
  const size_t gu = gu_rows_for(L, M);
  const size_t fixed = carve(L, M, 0, gu, 0, nullptr, nullptr);
  const size_t per_part = (size_t)kTile * kHd * 4 + (size_t)2 * kTile * 4;   // opart + mlpart
  if (fixed + 2 * 256 + per_part > kScratchBytes)
    return layer_fail(nullptr, XP_EINVAL,
                      "%zu positions need %zu bytes of buffers; the static scratch holds %zu",
                      M, fixed + per_part, kScratchBytes);
  const size_t max_parts = (kScratchBytes - fixed - 2 * 256) / per_part;
  AttnPlan ap = attn_plan_default(L, batch, B, C_max);
  if (ap.parts > max_parts) {
    const int chunks64 = attn_chunks(C_max, B, kSub);
    int lo = ap.nsub, hi = chunks64;             // ap at nsub = chunks64 has ns = 1
    if (attn_plan(L, batch, B, C_max, hi).parts > max_parts)
      return layer_fail(nullptr, XP_EINVAL,
                        "%d sequences x %d KV heads need more attention partials than the static "
                        "scratch holds beside %zu positions", batch, L.nkv, M);
    while (lo + 1 < hi) {                        // smallest nsub whose partials fit
      const int mid = lo + (hi - lo) / 2;
      if (attn_plan(L, batch, B, C_max, mid).parts > max_parts) lo = mid;
      else hi = mid;
    }
    ap = attn_plan(L, batch, B, C_max, hi);
  }
  char* base = nullptr;
  const hipError_t e = scratch_ptr(&base);
  if (e != hipSuccess)
    return layer_fail(nullptr, XP_EHIP, "static scratch address: %s", hipGetErrorString(e));
  LayerBufs b;
  const size_t used = carve(L, M, ap.parts, gu, 0, base, &b);
  if (used > kScratchBytes)                      // not reached: sized above
    return layer_fail(nullptr, XP_EINVAL, "buffers of %zu bytes exceed the static scratch", used);
  return forward(L, b, ap, nullptr, batch, B, causal, x, k_cache, v_cache, C_max, ctx_len, h_f32,
                 h_bf16, (hipStream_t)stream);
}
