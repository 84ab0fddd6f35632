// The context layer's projections for many positions on the tiled bf16 GEMM
// pipeline of xp_gemm_pipe.h (the LM-head GEMM's), in three forms:
//   plain    y = X W^T (+ residual), fp32 and/or bf16;
//   split-K  the k range cut into S equal parts, each tile writing its fp32
//            partial product to slab s of [S][M][N]; the kernel that reads
//            y next adds the slabs in slab order (so the result does not
//            depend on timing);
//   GLU      bf16(silu(X Wg^T) * (X Wu^T)): a tile's rows are gate and up
//            rows of the same features, so the product is formed in the
//            epilogue.
//
// Above one 64-position pass of the streaming projection kernel the weights
// would be re-read per 64 positions; here a tile is BN weight rows x BM
// positions (128 x 128 or 256 x 256, layer_plan), so every weight is read
// once per BM positions.  Where the tiles are fewer than the CUs (the output
// and down projections of a few hundred positions), split-K multiplies the
// work items up to one per CU.  Up to three weights stacked by rows share the
// launch (the q, k and v projections of one input); BN divides each one's
// row count, so a tile never straddles two of them.  Persistent and XCD-aware as the LM-head GEMM
// (GemmSched), over the virtual row tiles rt S + s.
#include "xp_internal.h"
#include "xp_gemm_pipe.h"

namespace xp {


// Rows of tile ti (virtual row tile v = sc.tile(ti) = rt S + s, k from s kt).
// Plain: BN consecutive rows of whichever of W0 | W1 | W2 holds stacked row
// rt BN.  GLU: the features f0 = rt BN / 2 .. + BN / 2 of the gate (W0) and up
// (W1) weights; in each wave's half of the tile the first half of the 32-row
// blocks are gate rows and the second half the up rows of the same features.
template <int BN, bool GLU>
struct LayerRows {
  const uint16_t *W0, *W1, *W2;
  int n0, n1, K, S, kt;
  const GemmSched* sc;
  const uint16_t *w = nullptr, *wu = nullptr;
  int xk = 0;
  __device__ void prep(int ti) {
    const int v = sc->tile(ti), rt = v / S, s = v - rt * S;
    xk = s * kt;
    if constexpr (GLU) {
      const size_t f0 = (size_t)rt * (BN / 2);
      w = W0 + f0 * K + xk;
      wu = W1 + f0 * K + xk;
    } else {
      const int r = rt * BN;
      if (r < n0)
        w = W0 + (size_t)r * K;
      else if (r < n0 + n1)
        w = W1 + (size_t)(r - n0) * K;
      else
        w = W2 + (size_t)(r - n0 - n1) * K;
      w += xk;
    }
  }
  __device__ const uint16_t* row(int r) const {
    if constexpr (GLU) {
      constexpr int RW = BN / 2, NH = RW / 64;    // gate blocks per wave half
      const int h = r / RW, rr = r - h * RW, a = rr >> 5;
      const int f = h * (RW / 2) + (a % NH) * 32 + (rr & 31);
      return (a < NH ? w : wu) + (size_t)f * K;
    } else {
      return w + (size_t)r * K;
    }
  }
};

// Plain / split-K: y (+ residual) for the wave's rows and positions, four
// consecutive rows of one position per 16-byte store; a split tile writes
// its slab (no residual, no bf16).  GLU: the wave's gate blocks a and up
// blocks a + NA/2 hold the same features, bf16(silu(gate) * up) four
// features per 8-byte store.
template <int BN, int BM, bool GLU>
struct LayerEpi {
  using G = GemmShape<BN, BM>;
  static constexpr int NA = G::NA, NB = G::NB, RW = G::RW, PW = G::PW;
  const GemmSched* sc;
  const float* R;
  float* Y;
  uint16_t* Yb;
  int M, ldr, ldy, p0, S;
  size_t slab;
  __device__ void operator()(int ti, floatx16 (&acc)[NA][NB], const GemmLane& w) {
    const int v = sc->tile(ti), rt = v / S, s = v - rt * S;
    if constexpr (GLU) {
      constexpr int NH = NA / 2;
      const int fbase = rt * (BN / 2) + w.wv * (RW / 2);
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        const int p = p0 + w.wp * PW + c * 32 + w.lr;
        if (p < M) {
#pragma unroll
          for (int a = 0; a < NH; ++a)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int f = fbase + a * 32 + 8 * q + 4 * w.lk;
              uint16_t o[4];
#pragma unroll
              for (int e = 0; e < 4; ++e)
                o[e] = f32_to_bf16_rne(silu_mul(acc[a][c][4 * q + e], acc[a + NH][c][4 * q + e]));
              *reinterpret_cast<uint2*>(Yb + (size_t)p * ldy + f) =
                  make_uint2(o[0] | ((uint32_t)o[1] << 16), o[2] | ((uint32_t)o[3] << 16));
            }
        }
      }
    } else {
      const int rbase = rt * BN + w.wv * RW;
      float* Ys = Y ? Y + (size_t)s * slab : nullptr;
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        const int p = p0 + w.wp * PW + c * 32 + w.lr;
        if (p < M) {
#pragma unroll
          for (int a = 0; a < NA; ++a)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int n = rbase + a * 32 + 8 * q + 4 * w.lk;
              floatx4 v4{acc[a][c][4 * q], acc[a][c][4 * q + 1], acc[a][c][4 * q + 2],
                         acc[a][c][4 * q + 3]};
              if (R) v4 += *reinterpret_cast<const floatx4*>(R + (size_t)p * ldr + n);
              if (Ys) *reinterpret_cast<floatx4*>(Ys + (size_t)p * ldy + n) = v4;
              if (Yb) {
                const uint32_t lo =
                    f32_to_bf16_rne(v4[0]) | ((uint32_t)f32_to_bf16_rne(v4[1]) << 16);
                const uint32_t hi =
                    f32_to_bf16_rne(v4[2]) | ((uint32_t)f32_to_bf16_rne(v4[3]) << 16);
                *reinterpret_cast<uint2*>(Yb + (size_t)p * ldy + n) = make_uint2(lo, hi);
              }
            }
        }
      }
    }
  }
};

// N stacked rows (GLU: 2F, gate and up), S k splits of K / S each.
template <int BN, int BM, bool GLU>
__global__ __launch_bounds__(kGWaves * kWave) void k_layer_gemm(
    const uint16_t* __restrict__ W0, const uint16_t* __restrict__ W1,
    const uint16_t* __restrict__ W2, int n0, int n1, int N, int K, int S,
    const uint16_t* __restrict__ X, int M, int nMb, int gpx, const float* __restrict__ R,
    int ldr, float* __restrict__ Y, size_t slab, uint16_t* __restrict__ Yb, int ldy) {
  __shared__ u32x4 lds[GemmShape<BN, BM>::SLOTS];                  // [stage][W | X]
  const GemmSched sc(nMb, gpx);
  const int ntl = sc.count(N / BN * S);
  if (ntl == 0) return;                                            // whole workgroup
  const int p0 = sc.mb * BM, kt = K / S;
  LayerRows<BN, GLU> rows{W0, W1, W2, n0, n1, K, S, kt, &sc};
  LayerEpi<BN, BM, GLU> epi{&sc, R, Y, Yb, M, ldr, ldy, p0, S, slab};
  gemm_tiles<BN, BM>(rows, epi, X, K, M, kt, ntl, p0, lds);
}

// Tile size and k splits of one projection: among 128 x 128 and 256 x 256
// tiles (BN dividing every stacked weight's rows) and S = 1 .. kLayerSplitMax
// splits (S dividing the k steps, at least 16 k steps per split, S M N fp32
// slab values within part_floats; GLU: S = 1), the one with the least
// estimated time: rounds of one work item per workgroup of the persistent
// grid, an item costing 17 us plus its flops at 3.6 TFLOP/s per CU on 128 x
// 128 tiles or 4.3 on 256 x 256 (fitted to the measured launches of the
// Qwen3-8B projections at 128 to 2048 positions), plus one read of the slabs
// at 5 TB/s by the kernel that adds them.  bn = 0: no plan (K not a multiple
// of 32 or no tile divides the rows).
LayerPlan layer_plan(int n0, int n1, int N, int K, int M, bool glu, size_t part_floats) {
  LayerPlan best{0, 1};
  if (K % kGK != 0 || M < 1) return best;
  const int nk = K / kGK, slots = 8 * kGPerXcd;
  double tbest = 0.0;
  for (int bn = 128; bn <= 256; bn *= 2) {
    if (N % bn != 0 || n0 % bn != 0 || n1 % bn != 0) continue;
    const double rate = bn == 128 ? 3.6e12 : 4.3e12;
    const long tiles = (long)(N / bn) * ((M + bn - 1) / bn);
    for (int S = 1; S <= (glu ? 1 : kLayerSplitMax); ++S) {
      if (nk % S != 0 || (S > 1 && nk / S < 16)) continue;
      if (S > 1 && (double)S * M * N > (double)part_floats) continue;
      const long items = tiles * S;
      const double rounds = (double)((items + slots - 1) / slots);
      double t = rounds * (17e-6 + 2.0 * bn * bn * (double)(K / S) / rate);
      if (S > 1) t += 4.0 * S * (double)M * N / 5e12;
      if (best.bn == 0 || t < tbest) {
        best = LayerPlan{bn, S};
        tbest = t;
      }
    }
  }
  return best;
}

template <bool GLU>
static void launch(LayerPlan pl, const uint16_t* W0, const uint16_t* W1, const uint16_t* W2,
                   int n0, int n1, int N, int K, const uint16_t* X, int M, const float* R, int ldr,
                   float* Y, uint16_t* Yb, int ldy, hipStream_t st) {
  const int bm = pl.bn;
  const int nMb = (M + bm - 1) / bm;
  const int per = gemm_per_xcd(nMb);              // workgroups per XCD: whole position groups
  const int gpx = per / nMb;
  const size_t slab = (size_t)M * ldy;
  if (bm == 128)
    hipLaunchKernelGGL((k_layer_gemm<128, 128, GLU>), dim3(8 * per), dim3(kGWaves * kWave), 0, st,
                       W0, W1, W2, n0, n1, N, K, pl.S, X, M, nMb, gpx, R, ldr, Y, slab, Yb, ldy);
  else
    hipLaunchKernelGGL((k_layer_gemm<256, 256, GLU>), dim3(8 * per), dim3(kGWaves * kWave), 0, st,
                       W0, W1, W2, n0, n1, N, K, pl.S, X, M, nMb, gpx, R, ldr, Y, slab, Yb, ldy);
}

hipError_t launch_layer_gemm(LayerPlan pl, const uint16_t* W0, const uint16_t* W1,
                             const uint16_t* W2, int n0, int n1, int N, int K, const uint16_t* X,
                             int M, const float* R, int ldr, float* Y, uint16_t* Yb, int ldy,
                             hipStream_t st) {
  if ((pl.bn != 128 && pl.bn != 256) || pl.S < 1 || K % (pl.S * kGK) != 0 || N % pl.bn != 0 ||
      n0 % pl.bn != 0 || n1 % pl.bn != 0 || (pl.S > 1 && (R || Yb || !Y || ldy != N)))
    return hipErrorInvalidValue;
  launch<false>(pl, W0, W1, W2, n0, n1, N, K, X, M, R, ldr, Y, Yb, ldy, st);
  return hipGetLastError();
}

hipError_t launch_layer_glu(LayerPlan pl, const uint16_t* Wg, const uint16_t* Wu, int F, int K,
                            const uint16_t* X, int M, uint16_t* act, int ldy, hipStream_t st) {
  if ((pl.bn != 128 && pl.bn != 256) || pl.S != 1 || K % kGK != 0 || (2 * F) % pl.bn != 0 ||
      F % pl.bn != 0)
    return hipErrorInvalidValue;
  launch<true>(pl, Wg, Wu, Wu, F, F, 2 * F, K, X, M, nullptr, 0, nullptr, act, ldy, st);
  return hipGetLastError();
}

}  // namespace xp
