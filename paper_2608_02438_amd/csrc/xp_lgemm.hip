// The context layer's projections for many positions: y = X W^T (+ residual)
// on the tiled bf16 GEMM pipeline of xp_gemm_pipe.h (the LM-head GEMM's) with
// a plain epilogue.
//
// Above one 64-position pass of the streaming projection kernel the weights
// would be re-read per 64 positions; here a tile is BN weight rows x BM
// positions (256 x 256 where every workgroup then gets two tiles or more, else
// 128 x 128), so every weight is read once per BM positions.  Up to three
// weights stacked by rows share the launch (the q, k and v projections of one
// input); BN divides each one's row count, so a tile never straddles two of
// them.  Persistent and XCD-aware as the LM-head GEMM (GemmSched).
#include "xp_internal.h"
#include "xp_gemm_pipe.h"

namespace xp {

// Rows of tile ti: BN consecutive rows of whichever of W0 | W1 | W2 holds
// stacked row sc.tile(ti) * BN.
struct LayerRows {
  const uint16_t *W0, *W1, *W2;
  int n0, n1, K;
  const GemmSched* sc;
  int BN;
  const uint16_t* w = nullptr;
  __device__ void prep(int ti) {
    const int r = sc->tile(ti) * BN;
    if (r < n0)
      w = W0 + (size_t)r * K;
    else if (r < n0 + n1)
      w = W1 + (size_t)(r - n0) * K;
    else
      w = W2 + (size_t)(r - n0 - n1) * K;
  }
  __device__ const uint16_t* row(int r) const { return w + (size_t)r * K; }
};

// y (+ residual) for the wave's rows and positions; four consecutive rows of
// one position are one 16-byte store.
template <int BN, int BM>
struct LayerEpi {
  using G = GemmShape<BN, BM>;
  static constexpr int NA = G::NA, NB = G::NB, RW = G::RW, PW = G::PW;
  const GemmSched* sc;
  const float* R;
  float* Y;
  uint16_t* Yb;
  int M, ldr, ldy, p0;
  __device__ void operator()(int ti, floatx16 (&acc)[NA][NB], const GemmLane& w) {
    const int rbase = sc->tile(ti) * BN + w.wv * RW;
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      const int p = p0 + w.wp * PW + c * 32 + w.lr;
      if (p < M) {
#pragma unroll
        for (int a = 0; a < NA; ++a)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int n = rbase + a * 32 + 8 * q + 4 * w.lk;
            floatx4 v{acc[a][c][4 * q], acc[a][c][4 * q + 1], acc[a][c][4 * q + 2],
                      acc[a][c][4 * q + 3]};
            if (R) v += *reinterpret_cast<const floatx4*>(R + (size_t)p * ldr + n);
            if (Y) *reinterpret_cast<floatx4*>(Y + (size_t)p * ldy + n) = v;
            if (Yb) {
              const uint32_t lo = f32_to_bf16_rne(v[0]) | ((uint32_t)f32_to_bf16_rne(v[1]) << 16);
              const uint32_t hi = f32_to_bf16_rne(v[2]) | ((uint32_t)f32_to_bf16_rne(v[3]) << 16);
              *reinterpret_cast<uint2*>(Yb + (size_t)p * ldy + n) = make_uint2(lo, hi);
            }
          }
      }
    }
  }
};

template <int BN, int BM>
__global__ __launch_bounds__(kGWaves * kWave) void k_layer_gemm(
    const uint16_t* __restrict__ W0, const uint16_t* __restrict__ W1,
    const uint16_t* __restrict__ W2, int n0, int n1, int N, int K,
    const uint16_t* __restrict__ X, int M, int nMb, int gpx, const float* __restrict__ R,
    int ldr, float* __restrict__ Y, uint16_t* __restrict__ Yb, int ldy) {
  __shared__ u32x4 lds[GemmShape<BN, BM>::SLOTS];                  // [stage][W | X]
  const GemmSched sc(nMb, gpx);
  const int ntl = sc.count(N / BN);
  if (ntl == 0) return;                                            // whole workgroup
  const int p0 = sc.mb * BM;
  LayerRows rows{W0, W1, W2, n0, n1, K, &sc, BN};
  LayerEpi<BN, BM> epi{&sc, R, Y, Yb, M, ldr, ldy, p0};
  gemm_tiles<BN, BM>(rows, epi, X, M, K, ntl, p0, lds);
}

}  // namespace xp

using namespace xp;

namespace xp {

// Rows of W0 | W1 | W2 stacked (n0, n1 rows of the first two; BN must divide
// n0, n1 and N); K a multiple of 32; M >= 1.
// Position and row tile size: 256 x 256 only when that still gives every
// workgroup of the persistent grid two tiles or more; else 128 x 128 (four
// times as many tiles for the same work).
static int layer_bm(int N, int M) {
  const long t256 = (long)(N / 256) * ((M + 255) / 256);
  return M <= 128 || t256 < 2 * 8 * kGPerXcd ? 128 : 256;
}

bool layer_gemm_ok(int n0, int n1, int N, int K, int M) {
  const int bn = layer_bm(N, M);
  return K % kGK == 0 && N % bn == 0 && n0 % bn == 0 && n1 % bn == 0 && M >= 1;
}

hipError_t launch_layer_gemm(const uint16_t* W0, const uint16_t* W1, const uint16_t* W2, int n0,
                             int n1, int N, int K, const uint16_t* X, int M, const float* R,
                             int ldr, float* Y, uint16_t* Yb, int ldy, hipStream_t st) {
  const int bm = layer_bm(N, M);
  const int nMb = (M + bm - 1) / bm;
  const int per = gemm_per_xcd(nMb);              // workgroups per XCD: whole position groups
  const int gpx = per / nMb;
  if (bm == 128)
    hipLaunchKernelGGL((k_layer_gemm<128, 128>), dim3(8 * per), dim3(kGWaves * kWave), 0, st, W0,
                       W1, W2, n0, n1, N, K, X, M, nMb, gpx, R, ldr, Y, Yb, ldy);
  else
    hipLaunchKernelGGL((k_layer_gemm<256, 256>), dim3(8 * per), dim3(kGWaves * kWave), 0, st, W0,
                       W1, W2, n0, n1, N, K, X, M, nMb, gpx, R, ldr, Y, Yb, ldy);
  return hipGetLastError();
}

}  // namespace xp
