// The context layer's projections for many positions: y = X W^T (+ residual)
// as a tiled GEMM on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16), the
// LM-head GEMM's machinery with a plain epilogue.
//
// Above one 64-position pass of the streaming projection kernel the weights
// would be re-read per 64 positions; here a tile is BN weight rows x BM
// positions (256 x 256 where every workgroup then gets two tiles or more, else
// 128 x 128), so every weight
// is read once per BM positions.  Up to three weights stacked by rows share
// the launch (the q, k and v projections of one input); BN divides each
// one's row count, so a tile never straddles two of them.
//
// Persistent and XCD-aware as the LM-head GEMM: one workgroup per CU walks
// its row tiles for one position tile, the position tiles of one row tile run
// on the same XCD at about the same time (their reads of the rows share that
// XCD's L2), and the global-to-LDS stage ring runs on across tile boundaries.
// Each of the 8 waves owns BN/2 rows x BM/4 positions of the tile.
//
// Layout of the 32x32x16 operation: lane l holds row l % 32 of A and column
// l % 32 of B, k = 8 (l / 32) .. + 8; result register i of lane l is
// D[8 (i / 4) + 4 (l / 32) + i % 4][l % 32]; A = weight rows, B = positions.
#include "xp_internal.h"

namespace xp {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kLK = 32;             // k per LDS stage
constexpr int kLWaves = 8;          // 2 (rows) x 4 (positions) waves
constexpr int kLPerXcd = 32;        // workgroups per XCD (one per CU)

__device__ __forceinline__ floatx16 lmma32(u32x4 a, u32x4 b, floatx16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// A stage row holds 32 k (four 16-byte chunks); chunk c of row r sits in slot
// 4 r + (c ^ swz(r)), so the operand reads (32 rows, one chunk) are
// conflict-free.
__device__ __forceinline__ int lslot(int r, int c) { return 4 * r + (c ^ (((r >> 1) ^ (r >> 3)) & 3)); }

template <int BN, int BM>
__global__ __launch_bounds__(kLWaves * kWave) void k_layer_gemm(
    const uint16_t* __restrict__ W0, const uint16_t* __restrict__ W1,
    const uint16_t* __restrict__ W2, int n0, int n1, int N, int K,
    const uint16_t* __restrict__ X, int M, int nMb, int gpx, const float* __restrict__ R,
    int ldr, float* __restrict__ Y, uint16_t* __restrict__ Yb, int ldy) {
  constexpr int RW = BN / 2, PW = BM / 4;                          // rows, positions per wave
  constexpr int NA = RW / 32, NB = PW / 32;                        // 32 x 32 blocks per wave
  constexpr int WS = BN * kLK * 2 / 16, HS = BM * kLK * 2 / 16;    // slots per operand stage
  constexpr int WI = WS / 64 / kLWaves, HI = HS / 64 / kLWaves;    // 1 KB loads per wave
  constexpr int NS0 = 163840 / ((WS + HS) * 16);
  constexpr int NS = NS0 < 8 ? NS0 : 8;                            // ring stages
  static_assert(WI >= 1 && HI >= 1 && NA >= 1 && NB >= 1, "tile shape");
  static_assert(NS * (WS + HS) * 16 <= 163840, "LDS");
  __shared__ u32x4 lds[NS * (WS + HS)];                            // [stage][W | X]

  const int ntn = N / BN;
  const int xcd = blockIdx.x & 7, k8 = blockIdx.x >> 3;
  const int k8q = k8 / nMb, mb = k8 - k8q * nMb;
  auto rtile = [&](int i) { return 8 * (i * gpx + k8q) + xcd; };  // i-th row tile
  const int first = 8 * k8q + xcd;
  const int ntl = first < ntn ? (ntn - first + 8 * gpx - 1) / (8 * gpx) : 0;
  if (ntl == 0) return;                                            // whole workgroup
  const int nk = K / kLK;
  const int nstages = ntl * nk;
  const int p0 = mb * BM;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave & 1, wp = wave >> 1;                         // row half, position block

  // stage loads: wave w fills W slots [64 WI w, 64 WI (w + 1)) and X slots
  // [64 HI w, 64 HI (w + 1)) with 1 KB instructions; lane l of an instruction
  // writes the next slot, i.e. LDS row slot / 4, stored chunk l % 4, which
  // holds logical chunk (l % 4) ^ swz(row)
  int wrow[WI], wcol[WI], hrow[HI];
#pragma unroll
  for (int j = 0; j < WI; ++j) {
    const int row = (64 * (WI * wave + j) + lane) >> 2;
    wrow[j] = row;
    wcol[j] = 8 * ((lane & 3) ^ (((row >> 1) ^ (row >> 3)) & 3));
  }
#pragma unroll
  for (int j = 0; j < HI; ++j) {
    const int row = (64 * (HI * wave + j) + lane) >> 2;
    int hr = p0 + row;
    hr = hr < M ? hr : M - 1;
    hrow[j] = hr * K + 8 * ((lane & 3) ^ (((row >> 1) ^ (row >> 3)) & 3));
  }
  // weight and first row of the tile being issued (cached per tile)
  int iss_tile = -1;
  const uint16_t* iss_w = W0;
  int iss_r = 0;
  auto prep = [&](int gs) {
    gs = gs < nstages ? gs : nstages - 1;
    const int ti = gs / nk;
    if (ti != iss_tile) {                                          // wave-uniform
      const int r = rtile(ti) * BN;
      iss_tile = ti;
      if (r < n0) {
        iss_w = W0;
        iss_r = r;
      } else if (r < n0 + n1) {
        iss_w = W1;
        iss_r = r - n0;
      } else {
        iss_w = W2;
        iss_r = r - n0 - n1;
      }
    }
  };
  auto issue = [&](int gs) {                                       // global stage gs (clamped)
    gs = gs < nstages ? gs : nstages - 1;
    const int ti = gs / nk, kc = gs - ti * nk;
    const int st = gs % NS;
#pragma unroll
    for (int j = 0; j < WI; ++j)
      lds_dma16(iss_w + (size_t)(iss_r + wrow[j]) * K + kc * kLK + wcol[j],
                &lds[st * (WS + HS) + 64 * (WI * wave + j)]);
#pragma unroll
    for (int j = 0; j < HI; ++j)
      lds_dma16(X + (size_t)(unsigned)hrow[j] + kc * kLK,
                &lds[st * (WS + HS) + WS + 64 * (HI * wave + j)]);
  };

  floatx16 acc[NA][NB];
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][c][i] = 0.f;

  const int lr = lane & 31, lk = lane >> 5;
  auto rd = [&](int gs, int ks, u32x4 (&av)[NA], u32x4 (&bv)[NB]) {
    const int base = (gs % NS) * (WS + HS);
    const int c = 2 * ks + lk;
#pragma unroll
    for (int a = 0; a < NA; ++a) av[a] = lds[base + lslot(wv * RW + a * 32 + lr, c)];
#pragma unroll
    for (int cc = 0; cc < NB; ++cc) bv[cc] = lds[base + WS + lslot(wp * PW + cc * 32 + lr, c)];
  };
  auto mm = [&](const u32x4 (&av)[NA], const u32x4 (&bv)[NB]) {
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int cc = 0; cc < NB; ++cc) acc[a][cc] = lmma32(av[a], bv[cc], acc[a][cc]);
  };
  // epilogue of tile ti: y (+ residual) for this wave's rows and positions;
  // four consecutive rows of one position are one 16-byte store
  auto epilogue = [&](int ti) {
    const int rbase = rtile(ti) * BN + wv * RW;
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      const int p = p0 + wp * PW + c * 32 + lr;
      if (p < M) {
#pragma unroll
        for (int a = 0; a < NA; ++a)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int n = rbase + a * 32 + 8 * q + 4 * lk;
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
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int c = 0; c < NB; ++c)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[a][c][i] = 0.f;
  };

#pragma unroll
  for (int s = 0; s < NS; ++s) {
    prep(s);
    issue(s);
  }
  constexpr int kP0 = (WI + HI) * (NS - 1), kP = (WI + HI) * (NS - 2);
  static_assert(kP0 < 64, "vmcnt field");
  // stage 0 landed (this wave's loads), then every wave's
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0070 | (kP0 & 15) | ((kP0 >> 4) << 14));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  u32x4 fa[2][NA], fb[2][NB];               // fragment sets of the two k steps of a stage
  rd(0, 0, fa[0], fb[0]);
  __builtin_amdgcn_s_waitcnt(0xc07f);
  int ti = 0, kc = 0;
  for (int gs = 0; gs < nstages; ++gs) {
    // as in the LM-head GEMM: k step 1 of stage gs is read while k step 0
    // multiplies; the barrier between the two k steps (stage gs + 1 landed for
    // this wave, its reads of stage gs done) publishes stage gs + 1 and frees
    // the slot of stage gs for stage gs + NS; the fragment reads go one by one
    // between the matrix operations, the loads of stage gs + NS behind them
    rd(gs, 1, fa[1], fb[1]);
    mm(fa[0], fb[0]);
#pragma unroll
    for (int q = 0; q < NA + NB; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 16, 0);
    __builtin_amdgcn_sched_barrier(0);
    prep(gs + NS);
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0x0070 | (kP & 15) | ((kP >> 4) << 14));
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    rd(gs + 1, 0, fa[0], fb[0]);
    mm(fa[1], fb[1]);
    issue(gs + NS);
#pragma unroll
    for (int q = 0; q < NA + NB; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 16, 0);
    __builtin_amdgcn_sched_group_barrier(0x020, 16, 0);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_sched_barrier(0);
    if (++kc == nk) {                                              // wave-uniform
      epilogue(ti);
      kc = 0;
      ++ti;
    }
  }
  __builtin_amdgcn_s_waitcnt(0x0070);        // the clamped loads past the end
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
  return M <= 128 || t256 < 2 * 8 * kLPerXcd ? 128 : 256;
}

bool layer_gemm_ok(int n0, int n1, int N, int K, int M) {
  const int bn = layer_bm(N, M);
  return K % kLK == 0 && N % bn == 0 && n0 % bn == 0 && n1 % bn == 0 && M >= 1;
}

hipError_t launch_layer_gemm(const uint16_t* W0, const uint16_t* W1, const uint16_t* W2, int n0,
                             int n1, int N, int K, const uint16_t* X, int M, const float* R,
                             int ldr, float* Y, uint16_t* Yb, int ldy, hipStream_t st) {
  const int bm = layer_bm(N, M);
  const int nMb = (M + bm - 1) / bm;
  int per = kLPerXcd / nMb * nMb;                // workgroups per XCD: whole position tiles
  per = per > 0 ? per : nMb;
  const int gpx = per / nMb;
  if (bm == 128)
    hipLaunchKernelGGL((k_layer_gemm<128, 128>), dim3(8 * per), dim3(kLWaves * kWave), 0, st, W0,
                       W1, W2, n0, n1, N, K, X, M, nMb, gpx, R, ldr, Y, Yb, ldy);
  else
    hipLaunchKernelGGL((k_layer_gemm<256, 256>), dim3(8 * per), dim3(kLWaves * kWave), 0, st, W0,
                       W1, W2, n0, n1, N, K, X, M, nMb, gpx, R, ldr, Y, Yb, ldy);
  return hipGetLastError();
}

}  // namespace xp
