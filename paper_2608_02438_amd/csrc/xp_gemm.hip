// A1 for many positions: s = W_lm h as a tiled GEMM on the bf16 matrix cores
// (v_mfma_f32_32x32x16_bf16), fused with the first stage of token selection.
//
// Once the position count M exceeds one 16-position block, streaming W_lm per
// block (the A1 stream kernels) would read the 1.2 GB head M/16 times; here a
// tile is BN vocabulary rows x BM positions, so W_lm is read once per BM
// positions.  Two shapes: 256 x 256 for more than 128 positions (the matrix
// cores, not HBM, bound the time at M = 512), and 128 x 128 up to 128
// positions, where the launch is HBM-bound and the smaller tile gives 4x more
// tiles to balance over the CUs and a deeper stage ring.
//
// Selection units: the vocabulary tiles are split into U = 2 ceil(ntiles /
// (BN/16)) units (unit_tile_lo partition, at most BN/32 tiles each); a
// workgroup tile covers the units 2u and 2u+1, LDS rows [0, BN/2) holding the
// first and [BN/2, BN) the second.  Each wave owns BN/2 rows (one unit) x BM/4
// positions, so it forms the selection partials of its unit directly from its
// accumulators: no reduction across waves.
//
// The kernel is persistent: one workgroup per CU walks its list of tiles, and
// the global-to-LDS stage ring runs on across tile boundaries, so the next
// tile's first stages load while the previous tile's epilogue (the s stores
// and the selection partials) runs.  The tile order is XCD-aware: the
// position tiles of one unit run on the same XCD at the same time, so their
// reads of the unit's W_lm rows share that XCD's L2.
//
// Layout of the 32x32x16 operation (checked on gfx950): lane l holds row
// l % 32 of A and column l % 32 of B, k = 8 (l / 32) .. + 8; result register
// i of lane l is D[8 (i / 4) + 4 (l / 32) + i % 4][l % 32].  Here A = W_lm rows
// and B = h rows (positions), so D[row][position].
#include "xp_internal.h"
#include "xp_gemm_pipe.h"

namespace xp {

// Rows of tile ti: selection units 2u and 2u + 1 of unit pair u = sc.tile(ti);
// LDS rows [0, BN/2) hold the first, [BN/2, BN) the second (rows past a unit
// are loaded, never used; rows past V repeat row V - 1).
template <int BN>
struct LmRows {
  const uint16_t* W;
  int V, H, ntiles, U2;
  const GemmSched* sc;
  int r0 = 0, r1 = 0;
  static constexpr int xk = 0;                     // every tile spans all of k
  __device__ void prep(int ti) {
    const int u = sc->tile(ti);
    r0 = unit_tile_lo(2 * u, ntiles, U2) * kTile;
    r1 = unit_tile_lo(2 * u + 1, ntiles, U2) * kTile;
  }
  __device__ const uint16_t* row(int r) const {
    int rr = (r < BN / 2 ? r0 : r1) + (r % (BN / 2));
    rr = rr < V ? rr : V - 1;
    return W + (size_t)rr * H;
  }
};

// Epilogue of tile ti: s from the accumulators, and the selection partials of
// the wave's unit (its BN/2 rows) for its BM/4 positions.
template <int BN, int BM>
struct LmEpi {
  using G = GemmShape<BN, BM>;
  static constexpr int NA = G::NA, NB = G::NB, PW = G::PW;
  const GemmSched* sc;
  float* S;
  uint64_t* keys;
  Stat* stats;
  int M, Ms, V, ntiles, U2, p0;
  bool psamp[NB];
  float pit[NB];                                   // sampled rows: softmax(s / T)
  // per 32-position block, wave-uniform: does any lane take the greedy
  // maximum, any the softmax partials?  (A block inside one sequence, as
  // with B a multiple of 32, does only one of the two.)
  bool do_max[NB], do_sum[NB];

  // The position tile is fixed per workgroup, so the sampling flags and 1/T
  // of this wave's positions are loaded once, before the stage loads, and
  // waited for here: no epilogue then waits for a load.
  __device__ LmEpi(const GemmSched* sc_, float* S_, int Ms_, uint64_t* keys_, Stat* stats_,
                   int M_, int V_, int ntiles_, int U2_, int p0_, const uint8_t* temp, int B,
                   const float* invT, const uint16_t* W)
      : sc(sc_), S(S_), keys(keys_), stats(stats_), M(M_), Ms(Ms_), V(V_), ntiles(ntiles_),
        U2(U2_), p0(p0_) {
    const int lane = threadIdx.x & 63, wp = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) >> 1;
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      const int p = p0 + wp * PW + c * 32 + (lane & 31);
      const int pc = p < M ? p : M - 1;
      psamp[c] = (p < M) & (load_flag(temp, pc / B, W) != 0);
      pit[c] = invT[pc / B];
      do_max[c] = __ballot((p < M) && !psamp[c]) != 0;
      do_sum[c] = __ballot(psamp[c]) != 0;
    }
#pragma unroll
    for (int c = 0; c < NB; ++c) asm volatile("" ::"v"(pit[c]));
  }

  __device__ void operator()(int ti, floatx16 (&acc)[NA][NB], const GemmLane& w) {
    const int hu = 2 * sc->tile(ti) + w.wv;
    const int rbase = unit_tile_lo(hu, ntiles, U2) * kTile;
    const int nr = unit_tile_lo(hu + 1, ntiles, U2) * kTile - rbase;   // <= BN/2, multiple of 16
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      const int p = p0 + w.wp * PW + c * 32 + w.lr;
      const bool pact = p < M;
      const bool psample = psamp[c];
      // running maximum and its row: rows increase along (a, q, e) in every
      // lane, so a strict comparison keeps the lowest index of a tie
      float bvv = -INFINITY;
      uint32_t bix = 0xFFFFFFFFu;
      Stat st = stat_empty();
#pragma unroll
      for (int a = 0; a < NA; ++a) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int rl = a * 32 + 8 * q + 4 * w.lk;                // local row of acc[a][c][4q]
          const bool rv = pact && rl < nr;
          if (rv)
            *reinterpret_cast<float4*>(S + s_index(p, rbase + rl, Ms)) =
                make_float4(acc[a][c][4 * q], acc[a][c][4 * q + 1], acc[a][c][4 * q + 2],
                            acc[a][c][4 * q + 3]);
          if (do_max[c]) {                                         // wave-uniform
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float x = acc[a][c][4 * q + e];
              const bool take = rv && !psample && rbase + rl + e < V && x > bvv;
              bvv = take ? x : bvv;
              bix = take ? (uint32_t)(rbase + rl + e) : bix;
            }
          }
          if (do_sum[c]) {                                         // wave-uniform
            float x[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
              x[e] = (rv && psample && rbase + rl + e < V) ? acc[a][c][4 * q + e] * pit[c] : -INFINITY;
            st = stat_add4(st, x[0], x[1], x[2], x[3]);
          }
        }
      }
      uint64_t best = bix == 0xFFFFFFFFu ? kKeyMin : argmax_key(bvv, bix);
      best = umax64(best, shfl_xor_u64(best, 32));
      const Stat o{__shfl_xor(st.m, 32, kWave), __shfl_xor(st.s, 32, kWave)};
      st = stat_merge(st, o);
      if (w.lk == 0 && pact) {
        keys[(size_t)hu * M + p] = best;
        if (psample) stats[(size_t)p * U2 + hu] = st;
      }
    }
  }
};

// Selection units: the vocabulary tiles are split into U2 = 2 ceil(ntiles /
// (BN/16)) units (unit_tile_lo partition, at most BN/32 tiles each); a
// workgroup tile covers the units 2u and 2u+1, one per wave row half, so each
// wave forms the selection partials of its unit straight from its
// accumulators: no reduction across waves.  Persistent: one workgroup per CU
// walks its list of tiles (GemmSched, XCD-aware).
template <int BN, int BM>
__global__ __launch_bounds__(kGWaves * kWave) void k_lmhead_gemm(
    const uint16_t* __restrict__ W, const uint16_t* __restrict__ X, int V, int H, int M,
    int ntiles, int U2, int nMb, int gpx, float* __restrict__ S, int Ms,
    uint64_t* __restrict__ keys, Stat* __restrict__ stats, const uint8_t* __restrict__ temp,
    int B, const float* __restrict__ invT) {
  __shared__ u32x4 lds[GemmShape<BN, BM>::SLOTS];                  // [stage][W | h]
  const GemmSched sc(nMb, gpx);
  const int ntl = sc.count(U2 / 2);
  if (ntl == 0) return;                                            // whole workgroup
  const int p0 = sc.mb * BM;
  LmRows<BN> rows{W, V, H, ntiles, U2, &sc};
  LmEpi<BN, BM> epi(&sc, S, Ms, keys, stats, M, V, ntiles, U2, p0, temp, B, invT, W);
  // HBM-bound 128 x 128 tiles: each group of workgroups sharing a row tile
  // starts its k walk at its own eighth of H, so that at any time the
  // launch's W_lm reads spread over the columns of the rows (the rows are
  // 8 KB apart; presumably more DRAM channels at once): 7% less time at 128
  // positions;
  // on 256 x 256 tiles (matrix-bound, and the h tile shared through L2 by
  // the row tiles of one position tile) it cost 1-3%
  const int kshift = BN == 128 ? ((sc.k8q & 7) * (H / kGK)) >> 3 : 0;
  gemm_tiles<BN, BM>(rows, epi, X, H, M, H, ntl, p0, lds, kshift);
}

// ---------------------------------------------------------------------------
// Tile shape for M positions: 128 x 128 up to 128 positions, 256 x 256 above.
static int gemm_bn(int M) { return M <= 128 ? 128 : 256; }

// Selection units of the GEMM path for M positions: 2 per workgroup tile of
// BN rows (at most BN/32 tiles each).  The launch and every reader of the
// per-unit partials use this one function; gemm_units_max bounds it.
int gemm_units(const xp_handle* h, int M) {
  const int bn = gemm_bn(M);
  return 2 * ((h->ntiles + bn / 16 - 1) / (bn / 16));
}
int gemm_units_max(const xp_handle* h) { return gemm_units(h, 1); }

bool lmhead_gemm_ok(const xp_handle* h, int M) {
  return h->dtype == XP_BF16 && M > kTile && h->H % kGK == 0;
}

hipError_t launch_lmhead_gemm(xp_handle* h, int M, const void* hidden, const uint8_t* temp,
                              hipStream_t st) {
  const int U2 = gemm_units(h, M);
  const int bm = gemm_bn(M);
  const int nMb = (M + bm - 1) / bm;
  const int per = gemm_per_xcd(nMb);              // workgroups per XCD: whole position groups
  const int gpx = per / nMb;
  if (bm == 128)
    hipLaunchKernelGGL((k_lmhead_gemm<128, 128>), dim3(8 * per), dim3(kGWaves * kWave), 0, st,
                       (const uint16_t*)h->W_lm, (const uint16_t*)hidden, h->V, h->H, M,
                       h->ntiles, U2, nMb, gpx, h->ws.s, M, h->ws.keys, h->ws.stats, temp, h->B,
                       h->ws.invT);
  else
    hipLaunchKernelGGL((k_lmhead_gemm<256, 256>), dim3(8 * per), dim3(kGWaves * kWave), 0, st,
                       (const uint16_t*)h->W_lm, (const uint16_t*)hidden, h->V, h->H, M,
                       h->ntiles, U2, nMb, gpx, h->ws.s, M, h->ws.keys, h->ws.stats, temp, h->B,
                       h->ws.invT);
  return hipGetLastError();
}

}  // namespace xp
