// A1 for many positions: s = W_lm h as a tiled GEMM on the bf16 matrix cores
// (v_mfma_f32_32x32x16_bf16), fused with the first stage of token selection.
//
// Once the position count M exceeds one 16-position block, streaming W_lm per
// block (the A1 stream kernels) would read the 1.2 GB head M/16 times; here
// every workgroup owns one selection unit of up to 256 vocabulary rows (16
// tiles, the unit partition of unit_tile_lo) and 256 positions, so W_lm is
// read once per 256 positions and the matrix cores, not HBM, bound the time
// at M = 512.  The tile order is XCD-aware: the position tiles of one unit run
// on the same XCD at the same time, so their reads of the unit's W_lm rows
// share that XCD's L2.
//
// Layout of the 32x32x16 operation (checked on gfx950): lane l holds row
// l % 32 of A and column l % 32 of B, k = 8 (l / 32) .. + 8; result register
// i of lane l is D[8 (i / 4) + 4 (l / 32) + i % 4][l % 32].  Here A = W_lm rows
// and B = h rows (positions), so D[row][position].
#include "xp_internal.h"

namespace xp {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kGK = 32;             // k per LDS stage
constexpr int kGWaves = 8;          // each wave: 128 rows x 64 positions (4 x 2 tiles of 32 x 32)
constexpr int kGLds = 163840 / 16;  // all of the 160 KB, in 16-byte slots

__device__ __forceinline__ floatx16 mma32(u32x4 a, u32x4 b, floatx16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// A stage row holds 32 k (64 B = four 16-byte chunks); chunk c of row r sits in
// slot 4 r + (c ^ swz(r)).  The swizzle makes the operand reads (32 rows, one
// chunk) conflict-free for both 32- and 64-bank LDS grouping.
__device__ __forceinline__ int gslot(int r, int c) { return 4 * r + (c ^ (((r >> 1) ^ (r >> 3)) & 3)); }

// Workgroup tile BN vocabulary rows (one selection unit of BN / 16 tiles) x BM
// positions; the 8 waves form a (BN / 128) x (BM / 64) grid, each owning a
// 128 x 64 block of D (128 accumulator registers), and per 16-wide k step a
// wave reads 4 + 2 operand fragments from LDS for 8 matrix operations.
//   BN = 256, BM = 256: up to 256 positions (one position tile).
//   BN = 128, BM = 512: 512 positions per tile, so W_lm is read once per 512
//     positions (the L2 cannot keep one workgroup's W_lm stages for a second
//     position tile) and h, 4 MB, is what the workgroups share through L2.
// Global data goes straight to LDS (global_load_lds_dwordx4, no staging
// registers) NS - 1 stages ahead of the stage being computed; a wave waits
// only for its own loads of the next stage, and the stage barrier does not
// drain the others.
template <int BN, int BM>
__global__ __launch_bounds__(kGWaves * kWave) void k_lmhead_gemm(
    const uint16_t* __restrict__ W, const uint16_t* __restrict__ X, int V, int H, int M,
    int ntiles, int U, int nMb, float* __restrict__ S, int Ms, uint64_t* __restrict__ keys,
    Stat* __restrict__ stats, const uint8_t* __restrict__ temp, int B) {
  constexpr int WS = BN * kGK * 2 / 16, HS = BM * kGK * 2 / 16;  // slots per operand stage
  constexpr int NS = kGLds / (WS + HS);                          // stages (5 or 4)
  constexpr int NWR = BN / 128;                                  // waves along the rows
  constexpr int WI = WS / 64 / kGWaves, HI = HS / 64 / kGWaves;  // 1 KB loads per wave and stage
  static_assert(NWR * (BM / 64) == kGWaves, "wave grid");
  __shared__ u32x4 lds[NS * (WS + HS)];                          // [stage][W | h]
  // XCD-aware tile order: workgroup b runs on XCD b % 8; its k-th workgroup
  // there takes unit 8 (k / nMb) + xcd and position tile k % nMb.
  const int b = blockIdx.x, xcd = b & 7, k8 = b >> 3;
  const int u = 8 * (k8 / nMb) + xcd, mb = k8 % nMb;
  if (u >= U) return;                                            // whole workgroup
  const int tlo = unit_tile_lo(u, ntiles, U), thi = unit_tile_lo(u + 1, ntiles, U);
  const int r0 = tlo * kTile, nrows = (thi - tlo) * kTile;      // <= BN rows
  const int p0 = mb * BM;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave % NWR, wp = wave / NWR;                    // 128-row block, 64-position block

  // loads of a stage: wave w fills W slots [64 WI w, 64 WI (w + 1)) and h slots
  // [64 HI w, 64 HI (w + 1)) with 1 KB instructions; lane l of an instruction
  // writes the next slot, i.e. row slot / 4, stored chunk l % 4, which holds
  // logical chunk (l % 4) ^ swz(row)
  int woff[WI], hoff[HI];
#pragma unroll
  for (int j = 0; j < WI; ++j) {
    const int row = (64 * (WI * wave + j) + lane) >> 2;
    const int c = (lane & 3) ^ (((row >> 1) ^ (row >> 3)) & 3);
    int wr = r0 + row;
    wr = wr < V ? wr : V - 1;
    woff[j] = wr * H + 8 * c;
  }
#pragma unroll
  for (int j = 0; j < HI; ++j) {
    const int row = (64 * (HI * wave + j) + lane) >> 2;
    const int c = (lane & 3) ^ (((row >> 1) ^ (row >> 3)) & 3);
    int hr = p0 + row;
    hr = hr < M ? hr : M - 1;
    hoff[j] = hr * H + 8 * c;
  }
  const int nk = H / kGK;
  auto issue = [&](int kc) {                                     // chunk kc (clamped) -> its stage
    const int st = kc % NS;
    const int kk = (kc < nk ? kc : nk - 1) * kGK;
#pragma unroll
    for (int j = 0; j < WI; ++j)
      lds_dma16(W + (size_t)(unsigned)woff[j] + kk, &lds[st * (WS + HS) + 64 * (WI * wave + j)]);
#pragma unroll
    for (int j = 0; j < HI; ++j)
      lds_dma16(X + (size_t)(unsigned)hoff[j] + kk, &lds[st * (WS + HS) + WS + 64 * (HI * wave + j)]);
  };

  floatx16 acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][c][i] = 0.f;

  const int lr = lane & 31, lk = lane >> 5;
  int arow[4], brow[2];
#pragma unroll
  for (int a = 0; a < 4; ++a) arow[a] = wv * 128 + a * 32 + lr;
#pragma unroll
  for (int c = 0; c < 2; ++c) brow[c] = wp * 64 + c * 32 + lr;

#pragma unroll
  for (int s = 0; s < NS - 1; ++s) issue(s);
  constexpr int kPend = (WI + HI) * (NS - 2);                    // loads of later stages in flight
  static_assert(kPend < 64, "vmcnt field");
  for (int kc = 0; kc < nk; ++kc) {
    // this wave's loads of chunk kc are done once at most kPend later loads
    // are outstanding; the barrier then covers every wave's loads of chunk kc
    // and every wave's reads of chunk kc - 1
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0x0f70 | (kPend & 15) | ((kPend >> 4) << 14));
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    issue(kc + NS - 1);                                          // into the stage read at kc - 1
    const int st = kc % NS;
    // both k steps' fragments first, so the second set of LDS reads overlaps
    // the first matrix operations
    u32x4 av[kGK / 16][4], bv[kGK / 16][2];
#pragma unroll
    for (int ks = 0; ks < kGK / 16; ++ks) {
      const int c = 2 * ks + lk;
#pragma unroll
      for (int a = 0; a < 4; ++a) av[ks][a] = lds[st * (WS + HS) + gslot(arow[a], c)];
#pragma unroll
      for (int cc = 0; cc < 2; ++cc) bv[ks][cc] = lds[st * (WS + HS) + WS + gslot(brow[cc], c)];
    }
#pragma unroll
    for (int ks = 0; ks < kGK / 16; ++ks)
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) acc[a][cc] = mma32(av[ks][a], bv[ks][cc], acc[a][cc]);
  }
  // drain the (clamped) loads issued past the last chunk before LDS is reused
  __builtin_amdgcn_s_waitcnt(0x0070);                            // vmcnt(0) lgkmcnt(0)
  __syncthreads();

  // --- epilogue: s straight from the accumulators; selection partials per
  //     position over this unit's rows (lanes l, l+32, then the row blocks) ---
  bool psamp[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int p = p0 + brow[c];
    psamp[c] = p < M && load_flag(temp, (p < M ? p : M - 1) / B, W) != 0;
  }
  const bool any_sample = __ballot(psamp[0] || psamp[1]) != 0;
  uint64_t* kr = reinterpret_cast<uint64_t*>(lds);               // [row block][BM positions]
  Stat* sr = reinterpret_cast<Stat*>(kr + NWR * BM);
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int p = p0 + brow[c];
    const bool pact = p < M;
    const bool psample = psamp[c];
    uint64_t best = kKeyMin;
    Stat st = stat_empty();
#pragma unroll
    for (int a = 0; a < 4; ++a) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int rl = wv * 128 + a * 32 + 8 * q + 4 * lk;       // local row of acc[a][c][4q]
        const bool rv = pact && rl < nrows;                      // nrows is a multiple of 16
        if (rv)
          *reinterpret_cast<float4*>(S + s_index(p, r0 + rl, Ms)) =
              make_float4(acc[a][c][4 * q], acc[a][c][4 * q + 1], acc[a][c][4 * q + 2],
                          acc[a][c][4 * q + 3]);
        // rows past V (the last unit's padding, computed from the clamped
        // row V-1) are stored into the padding of s but never selected
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool ev = rv && r0 + rl + e < V;
          const uint64_t key = umax64(best, argmax_key(acc[a][c][4 * q + e], (uint32_t)(r0 + rl + e)));
          best = (ev && !psample) ? key : best;
        }
        if (any_sample) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bool ev = rv && r0 + rl + e < V && psample;
            const Stat nx = stat_merge(st, Stat{acc[a][c][4 * q + e], 1.f});
            st.m = ev ? nx.m : st.m;
            st.s = ev ? nx.s : st.s;
          }
        }
      }
    }
    best = umax64(best, shfl_xor_u64(best, 32));
    const Stat o{__shfl_xor(st.m, 32, kWave), __shfl_xor(st.s, 32, kWave)};
    st = stat_merge(st, o);
    if (lk == 0) {
      kr[wv * BM + brow[c]] = best;
      sr[wv * BM + brow[c]] = st;
    }
  }
  __syncthreads();
  for (int pl = tid; pl < BM; pl += kGWaves * kWave) {
    const int p = p0 + pl;
    if (p < M) {
      uint64_t bb = kr[pl];
      Stat ss = sr[pl];
#pragma unroll
      for (int w = 1; w < NWR; ++w) {
        bb = umax64(bb, kr[w * BM + pl]);
        ss = stat_merge(ss, sr[w * BM + pl]);
      }
      keys[(size_t)u * M + p] = bb;
      stats[(size_t)u * M + p] = ss;
    }
  }
}

// ---------------------------------------------------------------------------
// Selection units of the GEMM path: 16 tiles (256 rows).  The launch and
// every reader of the per-unit partials use this one function.
int gemm_units(const xp_handle* h, int M) {
  (void)M;
  return (h->ntiles + 15) / 16;
}

bool lmhead_gemm_ok(const xp_handle* h, int M) {
  return h->dtype == XP_BF16 && M > kTile && h->H % kGK == 0;
}

hipError_t launch_lmhead_gemm(xp_handle* h, int M, const void* hidden, const uint8_t* temp,
                              hipStream_t st) {
  const int U = gemm_units(h, M);
  if (true) {                                  // 256 x 256 tiles for every M (measured faster)
    const int nMb = (M + 255) / 256;
    hipLaunchKernelGGL((k_lmhead_gemm<256, 256>), dim3(8 * nMb * ((U + 7) / 8)),
                       dim3(kGWaves * kWave), 0, st, (const uint16_t*)h->W_lm,
                       (const uint16_t*)hidden, h->V, h->H, M, h->ntiles, U, nMb, h->ws.s,
                       M, h->ws.keys, h->ws.stats, temp, h->B);
  } else {
    const int nMb = (M + 511) / 512;
    hipLaunchKernelGGL((k_lmhead_gemm<128, 512>), dim3(8 * nMb * ((U + 7) / 8)),
                       dim3(kGWaves * kWave), 0, st, (const uint16_t*)h->W_lm,
                       (const uint16_t*)hidden, h->V, h->H, M, h->ntiles, U, nMb, h->ws.s,
                       M, h->ws.keys, h->ws.stats, temp, h->B);
  }
  return hipGetLastError();
}

}  // namespace xp
