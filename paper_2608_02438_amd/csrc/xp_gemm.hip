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

namespace xp {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kGK = 32;             // k per LDS stage
constexpr int kGWaves = 8;          // 2 (rows) x 4 (positions) waves
constexpr int kGPerXcd = 32;        // workgroups per XCD (one per CU)

__device__ __forceinline__ floatx16 mma32(u32x4 a, u32x4 b, floatx16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// A stage row holds 32 k (64 B = four 16-byte chunks); chunk c of row r sits in
// slot 4 r + (c ^ swz(r)).  The swizzle makes the operand reads (32 rows, one
// chunk) conflict-free.
__device__ __forceinline__ int gslot(int r, int c) { return 4 * r + (c ^ (((r >> 1) ^ (r >> 3)) & 3)); }

// Workgroup (XCD xcd, index k8 on it) -> its i-th tile: unit slot
// s = i * gpx + k8 / nMb (unit u = 8 s + xcd), position tile k8 % nMb.
struct GemmSched {
  int xcd, k8q, mb, gpx;
  __device__ int unit(int i) const { return 8 * (i * gpx + k8q) + xcd; }
};

template <int BN, int BM>
__global__ __launch_bounds__(kGWaves * kWave) void k_lmhead_gemm(
    const uint16_t* __restrict__ W, const uint16_t* __restrict__ X, int V, int H, int M,
    int ntiles, int U2, int nMb, int gpx, float* __restrict__ S, int Ms,
    uint64_t* __restrict__ keys, Stat* __restrict__ stats, const uint8_t* __restrict__ temp,
    int B, const float* __restrict__ invT) {
  constexpr int RW = BN / 2, PW = BM / 4;                          // rows, positions per wave
  constexpr int NA = RW / 32, NB = PW / 32;                        // 32 x 32 blocks per wave
  constexpr int WS = BN * kGK * 2 / 16, HS = BM * kGK * 2 / 16;    // slots per operand stage
  constexpr int WI = WS / 64 / kGWaves, HI = HS / 64 / kGWaves;    // 1 KB loads per wave
  constexpr int NS0 = 163840 / ((WS + HS) * 16);
  constexpr int NS = NS0 < 8 ? NS0 : 8;                            // ring stages
  static_assert(WI >= 1 && HI >= 1 && NA >= 1 && NB >= 1, "tile shape");
  static_assert(NS * (WS + HS) * 16 <= 163840, "LDS");
  __shared__ u32x4 lds[NS * (WS + HS)];                            // [stage][W | h]

  const int Upair = U2 / 2;
  GemmSched sc;
  sc.xcd = blockIdx.x & 7;
  const int k8 = blockIdx.x >> 3;
  sc.k8q = k8 / nMb;
  sc.mb = k8 % nMb;
  sc.gpx = gpx;
  // tiles of this workgroup: i with unit(i) < Upair
  const int first = 8 * sc.k8q + sc.xcd;
  const int ntl = first < Upair ? (Upair - first + 8 * gpx - 1) / (8 * gpx) : 0;
  if (ntl == 0) return;                                            // whole workgroup
  const int nk = H / kGK;
  const int nstages = ntl * nk;
  const int p0 = sc.mb * BM;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave & 1, wp = wave >> 1;                         // unit, position block

  // stage loads: wave w fills W slots [64 WI w, 64 WI (w + 1)) and h slots
  // [64 HI w, 64 HI (w + 1)) with 1 KB instructions; lane l of an instruction
  // writes the next slot, i.e. LDS row slot / 4, stored chunk l % 4, which
  // holds logical chunk (l % 4) ^ swz(row).  LDS W row R is row R % RW of
  // unit 2u + R / RW (rows past the unit are loaded, never used).
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
    hrow[j] = hr * H + 8 * ((lane & 3) ^ (((row >> 1) ^ (row >> 3)) & 3));
  }
  // first rows of the two units of the tile being issued (cached per tile)
  int iss_tile = -1, iss_r0 = 0, iss_r1 = 0;
  auto prep = [&](int gs) {                                        // first rows of stage gs
    gs = gs < nstages ? gs : nstages - 1;
    const int ti = gs / nk;
    if (ti != iss_tile) {                                          // wave-uniform
      const int u = sc.unit(ti);
      iss_tile = ti;
      iss_r0 = unit_tile_lo(2 * u, ntiles, U2) * kTile;
      iss_r1 = unit_tile_lo(2 * u + 1, ntiles, U2) * kTile;
    }
  };
  auto issue = [&](int gs) {                                       // global stage gs (clamped)
    gs = gs < nstages ? gs : nstages - 1;
    const int ti = gs / nk, kc = gs - ti * nk;
    const int st = gs % NS;
#pragma unroll
    for (int j = 0; j < WI; ++j) {
      int r = (wrow[j] < RW ? iss_r0 : iss_r1) + (wrow[j] % RW);
      r = r < V ? r : V - 1;
      lds_dma16(W + (size_t)r * H + kc * kGK + wcol[j], &lds[st * (WS + HS) + 64 * (WI * wave + j)]);
    }
#pragma unroll
    for (int j = 0; j < HI; ++j)
      lds_dma16(X + (size_t)(unsigned)hrow[j] + kc * kGK,
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
  // fragment reads of k step ks of global stage gs
  auto rd = [&](int gs, int ks, u32x4 (&av)[NA], u32x4 (&bv)[NB]) {
    const int base = (gs % NS) * (WS + HS);
    const int c = 2 * ks + lk;
#pragma unroll
    for (int a = 0; a < NA; ++a) av[a] = lds[base + gslot(wv * RW + a * 32 + lr, c)];
#pragma unroll
    for (int cc = 0; cc < NB; ++cc) bv[cc] = lds[base + WS + gslot(wp * PW + cc * 32 + lr, c)];
  };
  auto mm = [&](const u32x4 (&av)[NA], const u32x4 (&bv)[NB]) {
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int cc = 0; cc < NB; ++cc) acc[a][cc] = mma32(av[a], bv[cc], acc[a][cc]);
  };

  // The position tile is fixed per workgroup, so the sampling flags and 1/T
  // of this wave's positions are loaded once, before the stage loads, and
  // waited for here: no epilogue then waits for a load.
  bool psamp[NB];
  float pit[NB];                                   // sampled rows: softmax(s / T)
  bool anyp = false;
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    const int p = p0 + wp * PW + c * 32 + lr;
    const int pc = p < M ? p : M - 1;
    psamp[c] = (p < M) & (load_flag(temp, pc / B, W) != 0);
    pit[c] = invT[pc / B];
    anyp = anyp | psamp[c];
  }
  const bool any_sample = __ballot(anyp) != 0;
#pragma unroll
  for (int c = 0; c < NB; ++c) asm volatile("" ::"v"(pit[c]));
  // epilogue of tile ti: s from the accumulators, and the selection partials
  // of this wave's unit for its PW positions
  auto epilogue = [&](int ti) {
    const int hu = 2 * sc.unit(ti) + wv;
    const int rbase = unit_tile_lo(hu, ntiles, U2) * kTile;
    const int nr = unit_tile_lo(hu + 1, ntiles, U2) * kTile - rbase;   // <= RW, multiple of 16
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      const int p = p0 + wp * PW + c * 32 + lr;
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
          const int rl = a * 32 + 8 * q + 4 * lk;                  // local row of acc[a][c][4q]
          const bool rv = pact && rl < nr;
          if (rv)
            *reinterpret_cast<float4*>(S + s_index(p, rbase + rl, Ms)) =
                make_float4(acc[a][c][4 * q], acc[a][c][4 * q + 1], acc[a][c][4 * q + 2],
                            acc[a][c][4 * q + 3]);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float x = acc[a][c][4 * q + e];
            const bool take = rv && !psample && rbase + rl + e < V && x > bvv;
            bvv = take ? x : bvv;
            bix = take ? (uint32_t)(rbase + rl + e) : bix;
          }
          if (any_sample) {
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
      if (lk == 0 && pact) {
        keys[(size_t)hu * M + p] = best;
        if (psample) stats[(size_t)p * U2 + hu] = st;
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
    // k step 1 of stage gs is read while k step 0 multiplies; the barrier
    // between the two k steps (wait: stage gs + 1 landed for this wave, and
    // this wave's reads of stage gs are done) makes stage gs + 1 readable for
    // everyone and frees the slot of stage gs for stage gs + NS.  Other
    // vector-memory operations (the epilogue's stores) only make the wait
    // stricter.  In both halves the fragment reads of the next k step go
    // one by one between the matrix operations of the current one (the
    // scheduling groups below), so the LDS reads overlap the matrix pipe; the
    // row bookkeeping of stage gs + NS runs before the wait and its loads are
    // issued after the barrier, behind those reads.
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
  // workgroups per XCD: a multiple of the position tiles per unit
  int per = kGPerXcd / nMb * nMb;
  per = per > 0 ? per : nMb;
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
