// The tiled bf16 GEMM pipeline on v_mfma_f32_32x32x16_bf16 shared by the
// LM-head GEMM (s = W_lm h with the selection partials, xp_gemm.hip) and the
// context layer's projections (y = X W^T, xp_lgemm.hip).  The callers differ
// only in which weight rows a tile covers (Rows) and in what they do with a
// finished tile (Epi).
//
// A tile is BN weight rows x BM positions, computed by 8 waves: wave w owns
// rows (w & 1) BN/2 .. + BN/2 and positions (w >> 1) BM/4 .. + BM/4 as
// 32 x 32 blocks.  k advances 32 per stage through an LDS ring of NS stages
// filled by global_load_lds_dwordx4 (no staging registers).  Only waves 0-3,
// one per SIMD (a workgroup's wave w runs on SIMD w mod 4), issue the loads:
// wave w < 4 fills W slots [64 WI w, 64 WI (w + 1)) and X slots
// [64 HI w, 64 HI (w + 1)) with 1 KB instructions (WI, HI for the 4 loading
// waves).  A load instruction can wait many cycles at issue while the
// address units work through the workgroup's 32 KB per stage (timestamps in
// a copy of the loop: 14% of a wave's time at 2048 positions); with every
// wave loading, both waves of a SIMD stall there at about the same time,
// while with one loading wave per SIMD the other one keeps issuing matrix
// operations.  Measured on the LM-head GEMM: 2-3% less time at 128 and 512
// positions, no change at 2048; waves 4-7 as the loading waves, or the loads
// split over both halves of a stage, were slower.
//
// A stage row holds 32 k (four 16-byte chunks); chunk c of row r sits in
// slot 4 r + (c ^ swz(r)), swz(r) = (r / 4) mod 4: four consecutive
// rows fill one 256-byte line of the 64 banks and the next three groups of
// four rotate their chunks, so an operand read (32 rows, one chunk) meets no
// bank conflict (SQ_LDS_BANK_CONFLICT reads zero; with swz(r) = ((r / 2) xor
// (r / 8)) mod 4 it counted conflicts on a fifth of the CU cycles and the
// GEMM ran 7-14% slower).  The ring runs on across tile boundaries, so the
// next tile's first stages load while the previous tile's epilogue runs.
//
// Layout of the 32x32x16 operation (checked on gfx950): lane l holds row
// l % 32 of A and column l % 32 of B, k = 8 (l / 32) .. + 8; result register i
// of lane l is D[8 (i / 4) + 4 (l / 32) + i % 4][l % 32].  A = weight rows,
// B = positions, so D[row][position].
#pragma once

#include "xp_device.h"

namespace xp {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kGK = 32;             // k per LDS stage
constexpr int kGWaves = 8;          // 2 (rows) x 4 (positions) waves
constexpr int kGLoaders = 4;        // waves that issue the stage loads (0 .. 3)
constexpr int kGPerXcd = 32;        // workgroups per XCD (one per CU)

__device__ __forceinline__ floatx16 mma32(u32x4 a, u32x4 b, floatx16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ int gswz(int r) { return (r >> 2) & 3; }
__device__ __forceinline__ int gslot(int r, int c) { return 4 * r + (c ^ gswz(r)); }

template <int BN, int BM>
struct GemmShape {
  static constexpr int RW = BN / 2, PW = BM / 4;                       // rows, positions per wave
  static constexpr int NA = RW / 32, NB = PW / 32;                     // 32 x 32 blocks per wave
  static constexpr int WS = BN * kGK * 2 / 16, HS = BM * kGK * 2 / 16; // slots per operand stage
  static constexpr int WI = WS / 64 / kGLoaders, HI = HS / 64 / kGLoaders; // 1 KB loads per loading wave
  static constexpr int NS0 = 163840 / ((WS + HS) * 16);
  static constexpr int NS = NS0 < 8 ? NS0 : 8;                         // ring stages
  static constexpr int SLOTS = NS * (WS + HS);
  static_assert(WI >= 1 && HI >= 1 && NA >= 1 && NB >= 1, "tile shape");
  static_assert(SLOTS * 16 <= 163840, "LDS");
};

// Where a wave sits in the tile, for the epilogues.
struct GemmLane {
  int wv, wp;        // row half, position block
  int lr, lk;        // lane % 32, lane / 32
};

// The ntl tiles of one workgroup for positions [p0, p0 + BM) of X (bf16 rows
// of ldx elements, rows past M read as row M - 1), each over K values of k.
// rows.prep(ti) selects tile ti's weight rows and its first k, rows.xk (an
// element offset into the X rows); rows.row(r) is then the address of its
// local row r (0 <= r < BN) at that k.  epi(ti, acc, where) consumes tile
// ti's accumulators; the pipeline clears them afterwards.  lds holds
// GemmShape<BN, BM>::SLOTS 16-byte slots.  Every tile walks its k chunks
// starting at chunk kshift (0 <= kshift < K / 32) and wrapping around.
template <int BN, int BM, class Rows, class Epi>
__device__ __forceinline__ void gemm_tiles(Rows& rows, Epi& epi, const uint16_t* __restrict__ X,
                                           int ldx, int M, int K, int ntl, int p0, u32x4* lds,
                                           int kshift = 0) {
  using G = GemmShape<BN, BM>;
  constexpr int RW = G::RW, PW = G::PW, NA = G::NA, NB = G::NB, WS = G::WS, HS = G::HS;
  constexpr int WI = G::WI, HI = G::HI, NS = G::NS;
  const int nk = K / kGK;
  const int nstages = ntl * nk;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  GemmLane where{wave & 1, wave >> 1, lane & 31, lane >> 5};
  const bool loader = wave < kGLoaders;                           // wave-uniform
  const int li = wave & (kGLoaders - 1);

  // lane l of a load instruction writes the next slot: LDS row slot / 4,
  // stored chunk l % 4, which holds logical chunk (l % 4) ^ swz(row)
  int wrow[WI], wcol[WI], hrow[HI];
#pragma unroll
  for (int j = 0; j < WI; ++j) {
    const int row = (64 * (WI * li + j) + lane) >> 2;
    wrow[j] = row;
    wcol[j] = 8 * ((lane & 3) ^ gswz(row));
  }
#pragma unroll
  for (int j = 0; j < HI; ++j) {
    const int row = (64 * (HI * li + j) + lane) >> 2;
    int hr = p0 + row;
    hr = hr < M ? hr : M - 1;
    hrow[j] = hr * ldx + 8 * ((lane & 3) ^ gswz(row));
  }
  int iss_tile = -1;                                               // tile whose rows are cached
  auto prep = [&](int gs) {
    gs = gs < nstages ? gs : nstages - 1;
    const int ti = gs / nk;
    if (ti != iss_tile) {                                          // wave-uniform
      iss_tile = ti;
      rows.prep(ti);
    }
  };
  auto issue = [&](int gs) {                                       // global stage gs (clamped)
    gs = gs < nstages ? gs : nstages - 1;
    const int ti = gs / nk, kq = gs - ti * nk + kshift, kc = kq < nk ? kq : kq - nk;
    const int st = gs % NS;
#pragma unroll
    for (int j = 0; j < WI; ++j)
      lds_dma16(rows.row(wrow[j]) + kc * kGK + wcol[j], &lds[st * (WS + HS) + 64 * (WI * li + j)]);
#pragma unroll
    for (int j = 0; j < HI; ++j)
      lds_dma16(X + (size_t)(unsigned)hrow[j] + rows.xk + kc * kGK,
                &lds[st * (WS + HS) + WS + 64 * (HI * li + j)]);
  };

  floatx16 acc[NA][NB];
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][c][i] = 0.f;

  // fragment reads of k step ks of global stage gs
  auto rd = [&](int gs, int ks, u32x4 (&av)[NA], u32x4 (&bv)[NB]) {
    const int base = (gs % NS) * (WS + HS);
    const int c = 2 * ks + where.lk;
#pragma unroll
    for (int a = 0; a < NA; ++a) av[a] = lds[base + gslot(where.wv * RW + a * 32 + where.lr, c)];
#pragma unroll
    for (int cc = 0; cc < NB; ++cc)
      bv[cc] = lds[base + WS + gslot(where.wp * PW + cc * 32 + where.lr, c)];
  };
  auto mm = [&](const u32x4 (&av)[NA], const u32x4 (&bv)[NB]) {
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int cc = 0; cc < NB; ++cc) acc[a][cc] = mma32(av[a], bv[cc], acc[a][cc]);
  };

#pragma unroll
  for (int s = 0; s < NS; ++s) {
    prep(s);
    if (loader) issue(s);
  }
  // (the other waves have no loads outstanding; for them the waits below
  // cover only the epilogue's stores)
  constexpr int kP0 = (WI + HI) * (NS - 1), kP = (WI + HI) * (NS - 2);
  static_assert(kP0 < 64, "vmcnt field");
  // stage 0 landed (this wave's loads), then every wave's
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0070 | (kP0 & 15) | ((kP0 >> 4) << 14));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  u32x4 fa[2][NA], fb[2][NB];               // fragment sets of the two k steps of a stage
  // the loading waves issue ahead of the others on their SIMD, so that the
  // stage loads (on which every wave's next barrier waits) go out first: 1-2%
  // less time at 512 positions, no change at 2048 (A/B on one box); raising it
  // only around the load issue instead gained nothing
  if (loader) __builtin_amdgcn_s_setprio(1);
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
    // issued after the barrier, behind the second half's matrix operations.
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
#pragma unroll
    for (int q = 0; q < NA + NB; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 16, 0);
    __builtin_amdgcn_sched_barrier(0);
    if (loader) issue(gs + NS);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_sched_barrier(0);
    if (++kc == nk) {                                              // wave-uniform
      epi(ti, acc, where);
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int c = 0; c < NB; ++c)
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[a][c][i] = 0.f;
      kc = 0;
      ++ti;
    }
  }
  __builtin_amdgcn_s_waitcnt(0x0070);        // the clamped loads past the end
}

// Workgroup (XCD xcd, index k8 on it) -> its i-th row tile:
// 8 (i gpx + k8 / nMb) + xcd, and position tile k8 % nMb.  The position tiles
// of one row tile run on the same XCD at about the same time, so their reads
// of the tile's rows share that XCD's L2.
struct GemmSched {
  int xcd, k8q, mb, gpx;
  __device__ GemmSched(int nMb, int gpx_) : gpx(gpx_) {
    xcd = blockIdx.x & 7;
    const int k8 = blockIdx.x >> 3;
    k8q = k8 / nMb;
    mb = k8 - k8q * nMb;
  }
  __device__ int tile(int i) const { return 8 * (i * gpx + k8q) + xcd; }
  // tiles of this workgroup among ntiles: i with tile(i) < ntiles
  __device__ int count(int ntiles) const {
    const int first = 8 * k8q + xcd;
    return first < ntiles ? (ntiles - first + 8 * gpx - 1) / (8 * gpx) : 0;
  }
};

// workgroups per XCD for nMb position tiles: whole groups of nMb
__host__ inline int gemm_per_xcd(int nMb) {
  const int per = kGPerXcd / nMb * nMb;
  return per > 0 ? per : nMb;
}

}  // namespace xp
