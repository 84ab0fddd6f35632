// A1: the base readout s = W_lm h (the target LM head read out on the drafter
// states, section 4.1 / Fig. 2a), fused with the first stage of token
// selection so that no logit row is ever re-read for it: per vocabulary unit
// the kernel leaves 64-bit argmax keys (greedy rows) or (max, sum exp(l - max))
// (sampled rows) next to the fp32 rows of s that the Jacobi passes add onto.
//
// W_lm is streamed exactly once per 16-position block; the 16 positions'
// activations stay on chip (LDS or registers) for the whole kernel.
#include "xp_internal.h"

namespace xp {

// ---------------------------------------------------------------------------
// A1: s = W_lm h.  Split-K across the waves of a workgroup: wave w owns k in
// [w*KS, (w+1)*KS) and keeps the 16 positions' h for that slice in registers;
// the per-wave 16x16 partial tiles are summed in LDS in a fixed wave order
// (deterministic), then written as fp32 s and folded into the selection state.
// One workgroup owns one vocabulary unit (a contiguous run of tiles).
// ---------------------------------------------------------------------------
template <typename T, int NU>
__global__ __launch_bounds__(1024) void k_lmhead(
    const T* __restrict__ W, const T* __restrict__ X, int V, int H, int M, int ntiles, int U,
    float* __restrict__ S, int Ms, uint64_t* __restrict__ keys, Stat* __restrict__ stats,
    const uint8_t* __restrict__ temp, int B, const float* __restrict__ invT) {
  using MF = Mfma<T>;
  constexpr int EPB = 16 / sizeof(T);
  constexpr int KS = NU * MF::KU;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, NW = blockDim.x >> 6;
  const int u = blockIdx.x, p0 = blockIdx.y * kTile;
  const int tlo = unit_tile_lo(u, ntiles, U), thi = unit_tile_lo(u + 1, ntiles, U);
  const size_t kofs = (size_t)wave * KS + (lane >> 4) * EPB;

  u32x4 bf[NU];
  {
    const int p = p0 + (lane & 15);
    const T* xr = X + (size_t)(p < M ? p : 0) * H + kofs;
#pragma unroll
    for (int i = 0; i < NU; ++i) bf[i] = (p < M) ? ld16(xr + i * MF::KU) : u32x4{0u, 0u, 0u, 0u};
  }

  __shared__ float red[16][kTile][20];   // [wave][position][row], rows padded to 20
  const int epos = threadIdx.x >> 4, erow = threadIdx.x & 15;
  const int ep = p0 + epos;
  const bool eact = threadIdx.x < 256 && ep < M;
  const bool esample = eact && temp != nullptr && temp[ep / B] != 0;
  const float eit = esample ? invT[ep / B] : 1.f;         // sampled rows: softmax(s / T)
  uint64_t best = kKeyMin;
  Stat st = stat_empty();

  auto load_tile = [&](int t, u32x4 (&a)[NU]) {
    int row = t * kTile + (lane & 15);
    row = row < V ? row : V - 1;
    const T* wr = W + (size_t)row * H + kofs;
#pragma unroll
    for (int i = 0; i < NU; ++i) a[i] = ld16_nt(wr + i * MF::KU);
  };

  u32x4 a[NU], an[NU];
  if (tlo < thi) load_tile(tlo, a);
  for (int t = tlo; t < thi; ++t) {
    if (t + 1 < thi) load_tile(t + 1, an);
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < NU; ++i) acc = MF::mma(a[i], bf[i], acc);
    *reinterpret_cast<floatx4*>(&red[wave][lane & 15][4 * (lane >> 4)]) = acc;
    __syncthreads();
    if (threadIdx.x < 256) {
      float v = 0.f;
      for (int w = 0; w < NW; ++w) v += red[w][epos][erow];
      const int row = t * kTile + erow;
      if (eact && row < V) {
        S[s_index(ep, row, Ms)] = v;
        if (esample)
          st = stat_merge(st, Stat{v * eit, 1.f});
        else
          best = umax64(best, argmax_key(v, (uint32_t)row));
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < NU; ++i) a[i] = an[i];
  }
  if (threadIdx.x < 256) {
#pragma unroll
    for (int m = 1; m < 16; m <<= 1) {
      best = umax64(best, shfl_xor_u64(best, m));
      Stat o{__shfl_xor(st.m, m, kWave), __shfl_xor(st.s, m, kWave)};
      st = stat_merge(st, o);
    }
    if (erow == 0 && ep < M) {
      keys[(size_t)u * M + ep] = best;
      stats[(size_t)ep * U + u] = st;
    }
  }
}

// ---------------------------------------------------------------------------
// A1, LDS variant (16 * H * sizeof(T) <= 128 KB): the 16 positions' h live in
// LDS (16-byte chunks XOR-swizzled by position so that the B-operand reads of a
// wave hit distinct banks), which frees registers for a three-deep ring of
// W_lm tiles in flight per wave.  Partial tiles go through a double-buffered
// LDS area, so one barrier per tile suffices.
// ---------------------------------------------------------------------------
constexpr int kHChunks = 512;          // 16-byte chunks of h per position (8 KB)

template <typename T, int NU>
__global__ __launch_bounds__(1024) void k_lmhead_lds(
    const T* __restrict__ W, const T* __restrict__ X, int V, int H, int M, int ntiles, int U,
    float* __restrict__ S, int Ms, uint64_t* __restrict__ keys, Stat* __restrict__ stats,
    const uint8_t* __restrict__ temp, int B, const float* __restrict__ invT) {
  using MF = Mfma<T>;
  constexpr int EPB = 16 / sizeof(T);
  constexpr int KS = NU * MF::KU;
  constexpr int CPU_ = MF::KU / EPB;                  // chunks per load unit (4)
  __shared__ u32x4 hl[16 * kHChunks];                 // 128 KB
  __shared__ floatx4 red[2][16][64];                  // 32 KB
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, NW = blockDim.x >> 6;
  const int u = blockIdx.x, p0 = blockIdx.y * kTile;
  const int tlo = unit_tile_lo(u, ntiles, U), thi = unit_tile_lo(u + 1, ntiles, U);
  const int nch = H / EPB;                            // chunks per position row

  for (int e = threadIdx.x; e < 16 * nch; e += blockDim.x) {
    const int p = e / nch, c = e % nch;
    const int cs = (c & ~15) | ((c & 15) ^ p);
    hl[p * kHChunks + cs] =
        (p0 + p < M) ? ld16(X + (size_t)(p0 + p) * H + (size_t)c * EPB) : u32x4{0u, 0u, 0u, 0u};
  }
  __syncthreads();

  const int li = lane & 15, g = lane >> 4;
  const int cbase = wave * (KS / EPB) + g;            // chunk of this lane's first unit
  const size_t kofs = (size_t)wave * KS + g * EPB;
  const int epos = threadIdx.x >> 4, erow = threadIdx.x & 15;
  const int ep = p0 + epos;
  const bool eact = threadIdx.x < 256 && ep < M;
  const bool esample = eact && temp != nullptr && temp[ep / B] != 0;
  const float eit = esample ? invT[ep / B] : 1.f;         // sampled rows: softmax(s / T)
  uint64_t best = kKeyMin;
  Stat st = stat_empty();
  int buf = 0;

  auto load_tile = [&](int t, u32x4 (&a)[NU]) {
    int row = t * kTile + li;
    row = row < V ? row : V - 1;
    const T* wr = W + (size_t)row * H + kofs;
#pragma unroll
    for (int i = 0; i < NU; ++i) a[i] = ld16_nt(wr + i * MF::KU);
  };
  auto step = [&](const u32x4 (&a)[NU], int t) {
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < NU; ++i) {
      const int c = cbase + i * CPU_;
      const u32x4 bfr = hl[li * kHChunks + ((c & ~15) | ((c & 15) ^ li))];
      acc = MF::mma(a[i], bfr, acc);
    }
    red[buf][wave][lane] = acc;
    __syncthreads();
    if (threadIdx.x < 256) {
      // red[.][w][lane'] holds rows 4*(lane'/16)+i of position lane'%16
      const int src = (erow >> 2) * 16 + epos, comp = erow & 3;
      float v = 0.f;
      for (int w = 0; w < NW; ++w) v += red[buf][w][src][comp];
      const int row = t * kTile + erow;
      if (eact && row < V) {
        S[s_index(ep, row, Ms)] = v;
        if (esample)
          st = stat_merge(st, Stat{v * eit, 1.f});
        else
          best = umax64(best, argmax_key(v, (uint32_t)row));
      }
    }
    buf ^= 1;
  };

  // Three register tiles in flight.  The steady-state loop has no conditional
  // loads, so the compiler's wait counts stay exact and never drain the ring;
  // the at most four remaining tiles are handled after it.
  u32x4 a0[NU], a1[NU], a2[NU];
  if (tlo < thi) load_tile(tlo, a0);
  if (tlo + 1 < thi) load_tile(tlo + 1, a1);
  int t = tlo;
  for (; t + 4 < thi; t += 3) {
    load_tile(t + 2, a2);
    step(a0, t);
    load_tile(t + 3, a0);
    step(a1, t + 1);
    load_tile(t + 4, a1);
    step(a2, t + 2);
  }
  if (t < thi) {
    if (t + 2 < thi) load_tile(t + 2, a2);
    step(a0, t);
  }
  if (t + 1 < thi) {
    if (t + 3 < thi) load_tile(t + 3, a0);
    step(a1, t + 1);
  }
  if (t + 2 < thi) step(a2, t + 2);
  if (t + 3 < thi) step(a0, t + 3);
  if (threadIdx.x < 256) {
#pragma unroll
    for (int m = 1; m < 16; m <<= 1) {
      best = umax64(best, shfl_xor_u64(best, m));
      Stat o{__shfl_xor(st.m, m, kWave), __shfl_xor(st.s, m, kWave)};
      st = stat_merge(st, o);
    }
    if (erow == 0 && ep < M) {
      keys[(size_t)u * M + ep] = best;
      stats[(size_t)ep * U + u] = st;
    }
  }
}

// ---------------------------------------------------------------------------
// A1, stream-K variant (bf16, 16 * H * 2 <= 128 KB).  W_lm is read with
// line-complete loads: an item is 16 rows x 64 k (2 KB), fetched by two
// instructions that each cover 8 rows x 128 B, then transposed through a
// per-wave 2 KB LDS tile into MFMA operand order; h (16 positions) lives in
// LDS for the whole kernel.  Every wave runs the full k range on its own
// contiguous share of the workgroup's (tile, k-group) items, so the main loop
// has no barrier.  A tile whose items straddle a wave boundary is finished
// once at the end: its partial tiles are added in wave order (= k order), so
// results do not depend on timing, batch or position block.
// ---------------------------------------------------------------------------
constexpr int kSkWaves = 16;
constexpr int kSkPF = 5;               // items in flight per wave

// XOR swizzle of the 8 16-byte chunks of a transpose-tile row: conflict-free
// for 8 consecutive lanes writing one row and for 16 lanes reading one chunk
// of 16 rows.
__device__ __forceinline__ int sk_slot(int row, int c) { return row * 8 + (c ^ ((row & 7) ^ (row >> 3))); }

// TT: the call gives temperatures (sampled rows scale by 1/T).  Without them
// the kernel keeps no 1/T register: it runs at its register limit, so the
// variant with temperatures keeps one item less in flight per wave.
template <int PF, bool TT>
__global__ __launch_bounds__(1024) void k_lmhead_sk(
    const uint16_t* __restrict__ W, const uint16_t* __restrict__ X, int V, int H, int M, int ntiles,
    int U, float* __restrict__ S, int Ms, uint64_t* __restrict__ keys, Stat* __restrict__ stats,
    const uint8_t* __restrict__ temp, int B, const float* __restrict__ invT) {
  using MF = Mfma<uint16_t>;
  __shared__ u32x4 lds[16 * kHChunks + kSkWaves * 128];   // h (128 KB) + transpose tiles (32 KB)
  u32x4* hl = lds;
  // the wave index is wave-uniform: make it a scalar, so that the item
  // bookkeeping below is scalar and never masks lanes
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  u32x4* tb = lds + 16 * kHChunks + wave * 128;
  const int u = blockIdx.x, p0 = blockIdx.y * kTile;
  const int tlo = unit_tile_lo(u, ntiles, U), thi = unit_tile_lo(u + 1, ntiles, U);
  const int nch = H / 8;                                  // 16-byte chunks per row
  const int G = H / 64;                                   // items per tile
  const int N = (thi - tlo) * G;
  auto wlo = [&](int w) { return (int)(((long)w * N) / kSkWaves); };
  const int i0 = wlo(wave), i1 = wlo(wave + 1);

  // the sampling flag of the lane's position first (its wait then covers no
  // other load), then h, then the first items of W_lm
  const int p_flag = p0 + (lane & 15);
  const int tvf = load_flag(temp, (p_flag < M ? p_flag : M - 1) / B, X);
  asm volatile("" ::: "memory");
  // h: every thread issues its (at most 8) chunk loads at once; rows past M
  // are loaded from row M-1 and zeroed
  constexpr int kHPer = 16 * kHChunks / (kSkWaves * kWave);
  u32x4 hv[kHPer];
#pragma unroll
  for (int j = 0; j < kHPer; ++j) {
    int e = threadIdx.x + kSkWaves * kWave * j;
    e = e < 16 * nch ? e : 0;
    const int pr = p0 + e / nch;
    hv[j] = ld16(X + (size_t)(pr < M ? pr : M - 1) * H + (size_t)(e % nch) * 8);
  }

  // load role: 8 lanes per row, lane -> (row ri of 8, chunk lc of 8)
  const int ri = lane >> 3, lc = lane & 7;
  // MFMA role: row / position li, k-group g
  const int li = lane & 15, g = lane >> 4;
  const int p = p0 + li;
  const bool pact = p < M;
  const bool psample = pact && tvf != 0;
  const bool any_sample = __ballot(psample) != 0;        // wave-uniform
  uint64_t best = kKeyMin;
  Stat st = stat_empty();

  // item counters of the next load: tile (relative) and k-group; frozen at the
  // wave's last item, so the loads past the end re-read it (no extra bytes)
  int lt = G > 0 ? i0 / G : 0, lq = i0 - lt * G, ln = i0;
  auto load_item = [&](u32x4 (&r)[2]) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      int row = (tlo + lt) * kTile + 8 * j + ri;
      row = row < V ? row : V - 1;
      r[j] = ld16_nt(W + (size_t)row * H + (size_t)(8 * lq + lc) * 8);
    }
    const int adv = ln + 1 < i1 ? 1 : 0;                  // scalar, branch-free
    ln += adv;
    lq += adv;
    const int wrap = lq == G ? 1 : 0;
    lq = wrap ? 0 : lq;
    lt += wrap;
  };
  // s of one finished tile, and its selection partials without branches on
  // the greedy path (every key is formed and kept or dropped by a select)
  float pit = 1.f;                                        // set after h is in LDS (TT)
  auto finalize = [&](floatx4 acc, int t) {
    const int row0 = t * kTile + 4 * g;
    if (pact)
      *reinterpret_cast<float4*>(S + s_index(p, row0, Ms)) = make_float4(acc[0], acc[1], acc[2], acc[3]);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool v = pact && row0 + i < V && !psample;
      const uint64_t key = umax64(best, argmax_key(acc[i], (uint32_t)(row0 + i)));
      best = v ? key : best;
    }
    if (any_sample) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool v = pact && row0 + i < V && psample;
        const Stat nx = stat_merge(st, Stat{acc[i] * pit, 1.f});
        st.m = v ? nx.m : st.m;
        st.s = v ? nx.s : st.s;
      }
    }
  };

  const int tf = G > 0 ? i0 / G : 0;                      // first (relative) tile of the wave
  floatx4 acc = {0.f, 0.f, 0.f, 0.f}, part0 = acc, part1 = acc;
  int ct = tf, cq = i0 - tf * G;                          // item being computed
  auto step = [&](const u32x4 (&r)[2], int i) {
#pragma unroll
    for (int j = 0; j < 2; ++j) tb[sk_slot(8 * j + ri, lc)] = r[j];
    wave_lds_order();
#pragma unroll
    for (int uu = 0; uu < 2; ++uu) {
      const int c = 4 * uu + g;
      const u32x4 a = tb[sk_slot(li, c)];
      const int cc = 8 * cq + c;
      const u32x4 b = hl[li * kHChunks + ((cc & ~15) | ((cc & 15) ^ li))];
      acc = MF::mma(a, b, acc);
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
  u32x4 ring[PF][2];
  if (i0 < i1) {
#pragma unroll
    for (int q = 0; q < PF; ++q) load_item(ring[q]);
  }
  asm volatile("" ::: "memory");
  // no guard on the stores (a guarded store would sink its load): chunks past
  // 16 * nch were loaded from chunk 0 and rewrite chunk 0's slot with its value
#pragma unroll
  for (int j = 0; j < kHPer; ++j) {
    int e = threadIdx.x + kSkWaves * kWave * j;
    e = e < 16 * nch ? e : 0;
    const int pp = e / nch, c = e % nch;
    hl[pp * kHChunks + ((c & ~15) | ((c & 15) ^ pp))] =
        p0 + pp < M ? hv[j] : u32x4{0u, 0u, 0u, 0u};
  }
  lds_barrier();                                          // h is in LDS; items stay in flight
  // 1/T of the lane's position for the sampled rows' partials (softmax(s / T)),
  // loaded once h's registers are free
  if constexpr (TT) pit = invT[(p_flag < M ? p_flag : M - 1) / B];
  if (i0 < i1) {
    int i = i0;
    for (; i + PF <= i1; i += PF) {
#pragma unroll
      for (int q = 0; q < PF; ++q) {
        step(ring[q], i + q);
        load_item(ring[q]);
      }
    }
#pragma unroll
    for (int q = 0; q < PF; ++q)
      if (i + q < i1) step(ring[q], i + q);
  }

  // tiles split between waves: partial tiles through LDS (the h area is free)
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
      for (int w = wave + 1; w < kSkWaves && wlo(w) < (tfin + 1) * G; ++w) {
        if (wlo(w + 1) > wlo(w)) {
          const floatx4 o = fx[(w * 2 + 0) * 64 + lane];
          a[0] += o[0]; a[1] += o[1]; a[2] += o[2]; a[3] += o[3];
        }
      }
      finalize(a, tlo + tfin);
    }
  }
  // per-position selection partials: lanes of one position, then waves in order
#pragma unroll
  for (int m = 16; m < 64; m <<= 1) {
    best = umax64(best, shfl_xor_u64(best, m));
    Stat o{__shfl_xor(st.m, m, kWave), __shfl_xor(st.s, m, kWave)};
    st = stat_merge(st, o);
  }
  uint64_t* kr = reinterpret_cast<uint64_t*>(lds + 2 * kSkWaves * 64);   // past fx
  Stat* sr = reinterpret_cast<Stat*>(kr + kSkWaves * 16);
  if (lane < 16) {
    kr[wave * 16 + lane] = best;
    sr[wave * 16 + lane] = st;
  }
  __syncthreads();
  if (threadIdx.x < 16) {
    uint64_t bb = kKeyMin;
    Stat ss = stat_empty();
    for (int w = 0; w < kSkWaves; ++w) {
      bb = umax64(bb, kr[w * 16 + threadIdx.x]);
      ss = stat_merge(ss, sr[w * 16 + threadIdx.x]);
    }
    const int pp = p0 + threadIdx.x;
    if (pp < M) {
      keys[(size_t)u * M + pp] = bb;
      stats[(size_t)pp * U + u] = ss;
    }
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
// Waves per workgroup and load units per wave for a hidden width H: the k
// range is split into NW slices of NU*KU values with 4 <= NW <= 16.
static bool pick_lm_split(int H, int KU, int* NU, int* NW) {
  for (int nu = 1; nu <= 16; nu *= 2) {
    if (H % (nu * KU)) continue;
    const int nw = H / (nu * KU);
    if (nw >= 4 && nw <= 16) {
      *NU = nu;
      *NW = nw;
      return true;
    }
  }
  return false;
}

bool lm_split_ok(int H, int dtype) {
  int nu, nw;
  return pick_lm_split(H, dtype == XP_BF16 ? 32 : 16, &nu, &nw);
}

template <typename T>
static hipError_t launch_lmhead_t(xp_handle* h, int M, const void* hidden, const uint8_t* temp,
                                  hipStream_t st) {
  int NU = 0, NW = 0;
  if (!pick_lm_split(h->H, Mfma<T>::KU, &NU, &NW)) return hipErrorInvalidValue;
  dim3 grid(h->lm_chunks, (M + kTile - 1) / kTile), block(NW * kWave);
  const bool lds = (size_t)h->H * sizeof(T) <= 16u * kHChunks;
  if constexpr (sizeof(T) == 2) {
    if (lds) {
      if (h->call_tempered)
        hipLaunchKernelGGL((k_lmhead_sk<kSkPF - 1, true>), grid, dim3(kSkWaves * kWave), 0, st,
                           (const uint16_t*)h->W_lm, (const uint16_t*)hidden, h->V, h->H, M,
                           h->ntiles, h->lm_chunks, h->ws.s, M, h->ws.keys, h->ws.stats, temp,
                           h->B, h->ws.invT);
      else
        hipLaunchKernelGGL((k_lmhead_sk<kSkPF, false>), grid, dim3(kSkWaves * kWave), 0, st,
                           (const uint16_t*)h->W_lm, (const uint16_t*)hidden, h->V, h->H, M,
                           h->ntiles, h->lm_chunks, h->ws.s, M, h->ws.keys, h->ws.stats, temp,
                           h->B, h->ws.invT);
      return hipGetLastError();
    }
  }
  auto args = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, block, 0, st, (const T*)h->W_lm, (const T*)hidden, h->V, h->H,
                       M, h->ntiles, h->lm_chunks, h->ws.s, M, h->ws.keys, h->ws.stats, temp,
                       h->B, h->ws.invT);
  };
  if (lds) {
    switch (NU) {
      case 1: args(k_lmhead_lds<T, 1>); break;
      case 2: args(k_lmhead_lds<T, 2>); break;
      case 4: args(k_lmhead_lds<T, 4>); break;
      case 8: args(k_lmhead_lds<T, 8>); break;
      default: args(k_lmhead_lds<T, 16>); break;
    }
  } else {
    switch (NU) {
      case 1: args(k_lmhead<T, 1>); break;
      case 2: args(k_lmhead<T, 2>); break;
      case 4: args(k_lmhead<T, 4>); break;
      case 8: args(k_lmhead<T, 8>); break;
      default: args(k_lmhead<T, 16>); break;
    }
  }
  return hipGetLastError();
}

hipError_t launch_lmhead(xp_handle* h, int M, const void* hidden, const uint8_t* temp,
                         hipStream_t st) {
  if (lmhead_gemm_ok(h, M)) {                 // many positions: one GEMM instead of M/16 streams
    h->lm_units_cur = gemm_units(h, M);
    return launch_lmhead_gemm(h, M, hidden, temp, st);
  }
  h->lm_units_cur = h->lm_chunks;
  if (h->dtype == XP_BF16) return launch_lmhead_t<uint16_t>(h, M, hidden, temp, st);
  return launch_lmhead_t<float>(h, M, hidden, temp, st);
}

}  // namespace xp
