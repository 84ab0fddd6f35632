// A7: Read + Correct, l = s + W_r z (eqs. read, correct), fused with the first
// stage of token selection: per vocabulary unit the kernel leaves argmax keys
// (greedy rows) or (max, sum exp(l - max)) (sampled rows); no logit row is
// written on the fast path.
//
// W_r is streamed once per pass and 16-position block, tile by tile (16
// vocabulary rows), straight into MFMA operand registers.
#include "xp_internal.h"
#include "xp_tiles.h"

namespace xp {

// ---------------------------------------------------------------------------
// A7: l = s + W_r z, r = 256.  Every wave streams its own unit of tiles with
// the full k range (one chain of MFMAs per tile, seeded with s); the position
// block's z fragments sit in LDS, shared by the waves.  A unit of at most
// kReadRes tiles (the common case) keeps all of them in registers: every W_r,
// s and z load of the wave is issued, unconditionally, before the first
// MFMA, so the whole unit is in flight at once (a short unit re-reads its
// last tile, which hits in L2).  Workgroups merge their waves' argmax keys;
// sampled rows write one (max, sum) per wave unit.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kReadWaves * kWave) void k_read(
    const T* __restrict__ W, const T* __restrict__ Z, const float* __restrict__ S, int Ms, int V,
    int M, int ntiles, int U, uint64_t* __restrict__ keys, Stat* __restrict__ stats,
    const uint8_t* __restrict__ temp, int B, float* __restrict__ out_logits,
    const int32_t* __restrict__ ctrl, int skip_when_done, const float* __restrict__ invT) {
  if (skip_when_done && ctrl[1]) return;          // every sequence is at its fixed point
  constexpr int NU = ReadTile<T>::NU;
  constexpr int NR = sizeof(T) == 2 ? 5 : 2;      // resident tiles per wave (32 / 64 VGPRs each)
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int u = blockIdx.x * kReadWaves + wave, p0 = blockIdx.y * kTile;
  const int tlo = unit_tile_lo(u, ntiles, U), thi = unit_tile_lo(u + 1, ntiles, U);
  const int n = thi - tlo;
  __shared__ u32x4 zl[NU][64];
  __shared__ uint64_t kred[kReadWaves][kTile];
  // per-wave transpose tile (16 rows x 32 chunks, chunk XOR-swizzled by row:
  // conflict-free for the row-contiguous writes and the MFMA-order reads)
  __shared__ u32x4 tbuf[sizeof(T) == 2 ? kReadWaves : 1][16 * 32];

  const int p = p0 + (lane & 15);
  const bool act = p < M;
  const int pc = act ? p : M - 1;
  const float pit = invT[pc / B];               // sampled rows: softmax(l / T)
  uint64_t best = kKeyMin;
  Stat st = stat_empty();
  bool sample = false;

  bool any_sample = false;                      // wave-uniform: some lane of the wave samples
  // Selection partials of one tile, without branches on the greedy path: the
  // key of every element is formed and kept or dropped by a select.
  auto epilogue = [&](const floatx4& acc, int t) {
    const int row0 = t * kTile + 4 * (lane >> 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool v = act && row0 + i < V && !sample;
      const uint64_t key = umax64(best, argmax_key(acc[i], (uint32_t)(row0 + i)));
      best = v ? key : best;
    }
    if (any_sample) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool v = act && row0 + i < V && sample;
        const Stat nx = stat_merge(st, Stat{acc[i] * pit, 1.f});
        st.m = v ? nx.m : st.m;
        st.s = v ? nx.s : st.s;
      }
    }
    if (out_logits) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (act && row0 + i < V) out_logits[(size_t)p * V + row0 + i] = acc[i];
    }
  };
  // z fragments, read once from LDS into registers after the barrier
  u32x4 zr[NU];
  auto fetch_z = [&]() {
#pragma unroll
    for (int i = 0; i < NU; ++i) zr[i] = zl[i][lane];
  };
  auto chain_lds = [&](const u32x4 (&a)[NU], floatx4 acc) {
#pragma unroll
    for (int i = 0; i < NU; ++i) acc = Mfma<T>::mma(a[i], zr[i], acc);
    return acc;
  };
  auto load_s = [&](int t) {
    const floatx4 v = *reinterpret_cast<const floatx4*>(S + s_index(pc, t * kTile + 4 * (lane >> 4), Ms));
    return act ? v : floatx4{0.f, 0.f, 0.f, 0.f};
  };
  // z fragments of the position block, one 16-byte chunk per thread
  constexpr int kZPer = (NU * 64 + kReadWaves * kWave - 1) / (kReadWaves * kWave);
  u32x4 zv[kZPer];
  auto load_z = [&]() {
#pragma unroll
    for (int j = 0; j < kZPer; ++j) {
      const int c = threadIdx.x + kReadWaves * kWave * j;
      const int zi = (c / 64) % NU, zlane = c % 64;
      const int zp = p0 + (zlane & 15);
      zv[j] = ld16(Z + (size_t)(zp < M ? zp : M - 1) * 256 + (zlane >> 4) * ReadTile<T>::EPB +
                   zi * ReadTile<T>::KU);
      if (zp >= M) zv[j] = u32x4{0u, 0u, 0u, 0u};
    }
  };
  static_assert(NU * 64 == kZPer * kReadWaves * kWave, "z chunks fill the workgroup exactly");
  auto put_z = [&]() {                          // no guard: a guarded store would sink its load
#pragma unroll
    for (int j = 0; j < kZPer; ++j) {
      const int c = threadIdx.x + kReadWaves * kWave * j;
      zl[c / 64][c % 64] = zv[j];
    }
  };

  if constexpr (sizeof(T) == 2) {
    if (n >= 1 && n <= NR) {
      // Line-complete loads: instruction i of a tile reads its rows 2i, 2i+1
      // (1 KB contiguous, non-temporal); each tile is then transposed through
      // the wave's LDS tile into the MFMA operand order of ReadTile::load_w,
      // so the chain sees exactly the operands of the rescans.
      // Issue order = use order (z, s, then the tiles): the vector-memory
      // counter drains in order, so tile j waits only for the loads before it.
      u32x4 a[NR][8];
      floatx4 c[NR];
      const int lrow = lane >> 5, lch = lane & 31;
      const int tv = load_flag(temp, pc / B, S);
      load_z();
      asm volatile("" ::: "memory");
#pragma unroll
      for (int j = 0; j < NR; ++j) c[j] = load_s(tlo + (j < n ? j : n - 1));
      asm volatile("" ::: "memory");
#pragma unroll
      for (int j = 0; j < NR; ++j) {
        const int t = tlo + (j < n ? j : n - 1);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          int row = t * kTile + 2 * i + lrow;
          row = row < V ? row : V - 1;
          a[j][i] = ld16_nt(W + (size_t)row * 256 + lch * 8);
        }
      }
      sample = act && tv != 0;
      any_sample = __ballot(sample) != 0;
      put_z();
      lds_barrier();
      fetch_z();
      u32x4* tb = tbuf[wave];
      const int li = lane & 15, g = lane >> 4;
#pragma unroll
      for (int j = 0; j < NR; ++j) {
        if (j < n) {
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const int row = 2 * i + lrow;
            tb[row * 32 + (lch ^ row)] = a[j][i];
          }
          wave_lds_order();
          u32x4 m[NU];
#pragma unroll
          for (int i = 0; i < NU; ++i) m[i] = tb[li * 32 + ((4 * i + g) ^ li)];
          wave_lds_order();
          epilogue(chain_lds(m, c[j]), tlo + j);
        }
      }
    } else {
      load_z();
      const int tv = load_flag(temp, pc / B, S);
      sample = act && tv != 0;
      any_sample = __ballot(sample) != 0;
      put_z();
      __syncthreads();
      fetch_z();
      u32x4 a[NU];
      for (int t = tlo; t < thi; ++t) {
        ReadTile<T>::load_w(W, V, t, lane, a);
        epilogue(chain_lds(a, load_s(t)), t);
      }
    }
  } else if (n >= 1 && n <= NR) {
    u32x4 a[NR][NU];
    floatx4 c[NR];
#pragma unroll
    for (int j = 0; j < NR; ++j) ReadTile<T>::load_w(W, V, tlo + (j < n ? j : n - 1), lane, a[j]);
#pragma unroll
    for (int j = 0; j < NR; ++j) c[j] = load_s(tlo + (j < n ? j : n - 1));
    load_z();
    const int tv = load_flag(temp, pc / B, S);
    sample = act && tv != 0;
    any_sample = __ballot(sample) != 0;
    put_z();
    __syncthreads();
    fetch_z();
#pragma unroll
    for (int j = 0; j < NR; ++j)
      if (j < n) epilogue(chain_lds(a[j], c[j]), tlo + j);
  } else {
    load_z();
    const int tv = load_flag(temp, pc / B, S);
    sample = act && tv != 0;
    any_sample = __ballot(sample) != 0;
    put_z();
    __syncthreads();
    fetch_z();
    u32x4 a[NU];
    for (int t = tlo; t < thi; ++t) {
      ReadTile<T>::load_w(W, V, t, lane, a);
      epilogue(chain_lds(a, load_s(t)), t);
    }
  }
#pragma unroll
  for (int m = 16; m < 64; m <<= 1) {
    best = umax64(best, shfl_xor_u64(best, m));
    Stat o{__shfl_xor(st.m, m, kWave), __shfl_xor(st.s, m, kWave)};
    st = stat_merge(st, o);
  }
  if (lane < 16 && sample) stats[(size_t)p * U + u] = st;

  if (lane < 16) kred[wave][lane] = best;
  __syncthreads();
  if (threadIdx.x < kTile) {
    uint64_t b = kKeyMin;
    for (int w = 0; w < kReadWaves; ++w) b = umax64(b, kred[w][threadIdx.x]);
    const int pp = p0 + threadIdx.x;
    if (pp < M) keys[(size_t)blockIdx.x * M + pp] = b;
  }
}

// ---------------------------------------------------------------------------
// A7 for many positions.  The stream kernel above re-reads W_r once per
// 16-position block; here a workgroup takes the tiles of one read workgroup
// (8 wave units) for 128 P positions: each wave keeps the z fragments of its
// 16 P positions in registers and runs through all the workgroup's tiles, so
// W_r is read once per 128 P positions and the pass is bound by reading s.
// The W_r tile and the s operands of every tile go through a ring of LDS
// stages filled by global-to-LDS loads three tiles ahead (each wave loads one
// 1 KB part of the W_r tile and the s of its own positions), so up to 100 KB
// per CU is in flight without staging registers.  Each (tile, 16 positions)
// product is the chain of matrix operations seeded with s used by the stream
// kernel and the sampling rescan (ReadTile), so all of them produce the same
// fp32 logits.  Outputs have the stream kernel's layout: one key row per
// workgroup, one (max, sum) per wave unit and position.
constexpr int kRmLds = 163840;                   // bytes of LDS the ring may take
constexpr int kRmMaxStages = 8;
constexpr int kRmMaxP = 4;                       // position blocks per wave (launch cap)

// W_r tile in LDS: 16 rows x 32 chunks of 16 bytes, chunk c of row r at slot
// 32 r + (c ^ r); s of 16 positions x 16 rows: chunk c (4 rows) of position q
// at slot 4 q + (c ^ (q / 4)).  The fragment reads (16 rows or positions, one
// chunk) then hit 16 different bank groups.
__device__ __forceinline__ int rm_wslot(int r, int c) { return 32 * r + (c ^ r); }
__device__ __forceinline__ int rm_sslot(int q, int c) { return 4 * q + ((c ^ (q >> 2)) & 3); }

// EE (early exit): a wave whose positions all belong to sequences at their
// fixed point is dead: its s loads go to one fixed address (every wave still
// issues the same number of loads per tile, which the waits count on, and its
// part of each W_r tile, which the other waves read), and its products,
// selection partials and outputs are skipped.
template <int P, bool EE>
__global__ __launch_bounds__(kReadWaves * kWave) void k_read_multi(
    const uint16_t* __restrict__ W, const uint16_t* __restrict__ Z, const float* __restrict__ S,
    int Ms, int V, int M, int ntiles, int U, uint64_t* __restrict__ keys,
    Stat* __restrict__ stats, const uint8_t* __restrict__ temp, int B,
    float* __restrict__ out_logits, const int32_t* __restrict__ ctrl, int skip_when_done,
    int nwg, int ny, int gs, const float* __restrict__ invT, const int32_t* __restrict__ iters) {
  static_assert(kReadWaves == 8, "one 1 KB load per wave fills a 16-row tile");
  if (skip_when_done && ctrl[1]) return;          // every sequence is at its fixed point
  using RT = ReadTile<uint16_t>;
  constexpr int NU = RT::NU;
  constexpr int WSL = 512, SSL = kReadWaves * P * 64;          // 16-byte slots per stage
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // A workgroup takes the gs consecutive read workgroups [g_lo, g_hi) (their
  // tiles in order, one key row per read workgroup) for position group py.
  // Workgroup b runs on XCD b % 8; the ny position groups of one group of
  // read workgroups sg are b = 8 (ny (sg / 8) + y) + sg % 8, y < ny: the
  // same XCD at about the same time, so W_r tiles read by the first come
  // from L2 for the others
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int sg = (slot / ny) * 8 + xcd, py = slot - (slot / ny) * ny;
  const int g_lo = sg * gs;
  if (g_lo >= nwg) return;                        // whole workgroup
  const int g_hi = min(nwg, g_lo + gs);
  const int u_lo = g_lo * kReadWaves, u_hi = g_hi * kReadWaves;
  const int t0 = unit_tile_lo(u_lo, ntiles, U), n = unit_tile_lo(u_hi, ntiles, U) - t0;
  const int pw = py * (kReadWaves * kTile * P) + wave * (kTile * P);
  // as many stages as fit: the deeper the ring, the more tiles are in flight
  constexpr int NS0 = kRmLds / ((WSL + SSL) * 16);
  constexpr int kRmStages = NS0 < kRmMaxStages ? NS0 : kRmMaxStages;
  __shared__ u32x4 lds[kRmStages * (WSL + SSL)];                // [stage][W tile | s]
  if (EE) {
    // early exit: nothing to do when every sequence of the workgroup's
    // positions is at its fixed point (the flag lives in the first ring
    // slot, which no load has touched yet)
    const int P0 = py * (kReadWaves * kTile * P);
    const int P1 = min(M, P0 + kReadWaves * kTile * P);
    const int b0 = P0 / B, nb = (P1 - 1) / B - b0 + 1;
    bool live = false;
    for (int i = threadIdx.x; i < nb; i += kReadWaves * kWave) live |= iters[b0 + i] == 0;
    uint32_t* flag = reinterpret_cast<uint32_t*>(&lds[0]);
    if (threadIdx.x == 0) *flag = 0u;
    __syncthreads();
    if (live) *flag = 1u;
    __syncthreads();
    const bool any = *flag != 0u;
    __syncthreads();
    if (!any) return;                             // whole workgroup
  }

  u32x4 zf[P][NU];
#pragma unroll
  for (int pb = 0; pb < P; ++pb) RT::load_z(Z, M, pw + kTile * pb, lane, zf[pb]);
  bool act[P], sample[P];
  float pit[P];                                   // sampled rows: softmax(l / T)
  bool any = false, live = false;
#pragma unroll
  for (int pb = 0; pb < P; ++pb) {
    const int p = pw + kTile * pb + (lane & 15);
    act[pb] = p < M;
    if (EE) live = live || (act[pb] && iters[(act[pb] ? p : M - 1) / B] == 0);
    sample[pb] = act[pb] && load_flag(temp, (act[pb] ? p : M - 1) / B, S) != 0;
    pit[pb] = invT[(act[pb] ? p : M - 1) / B];
    any = any || sample[pb];
  }
  const bool any_sample = __ballot(any) != 0;    // wave-uniform
  const bool wdead = EE && __ballot(live) == 0;   // wave-uniform
  // per position block, wave-uniform: does any lane take the greedy maximum,
  // any the softmax partials?  (With B a multiple of 16 a block lies in one
  // sequence and does only one of the two.)
  bool do_max[P], do_sum[P];
#pragma unroll
  for (int pb = 0; pb < P; ++pb) {
    do_max[pb] = __ballot(act[pb] && !sample[pb]) != 0;
    do_sum[pb] = __ballot(sample[pb]) != 0;
  }
  // greedy rows: running maximum and its row (rows arrive in increasing order
  // in every lane, so a strict comparison keeps the lowest index of a tie;
  // -0 == +0 as in the key order).  Other rows start at +inf, which no value
  // exceeds, so they keep the empty key without a mask in the loop.
  float bv[P];
  uint32_t bi[P];
  Stat st[P];
#pragma unroll
  for (int pb = 0; pb < P; ++pb) {
    bv[pb] = (act[pb] && !sample[pb]) ? -INFINITY : INFINITY;
    bi[pb] = 0xFFFFFFFFu;
    st[pb] = stat_empty();
  }
  // the key row of every read workgroup that ends at or before tile boundary
  // tend, from the running maxima, which then restart
  int gc = g_lo, ge = unit_tile_lo((g_lo + 1) * kReadWaves, ntiles, U);
  auto flush_keys = [&](int tend) {
    while (gc < g_hi && ge <= tend) {             // wave-uniform
#pragma unroll
      for (int pb = 0; pb < P; ++pb) {
        uint64_t best = bi[pb] == 0xFFFFFFFFu ? kKeyMin : argmax_key(bv[pb], bi[pb]);
#pragma unroll
        for (int m = 16; m < 64; m <<= 1) best = umax64(best, shfl_xor_u64(best, m));
        const int p = pw + kTile * pb + (lane & 15);
        if (lane < 16 && act[pb] && !wdead) keys[(size_t)gc * M + p] = best;
        bv[pb] = (act[pb] && !sample[pb]) ? -INFINITY : INFINITY;
        bi[pb] = 0xFFFFFFFFu;
      }
      ++gc;
      ge = unit_tile_lo((gc + 1) * kReadWaves, ntiles, U);
    }
  };

  // loads of tile j (clamped into the range, so that every wave issues the
  // same number of loads per tile) into stage j % kRmStages
  const int wrow = (kWave * wave + lane) >> 5;
  const int wchunk = ((kWave * wave + lane) & 31) ^ wrow;
  const int sq = lane >> 2, sc = (lane & 3) ^ ((sq >> 2) & 3);
  const float* sbase[P];
#pragma unroll
  for (int pb = 0; pb < P; ++pb) {
    const int p = pw + kTile * pb + sq;
    sbase[pb] = S + s_index(p < M ? p : M - 1, 4 * sc, Ms);
    if (wdead) sbase[pb] = S + 4 * (lane & 3);    // fixed, in cache after the first tile
  }
  auto issue = [&](int j) {
    const int t = t0 + (j < n ? j : n - 1);
    int row = t * kTile + wrow;
    row = row < V ? row : V - 1;
    u32x4* stage = lds + (j % kRmStages) * (WSL + SSL);
    lds_dma16(W + (size_t)row * 256 + 8 * wchunk, stage + kWave * wave);
#pragma unroll
    for (int pb = 0; pb < P; ++pb)
      lds_dma16_nt(sbase[pb] + (wdead ? (size_t)0 : (size_t)t * Ms * kTile),
                stage + WSL + kWave * (P * wave + pb));
  };
  // (max, sum) of every unit that ends at or before tile boundary tend
  int uc = u_lo, ue = unit_tile_lo(u_lo + 1, ntiles, U);
  auto flush_until = [&](int tend) {
    while (uc < u_hi && ue <= tend) {             // wave-uniform
      if (any_sample) {
#pragma unroll
        for (int pb = 0; pb < P; ++pb) {
          Stat q = st[pb];
#pragma unroll
          for (int m = 16; m < 64; m <<= 1) {
            const Stat o{__shfl_xor(q.m, m, kWave), __shfl_xor(q.s, m, kWave)};
            q = stat_merge(q, o);
          }
          const int p = pw + kTile * pb + (lane & 15);
          if (lane < 16 && sample[pb] && !wdead) stats[(size_t)p * U + uc] = q;
          st[pb] = stat_empty();
        }
      }
      ++uc;
      ue = unit_tile_lo(uc + 1, ntiles, U);
    }
  };

  flush_until(t0);                                // units without tiles
  flush_keys(t0);                                 // read workgroups without tiles
#pragma unroll
  for (int j = 0; j < kRmStages - 1; ++j) issue(j);
  constexpr int kPend = (kRmStages - 2) * (1 + P); // loads of the later tiles
  static_assert(kPend < 64, "vmcnt field");
  for (int j = 0; j < n; ++j) {
    // tile j's loads are done once only the later tiles' are outstanding;
    // the barrier then covers every wave's part of stage j, and every wave's
    // reads of the stage that the next issue overwrites (tile j - 1)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0x0070 | (kPend & 15) | ((kPend >> 4) << 14));
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    issue(j + kRmStages - 1);
    if (wdead) continue;                           // wave-uniform
    const u32x4* stage = lds + (j % kRmStages) * (WSL + SSL);
    u32x4 a[NU];
#pragma unroll
    for (int i = 0; i < NU; ++i) a[i] = stage[rm_wslot(lane & 15, (lane >> 4) + 4 * i)];
    floatx4 c[P];
#pragma unroll
    for (int pb = 0; pb < P; ++pb)
      c[pb] = __builtin_bit_cast(floatx4, stage[WSL + kWave * (P * wave + pb) +
                                               rm_sslot(lane & 15, lane >> 4)]);
    const int t = t0 + j;
    const int row0 = t * kTile + 4 * (lane >> 4);
    const bool last = (t + 1) * kTile > V;         // wave-uniform: rows past V in this tile
    // the P chains interleaved (each is RT::chain's sequence of operations)
    floatx4 accs[P];
#pragma unroll
    for (int pb = 0; pb < P; ++pb) accs[pb] = c[pb];
#pragma unroll
    for (int i = 0; i < NU; ++i)
#pragma unroll
      for (int pb = 0; pb < P; ++pb) accs[pb] = Mfma<uint16_t>::mma(a[i], zf[pb][i], accs[pb]);
    if (last) {                                    // wave-uniform
      // rows past V become -inf: no maximum takes them, no sum counts them
#pragma unroll
      for (int pb = 0; pb < P; ++pb)
#pragma unroll
        for (int i = 0; i < 4; ++i) accs[pb][i] = row0 + i < V ? accs[pb][i] : -INFINITY;
    }
#pragma unroll
    for (int pb = 0; pb < P; ++pb) {
      const floatx4 acc = accs[pb];
      if (do_max[pb]) {                            // wave-uniform
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool take = acc[i] > bv[pb];
          bv[pb] = take ? acc[i] : bv[pb];
          bi[pb] = take ? (uint32_t)(row0 + i) : bi[pb];
        }
      }
      if (do_sum[pb]) {                            // wave-uniform
        float x[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = sample[pb] ? acc[i] * pit[pb] : -INFINITY;
        st[pb] = stat_add4(st[pb], x[0], x[1], x[2], x[3]);
      }
      if (out_logits) {
        const int p = pw + kTile * pb + (lane & 15);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (act[pb] && row0 + i < V) out_logits[(size_t)p * V + row0 + i] = acc[i];
      }
    }
    flush_until(t + 1);
    flush_keys(t + 1);
  }
  __builtin_amdgcn_s_waitcnt(0x0070);             // the clamped loads past the end
}

hipError_t launch_read(xp_handle* h, int batch, int pass, uint32_t flags, const uint8_t* temp,
                       float* out_logits, hipStream_t st) {
  (void)pass;
  const int M = batch * h->B;
  dim3 grid(h->read_wgs, (M + kTile - 1) / kTile), block(kReadWaves * kWave);
  const int skip = (flags & XP_EARLY_EXIT) ? 1 : 0;
  if (h->dtype == XP_BF16 && M > kTile) {
    // 16 P positions per wave, P = 1..4 (P = 4 from 512 positions on)
    const int per = kReadWaves * kTile;
    int P = (M + per - 1) / per;
    P = P < kRmMaxP ? P : kRmMaxP;
    const int ny = (M + per * P - 1) / (per * P);
    // one workgroup per CU and position group at most: a workgroup takes gs
    // read workgroups in a row, so that the launch runs in one round
    const int gs = ny;
    const int nsg = (h->read_wgs + gs - 1) / gs;
    grid = dim3((nsg + 7) / 8 * 8 * ny);
    const uint16_t* Wr = (const uint16_t*)h->W_r;
    const uint16_t* Zb = (const uint16_t*)h->ws.z;
#define XP_RM(PP, EEV)                                                                       \
  hipLaunchKernelGGL((k_read_multi<PP, EEV>), grid, block, 0, st, Wr, Zb, h->ws.s, M, h->V, M, \
                     h->ntiles, h->read_units, h->ws.keys, h->ws.stats, temp, h->B, out_logits, \
                     h->ws.ctrl, skip, h->read_wgs, ny, gs, h->ws.invT, h->ws.iters)
    if (skip) {
      switch (P) {
        case 1: XP_RM(1, true); break;
        case 2: XP_RM(2, true); break;
        case 3: XP_RM(3, true); break;
        default: XP_RM(4, true);
      }
    } else {
      switch (P) {
        case 1: XP_RM(1, false); break;
        case 2: XP_RM(2, false); break;
        case 3: XP_RM(3, false); break;
        default: XP_RM(4, false);
      }
    }
#undef XP_RM
    return hipGetLastError();
  }
  if (h->dtype == XP_BF16)
    hipLaunchKernelGGL((k_read<uint16_t>), grid, block, 0, st, (const uint16_t*)h->W_r,
                       (const uint16_t*)h->ws.z, h->ws.s, M, h->V, M, h->ntiles,
                       h->read_units, h->ws.keys, h->ws.stats, temp, h->B, out_logits, h->ws.ctrl,
                       skip, h->ws.invT);
  else
    hipLaunchKernelGGL((k_read<float>), grid, block, 0, st, (const float*)h->W_r,
                       (const float*)h->ws.z, h->ws.s, M, h->V, M, h->ntiles, h->read_units,
                       h->ws.keys, h->ws.stats, temp, h->B, out_logits, h->ws.ctrl, skip,
                       h->ws.invT);
  return hipGetLastError();
}

}  // namespace xp
