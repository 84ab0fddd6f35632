// Token selection from the per-unit partials of a vocabulary stream, and the
// Jacobi bookkeeping of Algorithm 1 (fixed-point test, iteration count).
//
// Greedy rows: the maximum 64-bit key over the stream's workgroups gives
// argmax_v l_v with ties to the lowest index.
// Sampled rows at temperature T: with x_v = l_v / T (the fp32 product of l_v
// and the fp32 1/T, the same in every kernel), y = min{v : sum_{w<=v}
// e^{x_w - m} > u Z}, one workgroup per position (k_sample):
//   1. m = max over units; the unit masses sum_u e^{max_u - m} are summed in
//      fp64, each wave over a contiguous range of units (in-order wave
//      scans), then the wave totals in wave order: Z;
//   2. the first wave whose running total exceeds u Z redoes its scans (same
//      arithmetic) to find the crossing unit;
//   3. that unit's rows are recomputed with the stream's own MFMA tile code
//      (same fp32 logits) and scanned in vocabulary order in fp64.
// The log-sum-exp m + log Z of the x of the chosen pass is kept for
// verification.
#include "xp_internal.h"
#include "xp_tiles.h"

namespace xp {

__device__ __forceinline__ double wave_incl_scan(double x, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double y = __shfl_up(x, off, kWave);
    if (lane >= off) x += y;
  }
  return x;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) x = fmaxf(x, __shfl_xor(x, m, kWave));
  return x;
}

// Inverse-CDF selection of softmax(l / T), one workgroup per position (rows at
// temperature 0, and every row of a batch that is at its fixed point, return
// at once).  mode 0: the seed Y^(0) from the base logits (with caller seeds
// only the log-sum-exp is kept); mode 1: the selection of a Jacobi pass.  The
// chosen row goes to Ynew, where the selection kernel that follows picks it up.
// Every wave loads all of its unit partials at once, and the crossing unit's
// logits are recomputed by one wave per tile into LDS before one wave scans
// them, so a selection costs a few memory round trips.
// CH is the number of 64-unit chunks a wave holds, ceil(U / 512): the
// partition's size, not the largest one supported, so no fp64 exponential or
// scan runs on masked lanes and the registers allow more workgroups per CU.
constexpr int kSmpWaves = 8;
constexpr int kSmpChunks = 4096 / (kSmpWaves * 64);   // 64-unit chunks per wave at most: 4096 units
constexpr int kSmpRows = 128;        // rows of the largest unit (8 tiles)

template <typename T, int CH>
__global__ __launch_bounds__(kSmpWaves * kWave) void k_sample(
    int mode, int B, int V, int M, const float* __restrict__ S, int Ms,
    const T* __restrict__ W_r, const T* __restrict__ Z, const Stat* __restrict__ stats,
    int ntiles, int U, const int32_t* __restrict__ seed_ids, const uint8_t* __restrict__ temp,
    const float* __restrict__ u_draft, int32_t* __restrict__ Ynew, double* __restrict__ lse,
    const int32_t* __restrict__ iters, int early_exit, const float* __restrict__ invT) {
  const int p = blockIdx.x;
  if (temp[p / B] == 0) return;
  const float it = invT[p / B];                   // the unit partials hold l / T
  if (mode == 1 && early_exit && iters[p / B] != 0) return;   // the sequence keeps Y^(j)
  const bool pick = !(mode == 0 && seed_ids != nullptr);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __shared__ float wmax[kSmpWaves];
  __shared__ double wtot[kSmpWaves];
  __shared__ int s_ustar;
  __shared__ double s_pre;
  __shared__ float lrow[kSmpRows];

  // wave w owns the units [ua, ub) (in order), all loaded at once
  const int ua = (int)((int64_t)U * wave / kSmpWaves), ub = (int)((int64_t)U * (wave + 1) / kSmpWaves);
  Stat q[CH];
#pragma unroll
  for (int j = 0; j < CH; ++j) {
    const int i = ua + 64 * j + lane;
    q[j] = stats[(size_t)p * U + (i < ub ? i : (ub > 0 ? ub - 1 : 0))];
    if (i >= ub) q[j] = stat_empty();
  }
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < CH; ++j)
    if (q[j].s > 0.f) m = fmaxf(m, q[j].m);
  m = wave_max(m);
  if (lane == 0) wmax[wave] = m;
  __syncthreads();
  m = wmax[0];
#pragma unroll
  for (int w = 1; w < kSmpWaves; ++w) m = fmaxf(m, wmax[w]);

  // unit masses sum_u e^{max_u - m} in fp64; in-order wave scans per chunk
  double incl[CH], carry_before[CH];
  double carry = 0.0;
#pragma unroll
  for (int j = 0; j < CH; ++j) {
    const double w = q[j].s > 0.f ? (double)q[j].s * exp((double)q[j].m - (double)m) : 0.0;
    incl[j] = wave_incl_scan(w, lane);
    carry_before[j] = carry;
    if (ua + 64 * j < ub) carry += __shfl(incl[j], 63, kWave);
  }
  if (lane == 0) wtot[wave] = carry;
  __syncthreads();
  double Zs = 0.0, start = 0.0;
#pragma unroll
  for (int w = 0; w < kSmpWaves; ++w) {
    if (w == wave) start = Zs;
    Zs += wtot[w];
  }
  if (threadIdx.x == 0) lse[p] = (double)m + log(Zs);
  if (!pick) return;
  const double target = (double)u_draft[p] * Zs;
  // the first wave whose running total exceeds the target (the last wave
  // with units when rounding leaves none)
  int wstar = kSmpWaves - 1;
  while (wstar > 0 && (int64_t)U * wstar / kSmpWaves >= (int64_t)U * (wstar + 1) / kSmpWaves) --wstar;
  {
    double run = 0.0;
#pragma unroll
    for (int w = 0; w < kSmpWaves; ++w) {
      if (run + wtot[w] > target) {
        wstar = w;
        break;
      }
      run += wtot[w];
    }
  }
  if (wave == wstar) {
    // the crossing unit within this wave's range, from the same scans; when
    // rounding leaves none, the wave's last unit is rescanned from the wave's
    // total and yields its last row of nonzero mass
    int ustar = ub - 1;
    double pre = start + carry;
    bool found = false;
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      const int base = ua + 64 * j;
      const double tot = start + (carry_before[j] + incl[j]);
      const unsigned long long hit = __ballot(!found && base + lane < ub && tot > target);
      if (hit) {
        const int first = __ffsll((long long)hit) - 1;
        const double prev = __shfl_up(tot, 1, kWave);
        const double excl = lane == 0 ? start + carry_before[j] : prev;
        ustar = base + first;
        pre = __shfl(excl, first, kWave);
        found = true;
      }
    }
    if (lane == 0) {
      s_ustar = ustar;
      s_pre = pre;
    }
  }
  __syncthreads();
  const int ustar = s_ustar;
  const int tlo = unit_tile_lo(ustar, ntiles, U), thi = unit_tile_lo(ustar + 1, ntiles, U);
  const int rlo = tlo * kTile, rhi = min(V, thi * kTile);
  // logits of the unit's rows: mode 1 recomputes l = s + W_r z with the
  // stream's tile code, one wave per tile (a unit of a Read partition has at
  // most kSmpRows / 16 tiles); mode 0 reads s while scanning
  for (int tw = wave; mode == 1 && tw < thi - tlo; tw += kSmpWaves) {   // wave-uniform
    constexpr int NU = ReadTile<T>::NU;
    u32x4 bf[NU], a[NU];
    const int t = tlo + tw;
    ReadTile<T>::load_z(Z, M, p & ~15, lane, bf);
    ReadTile<T>::load_w(W_r, V, t, lane, a);
    const int pl = (p & ~15) + (lane & 15);
    const floatx4 acc = ReadTile<T>::chain(a, bf, ReadTile<T>::load_s(S, Ms, pl, pl < M, t, lane));
    if ((lane & 15) == (p & 15)) {
#pragma unroll
      for (int i = 0; i < 4; ++i) lrow[kTile * tw + 4 * (lane >> 4) + i] = acc[i];
    }
  }
  __syncthreads();
  if (wave != 0) return;
  // scan the rows in vocabulary order from the mass of the units before
  int chosen = -1, last_pos = -1;
  double cum = s_pre;
  for (int base = rlo; base < rhi; base += 64) {
    const int row = base + lane;
    const float l = row < rhi ? (mode == 0 ? S[s_index(p, row, Ms)] : lrow[row - rlo]) * it : 0.f;
    const double w = (row < rhi) ? exp((double)l - (double)m) : 0.0;
    const double tot = cum + wave_incl_scan(w, lane);
    const unsigned long long hit = __ballot(row < rhi && tot > target);
    const unsigned long long nz = __ballot(row < rhi && w > 0.0);
    if (nz) last_pos = base + 63 - __clzll((long long)nz);
    if (hit) {
      chosen = base + __ffsll((long long)hit) - 1;
      break;
    }
    cum = __shfl(tot, 63, kWave);
  }
  if (chosen < 0) chosen = last_pos >= 0 ? last_pos : rlo;   // rounding left no crossing
  if (lane == 0) Ynew[p] = chosen;
}

// One workgroup per sequence.  mode 0: seed Y^(0) from the base logits (or the
// caller's seed ids); mode 1: the selection of Jacobi pass `pass`.  Greedy
// rows take the maximum 64-bit key of every position over the nkeys unit
// rows: thread t takes position t % PP (PP = 16 or 32 >= B) of rows t / PP,
// t / PP + NRG, ..., so that one load instruction reads whole runs of
// consecutive positions of a key row (keys are [row][M]); every load of a
// thread is issued before its first compare, then lanes and waves holding
// the same position combine their maxima.  So a greedy selection costs one
// memory round trip with coalesced loads.
constexpr int kSelWaves = 8;

template <typename T>
__global__ __launch_bounds__(kSelWaves * kWave) void k_select(
    int mode, int pass, int batch, int B, int V, int M, const float* __restrict__ S, int Ms,
    const T* __restrict__ W_r, const T* __restrict__ Z, const uint64_t* __restrict__ keys,
    int nkeys, const Stat* __restrict__ stats, int ntiles, int U,
    const int32_t* __restrict__ seed_ids, const uint8_t* __restrict__ temp,
    const float* __restrict__ u_draft, const int32_t* __restrict__ Yprev, int32_t* __restrict__ Ynew,
    int32_t* __restrict__ traj, double* __restrict__ lse, int32_t* __restrict__ iters,
    int32_t* __restrict__ ctrl, uint32_t* __restrict__ err, int early_exit,
    int32_t* __restrict__ out_ids, int32_t* __restrict__ out_iters, int K) {
  constexpr int NT = kSelWaves * kWave, kRowsPerRound = 16;
  const int b = blockIdx.x, t = threadIdx.x;
  __shared__ int changed;
  __shared__ uint64_t sbest[kSelWaves][32];
  const bool skip = mode == 1 && early_exit && iters[b] != 0;   // at its fixed point
  if (skip) {                                     // the block carries over
    for (int k = t; k < B; k += NT) {
      const int p = b * B + k;
      const int y = Yprev[p];
      Ynew[p] = y;
      if (traj) traj[p] = y;
      if (out_ids) out_ids[p] = y;
    }
    if (t == 0 && out_iters) out_iters[b] = iters[b];
    return;
  }
  const int it0 = iters[b];
  const bool sample = temp != nullptr && temp[b] != 0;
  const bool seeded = mode == 0 && seed_ids != nullptr;
  if (t == 0) changed = 0;
  if (!sample && !seeded) {                       // workgroup-uniform
    const int PP = B <= 16 ? 16 : 32, NRG = NT / PP;
    const int pos = t % PP, rg = t / PP;
    const size_t col = (size_t)b * B + (pos < B ? pos : B - 1);
    uint64_t best = 0;
    for (int r0 = rg; r0 < nkeys; r0 += kRowsPerRound * NRG) {
      uint64_t kv[kRowsPerRound];
#pragma unroll
      for (int j = 0; j < kRowsPerRound; ++j) {
        const int r = r0 + j * NRG;               // rows past nkeys repeat the last
        kv[j] = keys[(size_t)(r < nkeys ? r : nkeys - 1) * M + col];
      }
#pragma unroll
      for (int j = 0; j < kRowsPerRound; ++j) best = umax64(best, kv[j]);
    }
    for (int o = PP; o < kWave; o <<= 1) best = umax64(best, shfl_xor_u64(best, o));
    if ((t & (kWave - 1)) < PP) sbest[t / kWave][pos] = best;
  }
  __syncthreads();
  if (t < B) {
    const int p = b * B + t;
    int y;
    if (seeded) {
      y = seed_ids[p];
      if (y < 0 || y >= V) {
        atomicOr(err, XP_DEVERR_TOKEN);
        y = 0;
      }
    } else if (!sample) {
      uint64_t bb = sbest[0][t];
#pragma unroll
      for (int w = 1; w < kSelWaves; ++w) bb = umax64(bb, sbest[w][t]);
      y = (int)key_index(bb);
    } else {
      y = Ynew[p];                                // chosen by k_sample
    }
    Ynew[p] = y;
    if (traj) traj[p] = y;
    if (out_ids) out_ids[p] = y;
    if (mode == 1 && y != Yprev[p]) atomicOr(&changed, 1);
  }
  __syncthreads();
  if (t == 0) {
    int it = it0;
    if (mode == 1 && changed == 0 && it == 0) {
      it = pass + 1;
      iters[b] = it;
      if (atomicAdd(&ctrl[0], 1) + 1 == batch) ctrl[1] = 1;
    }
    if (out_iters) out_iters[b] = mode == 0 ? 0 : (it ? it : K);
  }
}

__global__ void k_copy_logits(int M, int V, const float* __restrict__ S,
                              float* __restrict__ out) {
  const size_t n = (size_t)M * V;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x) {
    const size_t p = i / V, v = i % V;
    out[i] = S[s_index((int)p, (int)v, M)];
  }
}

// ---------------------------------------------------------------------------
hipError_t launch_select(xp_handle* h, int batch, int pass, int K, uint32_t flags,
                         const int32_t* seed_ids, const uint8_t* temp, const float* u_draft,
                         int32_t* out_traj, int32_t* out_ids, int32_t* out_iters,
                         hipStream_t st, bool filtering) {
  const int M = batch * h->B;
  const int mode = pass < 0 ? 0 : 1;
  int32_t* Yprev = h->ws.Y[(pass + 2) % 2];      // pass j reads Y[j % 2]
  int32_t* Ynew = h->ws.Y[(pass + 1) % 2];       // and writes Y[(j+1) % 2]
  int32_t* traj = out_traj ? out_traj + (size_t)(pass + 1) * M : nullptr;
  const int nkeys = mode == 0 ? h->lm_units_cur : h->read_wgs;
  const int U = mode == 0 ? h->lm_units_cur : h->read_units;
  const int early = (flags & XP_EARLY_EXIT) ? 1 : 0;
  if (temp) {
    // rows that truncate are sampled by k_fsample; k_sample takes the others
    const uint8_t* tsmp = filtering ? h->ws.temp_nf : temp;
    if (filtering) {
      const hipError_t e = launch_fsample(h, batch, pass, flags, seed_ids, u_draft, st);
      if (e != hipSuccess) return e;
    }
    // 64-unit chunks per wave (xp_create keeps U within kSmpWaves * 64 * kSmpChunks)
    const int ch = (U + kSmpWaves * kWave - 1) / (kSmpWaves * kWave);
#define XP_SMP(TT, CC)                                                                        \
  hipLaunchKernelGGL((k_sample<TT, CC>), dim3(M), dim3(kSmpWaves * kWave), 0, st, mode, h->B,  \
                     h->V, M, h->ws.s, M, (const TT*)h->W_r, (const TT*)h->ws.z, h->ws.stats,  \
                     h->ntiles, U, mode == 0 ? seed_ids : nullptr, tsmp, u_draft, Ynew,        \
                     h->ws.lse, h->ws.iters, early, h->ws.invT)
#define XP_SMP_CH(TT)                                                                         \
  switch (ch) {                                                                               \
    case 1: XP_SMP(TT, 1); break;                                                             \
    case 2: XP_SMP(TT, 2); break;                                                             \
    case 3: XP_SMP(TT, 3); break;                                                             \
    case 4: XP_SMP(TT, 4); break;                                                             \
    case 5: XP_SMP(TT, 5); break;                                                             \
    case 6: XP_SMP(TT, 6); break;                                                             \
    case 7: XP_SMP(TT, 7); break;                                                             \
    case 8: XP_SMP(TT, 8); break;                                                             \
    default:                                                                                  \
      if (ch <= 12) XP_SMP(TT, (kSmpChunks < 12 ? kSmpChunks : 12));                          \
      else XP_SMP(TT, kSmpChunks);                                                            \
  }
    if (h->dtype == XP_BF16) {
      XP_SMP_CH(uint16_t)
    } else {
      XP_SMP_CH(float)
    }
#undef XP_SMP_CH
#undef XP_SMP
  }
  if (h->dtype == XP_BF16)
    hipLaunchKernelGGL((k_select<uint16_t>), dim3(batch), dim3(kSelWaves * kWave), 0, st, mode, pass, batch,
                       h->B, h->V, M, h->ws.s, M, (const uint16_t*)h->W_r,
                       (const uint16_t*)h->ws.z, h->ws.keys, nkeys, h->ws.stats, h->ntiles, U,
                       mode == 0 ? seed_ids : nullptr, temp, u_draft, Yprev, Ynew, traj,
                       h->ws.lse, h->ws.iters, h->ws.ctrl, h->ws.err, early, out_ids, out_iters,
                       K);
  else
    hipLaunchKernelGGL((k_select<float>), dim3(batch), dim3(kSelWaves * kWave), 0, st, mode, pass, batch, h->B,
                       h->V, M, h->ws.s, M, (const float*)h->W_r, (const float*)h->ws.z,
                       h->ws.keys, nkeys, h->ws.stats, h->ntiles, U,
                       mode == 0 ? seed_ids : nullptr, temp, u_draft, Yprev, Ynew, traj,
                       h->ws.lse, h->ws.iters, h->ws.ctrl, h->ws.err, early, out_ids, out_iters,
                       K);
  return hipGetLastError();
}

hipError_t launch_finish(xp_handle* h, int batch, int K, uint32_t flags, int32_t* out_ids,
                         int32_t* out_iters, float* out_logits, hipStream_t st, bool filtering) {
  (void)out_ids;
  (void)out_iters;
  const int M = batch * h->B;
  if (K == 0 && (flags & XP_WRITE_LOGITS) && out_logits)
    hipLaunchKernelGGL(k_copy_logits, dim3(1024), dim3(256), 0, st, M, h->V, h->ws.s,
                       out_logits);
  // with truncation every pass writes its logits to the workspace row buffer
  // (the last executed pass's stay there): copy them out
  if (K > 0 && filtering && (flags & XP_WRITE_LOGITS) && out_logits)
    return hipMemcpyAsync(out_logits, h->ws.lf, (size_t)M * h->V * sizeof(float),
                          hipMemcpyDeviceToDevice, st);
  return hipGetLastError();
}

}  // namespace xp
