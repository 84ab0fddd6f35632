// Block verification (section 3.1).
//
// Greedy rows: n = longest prefix with y_i = t_i, next = t_{n+1}.
// Sampled rows at temperature T (that of the refine), speculative accept /
// reject:
//   accept y_k iff r_k q_k(y_k) <= p_k(y_k), q_k = softmax(l_k / T) of the
//   refine's last pass, p_k = softmax(target logits after the prefix y_{<k},
//   over T); every l / T is the fp32 product of l and the fp32 1/T, as in the
//   refine's kernels;
//   at the first rejection next ~ max(0, p_k - q_k) (p_k if that has no mass),
//   if all B are accepted next ~ p_{B+1}; both by inverse CDF at u_res.
// Kernels: target log-sum-exp per row -> accept scan -> residual mass per
// vocabulary unit (one W_r stream for all sequences) -> crossing unit + rescan.
#include "xp_internal.h"
#include "xp_tiles.h"

namespace xp {

// lseT[b][k] = log sum_v exp(t[b][k][v] / T) for sampled rows, k = 0..B (t
// the target logits), in two steps: every workgroup reduces one chunk of
// kVChunk entries of a row to (max, sum of exp(x - max)), the exponentials in
// fp32 and the sums in fp64;
// then one wave per row merges the chunks in a fixed order.
// Rows k0 + blockIdx.y only; with `more` given, only of sequences whose
// accept scan went past the first round's rows (vpos == kVMore).
__global__ __launch_bounds__(256) void k_vtarget_part(const float* __restrict__ tl, int B, int V,
                                                      const uint8_t* __restrict__ temp,
                                                      const float* __restrict__ invT,
                                                      double* __restrict__ part, int k0,
                                                      const int32_t* __restrict__ more) {
  constexpr int PER = kVChunk / 256;
  const int c = blockIdx.x, k = k0 + blockIdx.y, b = blockIdx.z, nc = gridDim.x;
  if (temp[b] == 0 || (more != nullptr && more[b] != kVMore)) return;
  const float it = invT[b];
  const float* row = tl + ((size_t)b * (B + 1) + k) * V;
  float x[PER];
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int v = c * kVChunk + i * 256 + threadIdx.x;
    x[i] = v < V ? row[v] * it : -INFINITY;
    m = fmaxf(m, x[i]);
  }
  __shared__ float sm[4];
  __shared__ double sd[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, kWave));
  if (lane == 0) sm[wave] = m;
  __syncthreads();
  m = fmaxf(fmaxf(sm[0], sm[1]), fmaxf(sm[2], sm[3]));
  double acc = 0.0;
#pragma unroll
  for (int i = 0; i < PER; ++i) acc += x[i] == -INFINITY ? 0.0 : (double)expf(x[i] - m);
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) acc += __shfl_xor(acc, o, kWave);
  if (lane == 0) sd[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double* q = part + (((size_t)b * (B + 1) + k) * nc + c) * 2;
    q[0] = (double)m;
    q[1] = (sd[0] + sd[1]) + (sd[2] + sd[3]);
  }
}

__global__ __launch_bounds__(64) void k_vtarget_comb(int B, int nc, const uint8_t* __restrict__ temp,
                                                     const double* __restrict__ part,
                                                     double* __restrict__ lseT, int k0,
                                                     const int32_t* __restrict__ more) {
  const int b = blockIdx.y, i = b * (B + 1) + k0 + blockIdx.x, lane = threadIdx.x;   // one wave per row
  if (temp[b] == 0 || (more != nullptr && more[b] != kVMore)) return;
  const double* q = part + (size_t)i * nc * 2;
  double m = -INFINITY;
  for (int c = lane; c < nc; c += kWave) m = fmax(m, q[2 * c]);
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) m = fmax(m, __shfl_xor(m, o, kWave));
  double sum = 0.0;
  for (int c = lane; c < nc; c += kWave) sum += q[2 * c + 1] > 0.0 ? q[2 * c + 1] * exp(q[2 * c] - m) : 0.0;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) sum += __shfl_xor(sum, o, kWave);
  if (lane == 0) lseT[i] = m + log(sum);
}

// l = s (+ W_r z) for position p at vocabulary row v, through the Read tile of
// the stream (all 64 lanes take part; every lane gets the value).
template <typename T>
__device__ float refined_logit(int with_read, const float* __restrict__ S, int Ms,
                               const T* __restrict__ W_r, const T* __restrict__ Z, int M, int V,
                               int p, int v) {
  const int lane = threadIdx.x & 63;
  float d = 0.f;
  if (with_read) {
    constexpr int NU = ReadTile<T>::NU;
    u32x4 bf[NU], a[NU];
    const int pl = (p & ~15) + (lane & 15);
    ReadTile<T>::load_z(Z, M, p & ~15, lane, bf);
    ReadTile<T>::load_w(W_r, V, v / 16, lane, a);
    const floatx4 acc =
        ReadTile<T>::chain(a, bf, ReadTile<T>::load_s(S, Ms, pl, pl < M, v / 16, lane));
    const int rr = v & 15, src = (rr >> 2) * 16 + (p & 15);
    const float c0 = __shfl(acc[0], src, kWave), c1 = __shfl(acc[1], src, kWave);
    const float c2 = __shfl(acc[2], src, kWave), c3 = __shfl(acc[3], src, kWave);
    const int comp = rr & 3;
    d = comp == 0 ? c0 : comp == 1 ? c1 : comp == 2 ? c2 : c3;
  }
  return with_read ? d : S[s_index(p, v, Ms)];
}

// One wave per sequence: accept scan over draft positions [kb, min(ke, B)),
// the target rows [kb, ke) having their log-sum-exp.  vpos[b] = rejected
// position, or B once all are accepted (which needs row B, ke = B + 1);
// kVMore when the scan got through without row B (the next round goes on).  kb > 0 continues only such sequences.  Rows
// marked in `skip` (truncated sampling: k_vfaccept) are left alone.
template <typename T>
__global__ __launch_bounds__(64) void k_vaccept(
    int B, int V, int M, int with_read, const int32_t* __restrict__ draft,
    const uint8_t* __restrict__ temp, const uint8_t* __restrict__ skip,
    const int32_t* __restrict__ tids,
    const float* __restrict__ tl, const float* __restrict__ racc, const float* __restrict__ S,
    int Ms, const T* __restrict__ W_r, const T* __restrict__ Z, const double* __restrict__ lse,
    const double* __restrict__ lseT, int32_t* __restrict__ vpos, int32_t* __restrict__ out_n,
    int32_t* __restrict__ out_next, uint32_t* __restrict__ err, const float* __restrict__ invT,
    int kb, int ke) {
  const int b = blockIdx.x, lane = threadIdx.x;
  if (skip != nullptr && skip[b] != 0) return;
  if (kb > 0 && vpos[b] != kVMore) return;        // decided in the first round
  const bool sample = temp != nullptr && temp[b] != 0;
  int bad = 0;
  if (!sample) {
    if (lane == 0) {
      int n = 0;
      while (n < B) {
        int t = tids[(size_t)b * (B + 1) + n];
        if (t < 0 || t >= V) bad = 1;
        if (draft[b * B + n] != t) break;
        ++n;
      }
      int nx = tids[(size_t)b * (B + 1) + n];
      if (nx < 0 || nx >= V) {
        bad = 1;
        nx = 0;
      }
      out_n[b] = n;
      out_next[b] = nx;
      vpos[b] = -1;
      if (bad) atomicOr(err, XP_DEVERR_TOKEN);
    }
    return;
  }
  const float it = invT[b];
  // rows [kb, ke) have their log-sum-exp: positions up to min(ke, B) can be
  // tested, and "all accepted" can be decided only with the bonus row B too
  const int kend = ke < B ? ke : B;
  int n = ke >= B + 1 ? B : kVMore;
  for (int k = kb; k < kend; ++k) {
    const int p = b * B + k;
    int y = draft[p];
    if (y < 0 || y >= V) {
      bad = 1;
      y = 0;
    }
    const float l = refined_logit<T>(with_read, S, Ms, W_r, Z, M, V, p, y);
    const double q = exp((double)(l * it) - lse[p]);
    const double pt =
        exp((double)(tl[((size_t)b * (B + 1) + k) * V + y] * it) - lseT[(size_t)b * (B + 1) + k]);
    if (!((double)racc[p] * q <= pt)) {
      n = k;
      break;
    }
  }
  if (lane == 0) {
    if (n != kVMore) out_n[b] = n;
    vpos[b] = n;
    if (bad) atomicOr(err, XP_DEVERR_TOKEN);
  }
}

// Resampling weight of vocabulary row v for sequence b: the residual
// max(0, p - q) at the rejected position, or p_{B+1} for the bonus token.
__device__ __forceinline__ void resample_weights(float tlv, double lseTk, bool resid, float l,
                                                 double lsep, double* res, double* pw) {
  const double pv = exp((double)tlv - lseTk);
  *pw = pv;
  if (resid) {
    const double qv = exp((double)l - lsep);
    *res = pv > qv ? pv - qv : 0.0;
  } else {
    *res = pv;
  }
}

// Residual (and plain p) mass per vocabulary unit, one W_r stream for up to
// 16 sequences per workgroup column; lanes of greedy sequences idle.
template <typename T>
__global__ __launch_bounds__(1024) void k_vresid(
    int batch, int B, int V, int M, int with_read, int ntiles, int U,
    const uint8_t* __restrict__ temp, const int32_t* __restrict__ vpos,
    const float* __restrict__ tl, const float* __restrict__ S, int Ms, const T* __restrict__ W_r,
    const T* __restrict__ Z, const double* __restrict__ lse, const double* __restrict__ lseT,
    double* __restrict__ vmass, const float* __restrict__ invT) {
  constexpr int NU = ReadTile<T>::NU;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, NW = blockDim.x >> 6;
  const int u = blockIdx.x * NW + wave;
  const int b = blockIdx.y * 16 + (lane & 15);
  const bool act = b < batch && temp != nullptr && temp[b] != 0;
  const float it = invT[act ? b : 0];
  const int k = act ? vpos[b] : 0;
  const bool resid = act && k < B;
  const int p = b * B + (k < B ? k : 0);
  const int tlo = unit_tile_lo(u, ntiles, U), thi = unit_tile_lo(u + 1, ntiles, U);
  u32x4 bf[NU], a[NU];
  ReadTile<T>::load_z_row(Z, resid ? p : -1, lane, bf);
  const float* trow = tl + ((size_t)(act ? b : 0) * (B + 1) + k) * V;
  const double lk = act ? lseT[(size_t)b * (B + 1) + k] : 0.0;
  const double lp = resid ? lse[p] : 0.0;
  double mr = 0.0, mp = 0.0;
  for (int t = tlo; t < thi; ++t) {
    floatx4 acc = ReadTile<T>::load_s(S, Ms, p, resid, t, lane);
    if (with_read) {
      ReadTile<T>::load_w(W_r, V, t, lane, a);
      acc = ReadTile<T>::chain(a, bf, acc);
    }
    if (act) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = t * kTile + 4 * (lane >> 4) + i;
        if (row < V) {
          const float l = resid ? acc[i] : 0.f;
          double res, pw;
          resample_weights(trow[row] * it, lk, resid, l * it, lp, &res, &pw);
          mr += res;
          mp += pw;
        }
      }
    }
  }
#pragma unroll
  for (int m = 16; m < 64; m <<= 1) {
    mr += __shfl_xor(mr, m, kWave);
    mp += __shfl_xor(mp, m, kWave);
  }
  if (lane < 16 && act) {
    vmass[((size_t)u * batch + b) * 2 + 0] = mr;
    vmass[((size_t)u * batch + b) * 2 + 1] = mp;
  }
}

__device__ __forceinline__ double wave_scan_d(double x, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double y = __shfl_up(x, off, kWave);
    if (lane >= off) x += y;
  }
  return x;
}

// One workgroup of 8 waves per sampled sequence: each wave sums the unit
// masses of a contiguous range of units (in-order fp64 wave scans), the wave
// totals are added in wave order; the first wave whose running total passes
// u Z redoes its scans (same arithmetic) to find the crossing unit and
// rescans that unit's rows in vocabulary order.
constexpr int kVfWaves = 8;

template <typename T>
__global__ __launch_bounds__(kVfWaves * kWave) void k_vfinal(
    int batch, int B, int V, int M, int with_read, int ntiles, int U,
    const uint8_t* __restrict__ temp, const int32_t* __restrict__ vpos,
    const float* __restrict__ tl, const float* __restrict__ S, int Ms, const T* __restrict__ W_r,
    const T* __restrict__ Z, const double* __restrict__ lse, const double* __restrict__ lseT,
    const double* __restrict__ vmass, const float* __restrict__ u_res,
    int32_t* __restrict__ out_next, const float* __restrict__ invT) {
  const int b = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (temp == nullptr || temp[b] == 0) return;
  const float it = invT[b];
  __shared__ double wt[2][kVfWaves];
  const int k = vpos[b];
  bool resid = k < B;
  const int p = b * B + (k < B ? k : 0);
  const int ua = (int)((int64_t)U * wave / kVfWaves), ub = (int)((int64_t)U * (wave + 1) / kVfWaves);
  auto mass = [&](int i, int comp) {
    return i < ub ? vmass[((size_t)i * batch + b) * 2 + comp] : 0.0;
  };
  // per-wave totals of both components (residual, plain p)
#pragma unroll
  for (int comp = 0; comp < 2; ++comp) {
    double c = 0.0;
    for (int base = ua; base < ub; base += 64) c += __shfl(wave_scan_d(mass(base + lane, comp), lane), 63, kWave);
    if (lane == 0) wt[comp][wave] = c;
  }
  __syncthreads();
  // residual with no mass falls back to p (component 1)
  double tot0 = 0.0;
#pragma unroll
  for (int w = 0; w < kVfWaves; ++w) tot0 += wt[0][w];
  const int comp = tot0 > 0.0 ? 0 : 1;
  const bool use_resid = resid && comp == 0;
  double Zs = 0.0, start = 0.0;
#pragma unroll
  for (int w = 0; w < kVfWaves; ++w) {
    if (w == wave) start = Zs;
    Zs += wt[comp][w];
  }
  const double target = (double)u_res[b] * Zs;
  int wstar = kVfWaves - 1;
  while (wstar > 0 && (int64_t)U * wstar / kVfWaves >= (int64_t)U * (wstar + 1) / kVfWaves) --wstar;
  {
    double run = 0.0;
#pragma unroll
    for (int w = 0; w < kVfWaves; ++w) {
      if (run + wt[comp][w] > target) {
        wstar = w;
        break;
      }
      run += wt[comp][w];
    }
  }
  if (wave != wstar) return;
  int ustar = ub - 1;
  double carry = 0.0, pre = start;
  for (int base = ua; base < ub; base += 64) {
    const double incl = wave_scan_d(mass(base + lane, comp), lane);
    const double tot = start + (carry + incl);
    const unsigned long long hit = __ballot(base + lane < ub && tot > target);
    if (hit) {
      const int first = __ffsll((long long)hit) - 1;
      const double prev = __shfl_up(tot, 1, kWave);
      const double excl = lane == 0 ? start + carry : prev;
      ustar = base + first;
      pre = __shfl(excl, first, kWave);
      break;
    }
    carry += __shfl(incl, 63, kWave);
    pre = start + carry;
  }
  const int tlo = unit_tile_lo(ustar, ntiles, U), thi = unit_tile_lo(ustar + 1, ntiles, U);
  const int rlo = tlo * kTile, rhi = min(V, thi * kTile);
  const float* trow = tl + ((size_t)b * (B + 1) + k) * V;
  const double lk = lseT[(size_t)b * (B + 1) + k];
  const double lp = resid ? lse[p] : 0.0;
  int chosen = -1, last_pos = -1;
  double cum = pre;
  for (int base = rlo; base < rhi; base += 64) {
    const int row = base + lane;
    float mine = 0.f;
    if (resid && with_read) {
      constexpr int NU = ReadTile<T>::NU;
      u32x4 bf[NU], a[NU];
      ReadTile<T>::load_z_row(Z, p, lane, bf);
      const int rr = lane & 15, src = (rr >> 2) * 16, cp = rr & 3;
      for (int tt = 0; tt < 4; ++tt) {
        const int t = (base - rlo) / kTile + tlo + tt;
        if (t >= thi) break;
        ReadTile<T>::load_w(W_r, V, t, lane, a);
        const floatx4 acc = ReadTile<T>::chain(a, bf, ReadTile<T>::load_s(S, Ms, p, true, t, lane));
        const float c0 = __shfl(acc[0], src, kWave), c1 = __shfl(acc[1], src, kWave);
        const float c2 = __shfl(acc[2], src, kWave), c3 = __shfl(acc[3], src, kWave);
        const float v = cp == 0 ? c0 : cp == 1 ? c1 : cp == 2 ? c2 : c3;
        if ((lane >> 4) == tt) mine = v;
      }
    }
    if (resid && !with_read && row < rhi) mine = S[s_index(p, row, Ms)];   // K = 0: l = s
    double w = 0.0;
    if (row < rhi) {
      const float l = resid ? mine : 0.f;
      double res, pw;
      resample_weights(trow[row] * it, lk, resid, l * it, lp, &res, &pw);
      w = use_resid ? res : pw;
    }
    const double tot = cum + wave_scan_d(w, lane);
    const unsigned long long hit = __ballot(row < rhi && tot > target);
    const unsigned long long nz = __ballot(row < rhi && w > 0.0);
    if (nz) last_pos = base + 63 - __clzll((long long)nz);
    if (hit) {
      chosen = base + __ffsll((long long)hit) - 1;
      break;
    }
    cum = __shfl(tot, 63, kWave);
  }
  if (chosen < 0) chosen = last_pos >= 0 ? last_pos : rlo;
  if (lane == 0) out_next[b] = chosen;
}

// ---------------------------------------------------------------------------
template <typename T>
static hipError_t verify_t(xp_handle* h, int batch, const int32_t* draft, const uint8_t* temp,
                           const int32_t* tids, const float* tl, const float* racc,
                           const float* ures, int32_t* out_n, int32_t* out_next, hipStream_t st) {
  const int M = batch * h->B;
  const int with_read = h->state_k0 ? 0 : 1;
  // truncated rows are verified by launch_vfilter; these kernels take the others
  const bool filtering = temp != nullptr && h->state_filtered;
  const uint8_t* skip = filtering ? h->ws.filt : nullptr;
  if (filtering) temp = h->ws.temp_nf;
  // Round 1: the target rows [0, r1) of every sampled sequence and the accept
  // scan over them; most sequences reject there.  Round 2: rows [r1, B] of
  // the sequences that accepted all of the first r1 drafts.
  const int nc = (h->V + kVChunk - 1) / kVChunk;
  const int r1 = h->B + 1 < kVRows1 ? h->B + 1 : kVRows1;
  if (temp) {
    hipLaunchKernelGGL(k_vtarget_part, dim3(nc, r1, batch), dim3(256), 0, st, tl, h->B, h->V,
                       temp, h->ws.invT, h->ws.vpart, 0, (const int32_t*)nullptr);
    hipLaunchKernelGGL(k_vtarget_comb, dim3(r1, batch), dim3(kWave), 0, st, h->B, nc, temp,
                       h->ws.vpart, h->ws.vstat, 0, (const int32_t*)nullptr);
  }
  hipLaunchKernelGGL((k_vaccept<T>), dim3(batch), dim3(64), 0, st, h->B, h->V, M, with_read,
                     draft, temp, skip, tids, tl, racc, h->ws.s, M, (const T*)h->W_r,
                     (const T*)h->ws.z, h->ws.lse, h->ws.vstat, h->ws.vpos, out_n, out_next,
                     h->ws.err, h->ws.invT, 0, r1);
  if (temp && r1 < h->B + 1) {
    hipLaunchKernelGGL(k_vtarget_part, dim3(nc, h->B + 1 - r1, batch), dim3(256), 0, st, tl,
                       h->B, h->V, temp, h->ws.invT, h->ws.vpart, r1, h->ws.vpos);
    hipLaunchKernelGGL(k_vtarget_comb, dim3(h->B + 1 - r1, batch), dim3(kWave), 0, st, h->B, nc,
                       temp, h->ws.vpart, h->ws.vstat, r1, h->ws.vpos);
    hipLaunchKernelGGL((k_vaccept<T>), dim3(batch), dim3(64), 0, st, h->B, h->V, M, with_read,
                       draft, temp, skip, tids, tl, racc, h->ws.s, M, (const T*)h->W_r,
                       (const T*)h->ws.z, h->ws.lse, h->ws.vstat, h->ws.vpos, out_n, out_next,
                       h->ws.err, h->ws.invT, r1, h->B + 1);
  }
  if (temp) {
    hipLaunchKernelGGL((k_vresid<T>), dim3(h->read_wgs, (batch + 15) / 16),
                       dim3(kReadWaves * kWave), 0, st, batch, h->B, h->V, M, with_read,
                       h->ntiles, h->read_units, temp, h->ws.vpos, tl, h->ws.s, M,
                       (const T*)h->W_r, (const T*)h->ws.z, h->ws.lse, h->ws.vstat, h->ws.vmass,
                       h->ws.invT);
    hipLaunchKernelGGL((k_vfinal<T>), dim3(batch), dim3(kVfWaves * kWave), 0, st, batch, h->B, h->V, M,
                       with_read, h->ntiles, h->read_units, temp, h->ws.vpos, tl, h->ws.s,
                       M, (const T*)h->W_r, (const T*)h->ws.z, h->ws.lse, h->ws.vstat,
                       h->ws.vmass, ures, out_next, h->ws.invT);
  }
  if (filtering) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_vfilter(h, batch, draft, tl, racc, ures, out_n, out_next, st);
  }
  return hipGetLastError();
}

hipError_t launch_verify(xp_handle* h, int batch, const int32_t* draft_ids, const uint8_t* temp,
                         const int32_t* target_ids, const float* target_logits,
                         const float* r_accept, const float* u_res, int32_t* out_n,
                         int32_t* out_next, hipStream_t st) {
  if (h->dtype == XP_BF16)
    return verify_t<uint16_t>(h, batch, draft_ids, temp, target_ids, target_logits, r_accept,
                              u_res, out_n, out_next, st);
  return verify_t<float>(h, batch, draft_ids, temp, target_ids, target_logits, r_accept, u_res,
                         out_n, out_next, st);
}

}  // namespace xp
