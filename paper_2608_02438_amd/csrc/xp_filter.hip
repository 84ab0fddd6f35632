// Truncated (top-k / top-p) sampling at temperature T, in refinement and in
// verification (the filtered form of the T > 0 sampling that speculative
// verification keeps lossless, section 3.1).
//
// On the scaled logits x_v = fl32(l_v * fl32(1/T)) of one row:
//   top-k keeps every v whose x_v is at least the k-th largest x (ties with it
//         stay);
//   top-p then orders the kept tokens by x descending, ties by lower index,
//         and keeps each token whose preceding mass in that order is below
//         p times the kept mass: the shortest prefix reaching p of it;
//   the kept tokens are sampled by inverse CDF in vocabulary order,
//         y = min{v : sum_{w <= v, kept} e^(x_w - m) > u Z}.
// A row's filter is a state (m, tk, tp, pidx, Z): v is kept iff
// key(x_v) >= tk and (key(x_v) > tp or (key(x_v) == tp and v <= pidx)), with
// key() the order-preserving 32-bit image of a float; Z is the kept mass.
//
// One workgroup of 16 waves per row, the row re-read from memory (L2) by
// every step:
//   1. m = max x, and a 256-bin count histogram of the keys' top byte;
//   2. top-k: radix select of the k-th largest key, one byte per step (bin
//      counts in LDS: integer atomics, so the result does not depend on their
//      order);
//   3. top-p: the same radix select on masses, each token's e^(x - m) held as
//      a 64-bit fixed-point integer (2^-44 units; at most 2^18 tokens of at
//      most 2^44 each), again order-independent; tokens tied at the cut value
//      are kept in index order while the mass before them stays below p Z;
//   4. Z and the inverse-CDF choice in fp64 in a fixed order: each wave sums
//      a contiguous range of the vocabulary with in-order wave scans, the
//      wave totals are added in wave order, and the wave whose running total
//      passes u Z rescans its range for the crossing token.
// Everything is deterministic: two runs give the same tokens and states.
#include "xp_internal.h"

namespace xp {

constexpr int kFWaves = 16;
constexpr int kFThreads = kFWaves * kWave;
constexpr double kFixScale = 17592186044416.0;   // 2^44

// order-preserving key: x < y  <=>  key(x) < key(y); -0 and +0 map alike
__device__ __forceinline__ uint32_t okey(float x) {
  const uint32_t b = x == 0.f ? 0u : __float_as_uint(x);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}
__device__ __forceinline__ double fweight(float x, float m) { return exp((double)x - (double)m); }
__device__ __forceinline__ uint64_t fixw(float x, float m) {
  return (uint64_t)(fweight(x, m) * kFixScale);     // truncation; e^(x - m) <= 1
}
__device__ __forceinline__ bool fkept(uint32_t key, int v, const FState& s) {
  return key >= s.tk && (key > s.tp || (key == s.tp && v <= s.pidx));
}

__device__ __forceinline__ double fwave_scan(double x, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double y = __shfl_up(x, off, kWave);
    if (lane >= off) x += y;
  }
  return x;
}

struct FShared {
  uint32_t hc[256];            // count histogram (top-k)
  unsigned long long hm[256];  // fixed-point mass histogram (top-p)
  float wmax[kFWaves];
  unsigned long long wsum[kFWaves];
  double wtot[kFWaves];
  uint32_t prefix;
  int need;
  unsigned long long above;
  int pidx;
  int pick;
  double start;
};

// Block-wide filter state of the row x(v), v < V (every thread calls it; on
// return s holds m, tk, tp and pidx of the row; Z is filled by the caller).
// k = 0: no top-k; p >= 1: no top-p.
template <class XF>
__device__ FState filter_state(XF x, int V, int k, float p, FShared& sh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool ka = k > 0 && k < V, pa = p < 1.f;
  for (int j = tid; j < 256; j += kFThreads) {
    sh.hc[j] = 0u;
    sh.hm[j] = 0ull;
  }
  __syncthreads();
  // 1. maximum, and the top-byte counts for top-k
  float mx = -INFINITY;
  for (int v = tid; v < V; v += kFThreads) {
    const float xv = x(v);
    mx = fmaxf(mx, xv);
    if (ka) atomicAdd(&sh.hc[okey(xv) >> 24], 1u);
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
  if (lane == 0) sh.wmax[wave] = mx;
  __syncthreads();
  float m = sh.wmax[0];
#pragma unroll
  for (int w = 1; w < kFWaves; ++w) m = fmaxf(m, sh.wmax[w]);
  FState s;
  s.m = m;
  s.tk = 0u;
  s.tp = 0u;
  s.pidx = 0x7FFFFFFF;
  s.Z = 0.0;
  // 2. top-k: the k-th largest key, one byte at a time from the top; `need`
  // is the rank still to find among the keys that match the prefix so far
  if (ka) {
    if (tid == 0) {
      sh.prefix = 0u;
      sh.need = k;
    }
    for (int byte = 3; byte >= 0; --byte) {
      if (byte < 3) {
        __syncthreads();
        for (int j = tid; j < 256; j += kFThreads) sh.hc[j] = 0u;
        __syncthreads();
        const int sh_hi = 8 * (byte + 1);
        const uint32_t pre = sh.prefix >> sh_hi;
        for (int v = tid; v < V; v += kFThreads) {
          const uint32_t kv = okey(x(v));
          if ((kv >> sh_hi) == pre) atomicAdd(&sh.hc[(kv >> (8 * byte)) & 255u], 1u);
        }
      }
      __syncthreads();
      if (tid == 0) {
        int cum = 0, sel = 0;
        for (int j = 255; j >= 0; --j) {
          const int c = (int)sh.hc[j];
          if (cum + c >= sh.need) {
            sel = j;
            break;
          }
          cum += c;
        }
        sh.need -= cum;
        sh.prefix |= (uint32_t)sel << (8 * byte);
      }
    }
    __syncthreads();
    s.tk = sh.prefix;
  }
  // 3. top-p over the top-k set: Zk, then the cut key, by fixed-point mass
  if (pa) {
    __syncthreads();
    for (int j = tid; j < 256; j += kFThreads) sh.hm[j] = 0ull;
    __syncthreads();
    unsigned long long zl = 0ull;
    for (int v = tid; v < V; v += kFThreads) {
      const float xv = x(v);
      const uint32_t kv = okey(xv);
      if (kv >= s.tk) {
        const unsigned long long w = fixw(xv, m);
        zl += w;
        atomicAdd(&sh.hm[kv >> 24], w);
      }
    }
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) zl += __shfl_xor(zl, o, kWave);
    if (lane == 0) sh.wsum[wave] = zl;
    if (tid == 0) {
      sh.prefix = 0u;
      sh.above = 0ull;
    }
    __syncthreads();
    unsigned long long Zk = 0ull;
#pragma unroll
    for (int w = 0; w < kFWaves; ++w) Zk += sh.wsum[w];
    const double target = (double)p * (double)Zk;
    for (int byte = 3; byte >= 0; --byte) {
      if (byte < 3) {
        __syncthreads();
        for (int j = tid; j < 256; j += kFThreads) sh.hm[j] = 0ull;
        __syncthreads();
        const int sh_hi = 8 * (byte + 1);
        const uint32_t pre = sh.prefix >> sh_hi;
        for (int v = tid; v < V; v += kFThreads) {
          const float xv = x(v);
          const uint32_t kv = okey(xv);
          if (kv >= s.tk && (kv >> sh_hi) == pre)
            atomicAdd(&sh.hm[(kv >> (8 * byte)) & 255u], fixw(xv, m));
        }
      }
      __syncthreads();
      if (tid == 0) {
        // the highest bin whose mass, with everything above it, reaches p Zk
        unsigned long long cum = sh.above;
        int sel = 0;
        for (int j = 255; j >= 0; --j) {
          const unsigned long long c = sh.hm[j];
          if (c != 0ull && (double)(cum + c) >= target) {
            sel = j;
            break;
          }
          cum += c;
        }
        sh.above = cum;
        sh.prefix |= (uint32_t)sel << (8 * byte);
      }
    }
    __syncthreads();
    s.tp = sh.prefix;
    // tokens tied at the cut value: keep them in index order while the mass
    // before them (all of equal weight wt) stays below p Zk
    const unsigned long long A = sh.above, wt = fixw(key_value(s.tp), m);
    const unsigned long long c = wt ? sh.hm[s.tp & 255u] / wt : 1ull;
    unsigned long long nt = wt ? (unsigned long long)ceil((target - (double)A) / (double)wt) : 1ull;
    nt = nt < 1ull ? 1ull : (nt > c ? c : nt);
    while (nt > 1ull && (double)(A + (nt - 1ull) * wt) >= target) --nt;
    while (nt < c && (double)(A + nt * wt) < target) ++nt;
    if (nt < c) {
      // index of the nt-th tied token: one wave counts them in order
      if (wave == 0) {
        unsigned long long seen = 0ull;
        int found = V - 1;
        for (int base = 0; base < V; base += kWave) {
          const int v = base + lane;
          const bool t = v < V && okey(x(v)) == s.tp;
          const unsigned long long bal = __ballot(t);
          const unsigned long long cnt = __popcll(bal);
          if (seen + cnt >= nt) {
            unsigned long long b2 = bal;
            for (unsigned long long r = seen + 1ull; r < nt; ++r) b2 &= b2 - 1ull;
            found = base + __ffsll((long long)b2) - 1;
            break;
          }
          seen += cnt;
        }
        if (lane == 0) sh.pidx = found;
      }
      __syncthreads();
      s.pidx = sh.pidx;
    }
  }
  return s;
}

// Ordered fp64 sum of weight(v) over v < V: wave w sums the contiguous range
// [V w / 16, V (w + 1) / 16) with in-order scans; the wave totals are added in
// wave order.  Leaves each wave's total in sh.wtot.
template <class WF>
__device__ double ordered_sum(WF weight, int V, FShared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lo = (int)((int64_t)V * wave / kFWaves), hi = (int)((int64_t)V * (wave + 1) / kFWaves);
  double carry = 0.0;
  for (int base = lo; base < hi; base += kWave) {
    const int v = base + lane;
    const double w = v < hi ? weight(v) : 0.0;
    carry += __shfl(fwave_scan(w, lane), 63, kWave);
  }
  __syncthreads();
  if (lane == 0) sh.wtot[wave] = carry;
  __syncthreads();
  double Z = 0.0;
#pragma unroll
  for (int w = 0; w < kFWaves; ++w) Z += sh.wtot[w];
  return Z;
}

// Inverse-CDF choice over weight(v) after ordered_sum() gave Z (its wave
// totals still in sh.wtot): the smallest v whose running sum exceeds u Z, in
// the same summation order; when rounding leaves no crossing, the last v of
// nonzero weight.  Returns the choice in every thread.
template <class WF>
__device__ int ordered_icdf(WF weight, int V, double Z, double u, FShared& sh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const double target = u * Z;
  if (tid == 0) {
    double run = 0.0;
    int ws = -1;
    for (int w = 0; w < kFWaves; ++w) {
      if (run + sh.wtot[w] > target) {
        ws = w;
        break;
      }
      run += sh.wtot[w];
    }
    if (ws < 0) {                                   // no crossing: the last wave with mass
      ws = kFWaves - 1;
      while (ws > 0 && !(sh.wtot[ws] > 0.0)) --ws;
      run = 0.0;
      for (int w = 0; w < ws; ++w) run += sh.wtot[w];
    }
    sh.pick = ws;
    sh.start = run;
  }
  __syncthreads();
  if (wave == sh.pick) {
    const int lo = (int)((int64_t)V * wave / kFWaves), hi = (int)((int64_t)V * (wave + 1) / kFWaves);
    double cum = sh.start;
    int chosen = -1, last_nz = -1;
    for (int base = lo; base < hi; base += kWave) {
      const int v = base + lane;
      const double w = v < hi ? weight(v) : 0.0;
      const double tot = cum + fwave_scan(w, lane);
      const unsigned long long hit = __ballot(v < hi && tot > target);
      const unsigned long long nz = __ballot(v < hi && w > 0.0);
      if (nz) last_nz = base + 63 - __clzll((long long)nz);
      if (hit) {
        chosen = base + __ffsll((long long)hit) - 1;
        break;
      }
      cum = __shfl(tot, 63, kWave);
    }
    if (chosen < 0) chosen = last_nz >= 0 ? last_nz : lo;
    if (lane == 0) sh.pidx = chosen;                // reuses the slot: filter state is kept in s
  }
  __syncthreads();
  return sh.pidx;
}

// Per-sequence sampling parameters: filt[b] = the row samples and truncates;
// temp_nf[b] = the row samples without truncation (the untruncated sampler's
// rows); fk, fp the effective top-k (0 = none) and top-p (1 = none).  A
// negative k or a p that is not positive is an error (XP_DEVERR_FILTER) and
// is replaced by no truncation; k >= V and p >= 1 mean none.  Greedy rows
// ignore both.
__global__ void k_filter_params(int batch, int V, const uint8_t* __restrict__ temp,
                                const int32_t* __restrict__ top_k, const float* __restrict__ top_p,
                                uint8_t* __restrict__ filt, uint8_t* __restrict__ temp_nf,
                                int32_t* __restrict__ fk, float* __restrict__ fp,
                                uint32_t* __restrict__ err) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= batch) return;
  const bool smp = temp != nullptr && temp[b] != 0;
  int k = top_k != nullptr ? top_k[b] : 0;
  float p = top_p != nullptr ? top_p[b] : 1.f;
  bool bad = false;
  if (k < 0) {
    bad = true;
    k = 0;
  }
  if (!(p > 0.f)) {                               // p <= 0 or NaN
    bad = true;
    p = 1.f;
  }
  if (k >= V) k = 0;
  if (!(p < 1.f)) p = 1.f;
  const bool f = smp && (k > 0 || p < 1.f);
  filt[b] = f ? 1 : 0;
  temp_nf[b] = (smp && !f) ? 1 : 0;
  fk[b] = k;
  fp[b] = p;
  if (smp && bad) atomicOr(err, XP_DEVERR_FILTER);
}

// Truncated sampling of one position per workgroup.  MODE 0: the seed Y^(0)
// from the base logits s (tile-major); with caller seed ids only the state is
// kept.  MODE 1: the selection of a Jacobi pass from the pass's logits
// (row-major, written by the Read stream).  The chosen token goes to Ynew for
// the selection kernel that follows; the state to fst for verification.
template <int MODE>
__global__ __launch_bounds__(kFThreads) void k_fsample(
    int B, int V, int M, const float* __restrict__ S, int Ms, const float* __restrict__ lf,
    const uint8_t* __restrict__ filt, const int32_t* __restrict__ fk, const float* __restrict__ fp,
    const float* __restrict__ invT, const float* __restrict__ u_draft,
    const int32_t* __restrict__ seed_ids, int32_t* __restrict__ Ynew, FState* __restrict__ fst,
    const int32_t* __restrict__ iters, int early_exit) {
  const int p = blockIdx.x, b = p / B;
  if (!filt[b]) return;
  if (MODE == 1 && early_exit && iters[b] != 0) return;     // the sequence keeps Y^(j)
  __shared__ FShared sh;
  const float it = invT[b];
  auto x = [&](int v) -> float {
    return (MODE == 0 ? S[s_index(p, v, Ms)] : lf[(size_t)p * V + v]) * it;
  };
  FState s = filter_state(x, V, fk[b], fp[b], sh);
  auto w = [&](int v) -> double {
    const float xv = x(v);
    return fkept(okey(xv), v, s) ? fweight(xv, s.m) : 0.0;
  };
  s.Z = ordered_sum(w, V, sh);
  if (!(MODE == 0 && seed_ids != nullptr)) {
    const int y = ordered_icdf(w, V, s.Z, (double)u_draft[p], sh);
    if (threadIdx.x == 0) Ynew[p] = y;
  }
  if (threadIdx.x == 0) fst[p] = s;
}

// Filter state (with Z) of the target rows of truncated sequences, one
// workgroup per (row k = 0..B, sequence).
__global__ __launch_bounds__(kFThreads) void k_vfstate(
    int B, int V, const float* __restrict__ tl, const uint8_t* __restrict__ filt,
    const int32_t* __restrict__ fk, const float* __restrict__ fp, const float* __restrict__ invT,
    FState* __restrict__ tst) {
  const int k = blockIdx.x, b = blockIdx.y;
  if (!filt[b]) return;
  __shared__ FShared sh;
  const float it = invT[b];
  const float* row = tl + ((size_t)b * (B + 1) + k) * V;
  auto x = [&](int v) -> float { return row[v] * it; };
  FState s = filter_state(x, V, fk[b], fp[b], sh);
  auto w = [&](int v) -> double {
    const float xv = x(v);
    return fkept(okey(xv), v, s) ? fweight(xv, s.m) : 0.0;
  };
  s.Z = ordered_sum(w, V, sh);
  if (threadIdx.x == 0) tst[(size_t)b * (B + 1) + k] = s;
}

// Probability of token y under a truncated row: e^(x_y - m) / Z if kept.
__device__ __forceinline__ double fprob(float xv, int y, const FState& s) {
  return fkept(okey(xv), y, s) ? fweight(xv, s.m) / s.Z : 0.0;
}

// Logit of draft position p at token v: the last pass's (row-major) or, after
// K = 0 passes, the base logits (tile-major).
__device__ __forceinline__ float draft_logit(int k0, const float* __restrict__ lf,
                                             const float* __restrict__ S, int Ms, int V, int p,
                                             int v) {
  return k0 ? S[s_index(p, v, Ms)] : lf[(size_t)p * V + v];
}

// Accept scan of truncated sequences, one wave per sequence: accept y_k iff
// r_k q_k(y_k) <= p_k(y_k), both truncated.  vpos[b] = rejected position or B.
__global__ __launch_bounds__(64) void k_vfaccept(
    int B, int V, int k0, const int32_t* __restrict__ draft, const uint8_t* __restrict__ filt,
    const float* __restrict__ tl, const float* __restrict__ racc, const float* __restrict__ lf,
    const float* __restrict__ S, int Ms, const FState* __restrict__ fst,
    const FState* __restrict__ tst, const float* __restrict__ invT, int32_t* __restrict__ vpos,
    int32_t* __restrict__ out_n, uint32_t* __restrict__ err) {
  const int b = blockIdx.x;
  if (!filt[b] || threadIdx.x != 0) return;
  const float it = invT[b];
  int n = B, bad = 0;
  for (int k = 0; k < B; ++k) {
    const int p = b * B + k;
    int y = draft[p];
    if (y < 0 || y >= V) {
      bad = 1;
      y = 0;
    }
    const double q = fprob(draft_logit(k0, lf, S, Ms, V, p, y) * it, y, fst[p]);
    const double pt = fprob(tl[((size_t)b * (B + 1) + k) * V + y] * it, y,
                            tst[(size_t)b * (B + 1) + k]);
    if (!((double)racc[p] * q <= pt)) {
      n = k;
      break;
    }
  }
  out_n[b] = n;
  vpos[b] = n;
  if (bad) atomicOr(err, XP_DEVERR_TOKEN);
}

// Next token of truncated sequences, one workgroup per sequence: at the
// rejected position k the inverse-CDF sample of max(0, p_k - q_k) (of p_k if
// that has no mass), after B accepts the sample of p_{B+1}; at u_res.
__global__ __launch_bounds__(kFThreads) void k_vffinal(
    int B, int V, int k0, const uint8_t* __restrict__ filt, const float* __restrict__ tl,
    const float* __restrict__ lf, const float* __restrict__ S, int Ms,
    const FState* __restrict__ fst, const FState* __restrict__ tst,
    const float* __restrict__ invT, const int32_t* __restrict__ vpos,
    const float* __restrict__ ures, int32_t* __restrict__ out_next) {
  const int b = blockIdx.x;
  if (!filt[b]) return;
  __shared__ FShared sh;
  const float it = invT[b];
  const int n = vpos[b];
  const float* trow = tl + ((size_t)b * (B + 1) + n) * V;
  const FState ts = tst[(size_t)b * (B + 1) + n];
  auto wp = [&](int v) -> double {
    const float xv = trow[v] * it;
    return fkept(okey(xv), v, ts) ? fweight(xv, ts.m) / ts.Z : 0.0;
  };
  const double u = (double)ures[b];
  int y;
  if (n < B) {
    const int p = b * B + n;
    const FState qs = fst[p];
    auto wr = [&](int v) -> double {
      const double pv = wp(v);
      const float xq = draft_logit(k0, lf, S, Ms, V, p, v) * it;
      const double qv = fkept(okey(xq), v, qs) ? fweight(xq, qs.m) / qs.Z : 0.0;
      return pv > qv ? pv - qv : 0.0;
    };
    const double Zr = ordered_sum(wr, V, sh);
    if (Zr > 0.0) {
      y = ordered_icdf(wr, V, Zr, u, sh);
    } else {
      const double Zp = ordered_sum(wp, V, sh);
      y = ordered_icdf(wp, V, Zp, u, sh);
    }
  } else {
    const double Zp = ordered_sum(wp, V, sh);
    y = ordered_icdf(wp, V, Zp, u, sh);
  }
  if (threadIdx.x == 0) out_next[b] = y;
}

// ---------------------------------------------------------------------------
hipError_t launch_filter_params(xp_handle* h, int batch, const uint8_t* temp, const int32_t* top_k,
                                const float* top_p, hipStream_t st) {
  hipLaunchKernelGGL(k_filter_params, dim3((batch + 255) / 256), dim3(256), 0, st, batch, h->V,
                     temp, top_k, top_p, h->ws.filt, h->ws.temp_nf, h->ws.fk, h->ws.fp,
                     h->ws.err);
  return hipGetLastError();
}

hipError_t launch_fsample(xp_handle* h, int batch, int pass, uint32_t flags,
                          const int32_t* seed_ids, const float* u_draft, hipStream_t st) {
  const int M = batch * h->B;
  int32_t* Ynew = h->ws.Y[(pass + 1) % 2];
  const int early = (flags & XP_EARLY_EXIT) ? 1 : 0;
  if (pass < 0)
    hipLaunchKernelGGL((k_fsample<0>), dim3(M), dim3(kFThreads), 0, st, h->B, h->V, M, h->ws.s, M,
                       h->ws.lf, h->ws.filt, h->ws.fk, h->ws.fp, h->ws.invT, u_draft, seed_ids,
                       Ynew, h->ws.fst, h->ws.iters, early);
  else
    hipLaunchKernelGGL((k_fsample<1>), dim3(M), dim3(kFThreads), 0, st, h->B, h->V, M, h->ws.s, M,
                       h->ws.lf, h->ws.filt, h->ws.fk, h->ws.fp, h->ws.invT, u_draft, nullptr,
                       Ynew, h->ws.fst, h->ws.iters, early);
  return hipGetLastError();
}

hipError_t launch_vfilter(xp_handle* h, int batch, const int32_t* draft, const float* tl,
                          const float* racc, const float* ures, int32_t* out_n, int32_t* out_next,
                          hipStream_t st) {
  const int M = batch * h->B;
  const int k0 = h->state_k0 ? 1 : 0;
  hipLaunchKernelGGL(k_vfstate, dim3(h->B + 1, batch), dim3(kFThreads), 0, st, h->B, h->V, tl,
                     h->ws.filt, h->ws.fk, h->ws.fp, h->ws.invT, h->ws.tst);
  hipLaunchKernelGGL(k_vfaccept, dim3(batch), dim3(64), 0, st, h->B, h->V, k0, draft, h->ws.filt,
                     tl, racc, h->ws.lf, h->ws.s, M, h->ws.fst, h->ws.tst, h->ws.invT, h->ws.vpos,
                     out_n, h->ws.err);
  hipLaunchKernelGGL(k_vffinal, dim3(batch), dim3(kFThreads), 0, st, h->B, h->V, k0, h->ws.filt,
                     tl, h->ws.lf, h->ws.s, M, h->ws.fst, h->ws.tst, h->ws.invT, h->ws.vpos, ures,
                     out_next);
  return hipGetLastError();
}

}  // namespace xp
