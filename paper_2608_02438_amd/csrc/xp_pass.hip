// One greedy Jacobi pass front half as a single kernel: the selection of the
// previous pass (Algorithm 1: argmax of the refined or base logits), the
// Fuse gather (a_k = Pa_k + T[x_{k-1}], section 4.1), Mix (eq. mix) and the
// first Trans product h1 = silu(W_1 c) (eq. mlp).
//
// Grid (batch, 32 row tiles of W_1).  Every workgroup of a sequence takes the
// argmax from the per-unit keys and runs Fuse + Mix for the whole sequence
// itself (a few tens of KB from L2), so the three steps need no kernel
// boundary between them; it then owns 16 rows of h1.  Workgroups rt < 16 also
// write the 16 feature dims [16 rt, 16 rt + 16) of c for the residual of
// Trans, and workgroup 0 does the bookkeeping of the selection (iterate,
// trajectory, fixed-point test).  Used for all-greedy batches with blocks of
// at most 16 positions and bf16 weights; other batches take the separate
// select / fusemix / trans1 kernels, which compute the same values.
#include "xp_internal.h"
#include "xp_split.h"

namespace xp {

constexpr int kPassUnits = 256;      // most key units per position
constexpr int kPassPairs = 120;      // L pairs of a 16-position block

__global__ __launch_bounds__(256) void k_pass(
    int mode, int pass, int batch, int B, int V, int M, const uint64_t* __restrict__ keys,
    int nkeys, const int32_t* __restrict__ seed_ids, const float* __restrict__ Pa,
    const float* __restrict__ Ttab, const uint16_t* __restrict__ Lp,
    const int32_t* __restrict__ anchor, const int32_t* __restrict__ Yprev,
    int32_t* __restrict__ Ynew, int32_t* __restrict__ traj, int32_t* __restrict__ iters,
    int32_t* __restrict__ ctrl, uint32_t* __restrict__ err, int early_exit,
    const uint16_t* __restrict__ W1, float* __restrict__ c, float* __restrict__ h1) {
  constexpr int r = 256, r2 = 512, CS = r + 4;
  constexpr int KPT = kPassUnits * 16 / 256;         // keys per thread
  constexpr int LPT = kPassPairs * r * 2 / 16 / 256; // 16-byte L chunks per thread
  __shared__ float A[16][CS];                        // a_k, then c_k
  __shared__ u32x4 Ls[kPassPairs * r * 2 / 16];      // L of the block (60 KB)
  __shared__ uint64_t kred[4][16];
  __shared__ int ys[16];
  __shared__ int chg;
  __shared__ floatx4 red[4][64];
  const int b = blockIdx.x, rt = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, g = lane >> 4, li = lane & 15;
  // early exit: a sequence already at its fixed point keeps its block (the
  // first workgroup carries it over to the next iterate buffer)
  const bool skip = mode == 1 && early_exit && iters[b] != 0;
  if (skip) {
    if (rt == 0 && tid < B) {
      const size_t p = (size_t)b * B + tid;
      const int y = Yprev[p];
      Ynew[p] = y;
      if (traj) traj[p] = y;
    }
    return;
  }

  // --- every independent load first -----------------------------------------
  const int kk = tid & 15, kkc = kk < B ? kk : B - 1;          // key role: position kk
  uint64_t kv[KPT];
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const int i = (tid >> 4) + 16 * j;
    kv[j] = keys[(size_t)(i < nkeys ? i : nkeys - 1) * M + (size_t)b * B + kkc];
  }
  const int nch = (B * (B - 1) / 2) * (r * 2 / 16);
  u32x4 lc[LPT];
  const u32x4* lsrc = reinterpret_cast<const u32x4*>(Lp);
#pragma unroll
  for (int j = 0; j < LPT; ++j) {
    const int q = tid + 256 * j;
    lc[j] = lsrc[q < nch ? q : (nch > 0 ? nch - 1 : 0)];
  }
  const int k0 = wave * (r / 4);                                // W_1 k slice of the wave
  const uint16_t* arow = W1 + (size_t)(rt * 16 + li) * r + k0;
  u32x4 w[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) w[u] = ld16(arow + u * 32 + 8 * g);
  const int pk = tid >> 4, pkc = pk < B ? pk : B - 1;          // gather role: position pk
  const int d0 = (tid & 15) * 16;
  float4 pa[4];
#pragma unroll
  for (int q = 0; q < 4; ++q)
    pa[q] = *reinterpret_cast<const float4*>(Pa + ((size_t)b * B + pkc) * r + d0 + 4 * q);
  const int ya = anchor[b];
  const int yp = mode == 1 ? Yprev[(size_t)b * B + kkc] : 0;
  const int sd = (mode == 0 && seed_ids != nullptr) ? seed_ids[(size_t)b * B + kkc] : 0;
  const int it0 = iters[b];

  // --- selection of the previous pass -----------------------------------------
  uint64_t best = kv[0];
#pragma unroll
  for (int j = 1; j < KPT; ++j) best = umax64(best, kv[j]);
  best = umax64(best, shfl_xor_u64(best, 16));
  best = umax64(best, shfl_xor_u64(best, 32));
  if (lane < 16) kred[wave][lane] = best;
#pragma unroll
  for (int j = 0; j < LPT; ++j) {
    const int q = tid + 256 * j;
    if (q < nch) Ls[q] = lc[j];
  }
  if (tid == 0) chg = 0;
  __syncthreads();
  if (tid < 16) {
    uint64_t bb = kred[0][tid];
#pragma unroll
    for (int w2 = 1; w2 < 4; ++w2) bb = umax64(bb, kred[w2][tid]);
    int y = (int)key_index(bb);
    if (skip) {
      y = yp;
    } else if (mode == 0 && seed_ids != nullptr) {
      y = sd;
      if (y < 0 || y >= V) {
        if (tid < B && rt == 0) atomicOr(err, XP_DEVERR_TOKEN);
        y = 0;
      }
    }
    ys[tid] = y;
    if (tid < B) {
      if (rt == 0) {
        const size_t p = (size_t)b * B + tid;
        Ynew[p] = y;
        if (traj) traj[p] = y;
      }
      if (mode == 1 && y != yp) atomicOr(&chg, 1);
    }
  }
  __syncthreads();
  // --- fixed-point bookkeeping of the selection (Algorithm 1) -----------------
  // Every workgroup of the sequence sees the same selection: when it has just
  // reached the fixed point (or had before), the rest of this pass is not
  // needed under the early exit.
  const bool now_fixed = mode == 1 && !skip && chg == 0 && it0 == 0;
  if (rt == 0 && tid == 0 && now_fixed) {
    iters[b] = pass;                               // the selection of pass `pass - 1`
    if (atomicAdd(&ctrl[0], 1) + 1 == batch) ctrl[1] = 1;
  }
  if (skip || (early_exit && now_fixed)) return;   // whole workgroup

  // --- Fuse: a_k = Pa_k + T[x_{k-1}] ------------------------------------------
  {
    int x = pk == 0 ? ya : ys[pk - 1];
    const bool ok = x >= 0 && x < V;
    if (!ok && pk < B && rt == 0 && (tid & 15) == 0) atomicOr(err, XP_DEVERR_TOKEN);
    x = ok ? x : 0;
    const float* trow = Ttab + (size_t)x * r + d0;
    float4 t[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) t[q] = *reinterpret_cast<const float4*>(trow + 4 * q);
    // rows past the block are zeroed arithmetically (no branch, so the loads
    // above stay unconditional and overlap)
    const float mask = pk < B ? 1.f : 0.f;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<float4*>(&A[pk][d0 + 4 * q]) =
          make_float4((pa[q].x + t[q].x) * mask, (pa[q].y + t[q].y) * mask,
                      (pa[q].z + t[q].z) * mask, (pa[q].w + t[q].w) * mask);
  }
  __syncthreads();

  // --- Mix: c_k = a_k + sum_{i<k} L[d][k][i] a_i, one feature dim per thread;
  //     the triangle is unrolled so that all its LDS reads are in flight -----
  {
    const int d = tid;
    const uint16_t* ls = reinterpret_cast<const uint16_t*>(Ls);
    float a[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) a[k] = A[k][d];
#pragma unroll
    for (int k = 1; k < 16; ++k) {
      if (k < B) {
        float acc = a[k];
#pragma unroll
        for (int i = 0; i < k; ++i) acc += bf16_to_f32(ls[(k * (k - 1) / 2 + i) * r + d]) * a[i];
        A[k][d] = acc;
      }
    }
  }
  __syncthreads();
  if (rt < 16 && pk < B) {                          // c columns of this workgroup
    const int dl = tid & 15;
    c[((size_t)b * B + pk) * r + rt * 16 + dl] = A[pk][rt * 16 + dl];
  }

  // --- h1 rows [16 rt, 16 rt + 16) = silu(W_1 c) ------------------------------
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const float* crow = &A[li][k0 + u * 32 + 8 * g];
    const float4 x0 = *reinterpret_cast<const float4*>(crow);
    const float4 x1 = *reinterpret_cast<const float4*>(crow + 4);
    acc = mma_split_b(w[u], x0, x1, acc);
  }
  red[wave][lane] = acc;
  __syncthreads();
  if (wave == 0) {
    const floatx4 q0 = red[0][lane], q1 = red[1][lane], q2 = red[2][lane], q3 = red[3][lane];
    if (li < B) {
      float o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = ((q0[i] + q1[i]) + q2[i]) + q3[i];
        o[i] = v / (1.f + expf(-v));
      }
      *reinterpret_cast<float4*>(h1 + ((size_t)b * B + li) * r2 + rt * 16 + 4 * g) =
          make_float4(o[0], o[1], o[2], o[3]);
    }
  }
}

// ---------------------------------------------------------------------------
// Call after the A1 launch of the same refine (it sets the unit count).
bool pass_fused_ok(const xp_handle* h, const uint8_t* temp) {
  return temp == nullptr && h->dtype == XP_BF16 && h->B <= 16 && h->lm_units_cur <= kPassUnits &&
         h->read_wgs <= kPassUnits;
}

hipError_t launch_pass(xp_handle* h, int batch, int pass, uint32_t flags, const int32_t* seed_ids,
                       const int32_t* anchor, int32_t* out_traj, hipStream_t st) {
  const int M = batch * h->B;
  const int mode = pass == 0 ? 0 : 1;
  int32_t* Ynew = h->ws.Y[pass % 2];
  const int32_t* Yprev = h->ws.Y[(pass + 1) % 2];
  int32_t* traj = out_traj ? out_traj + (size_t)pass * M : nullptr;
  const int nkeys = mode == 0 ? h->lm_units_cur : h->read_wgs;
  const int early = (flags & XP_EARLY_EXIT) ? 1 : 0;
  hipLaunchKernelGGL(k_pass, dim3(batch, 32), dim3(256), 0, st, mode, pass, batch, h->B, h->V, M,
                     h->ws.keys, nkeys, mode == 0 ? seed_ids : nullptr, h->ws.Pa, h->ws.T,
                     (const uint16_t*)h->ws.Lp, anchor, Yprev, Ynew, traj, h->ws.iters,
                     h->ws.ctrl, h->ws.err, early, (const uint16_t*)h->W_1, h->ws.c, h->ws.h1);
  return hipGetLastError();
}

}  // namespace xp
