// Host-side internals: the handle, its workspace, and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/xpress.h"
#include "xp_device.h"

namespace xp {

// Launch shapes of the two vocabulary streams (tuned for 256 CUs).
constexpr int kLmWaves = 16;    // A1: waves per workgroup, each owning H/16 of the k range
constexpr int kReadWaves = 8;   // A7: waves per workgroup, each streaming its own tiles
constexpr int kMaxK = 64;

// Truncation state of one row (xp_filter.hip): token v is kept iff
// key(x_v) >= tk and (key(x_v) > tp or (key(x_v) == tp and v <= pidx)), key()
// the order-preserving image of the scaled logit; m = max x, Z = kept mass.
struct FState {
  float m;
  uint32_t tk, tp;
  int32_t pidx;
  double Z;
};

struct Workspace {
  float* s = nullptr;         // base logits s_k, tile-major (s_index), Mmax x ldS floats
  float* T = nullptr;         // [V][r]        token table W_e W_in[:, 2r:3r]^T
  float* Fh = nullptr;        // [r][H]        W_in[:, 0:r] W_h
  float* Fg = nullptr;        // [r][H]        W_in[:, r:2r] W_g
  void* Lp = nullptr;         // [npairs][r]   L[d][k][i] (i < k) at pair k(k-1)/2 + i
  float* ppart = nullptr;     // [2][ksp][Mmax][r] k-slice partials of Fh h_k and Fg h_k
  float* Pa = nullptr;        // [Mmax][r]     Fh h_k + Fg g (pass-invariant part of Fuse)
  float* c = nullptr;         // [Mmax][r]     Mix output of the current pass
  float* h1 = nullptr;        // [Mmax][2r]    silu(W_1 c) of the current pass
  void* z = nullptr;          // [Mmax][r]     Trans output (dtype)
  int32_t* Y[2] = {nullptr, nullptr};   // [Mmax] iterates, ping-pong by pass parity
  uint64_t* keys = nullptr;   // [max chunks][Mmax]  greedy partials
  Stat* stats = nullptr;      // [Mmax][units]   sampling partials (position-major)
  double* lse = nullptr;      // [Mmax]        log-sum-exp of the last pass (sampled rows, l / T)
  float* invT = nullptr;      // [max_batch]   1 / temperature of each sequence (1 if none)
  int32_t* iters = nullptr;   // [max_batch]
  int32_t* ctrl = nullptr;    // [0] converged-sequence count, [1] all-converged flag
  uint32_t* err = nullptr;    // device error word
  // verification scratch
  double* vstat = nullptr;    // [max_batch][B+1][2] target (max, log-sum-exp) per row
  int32_t* vpos = nullptr;    // [max_batch][2] rejected position (or B), state
  double* vmass = nullptr;    // [max units][max_batch] residual / bonus mass per unit
  double* vpart = nullptr;    // [max_batch][B+1][vchunks][2] target row (max, sum) per chunk
  // truncated sampling (top-k / top-p)
  float* lf = nullptr;        // [Mmax][V]     logits of the current pass, row-major
  FState* fst = nullptr;      // [Mmax]        truncation state of each draft row (last pass)
  FState* tst = nullptr;      // [max_batch][B+1] truncation state of each target row
  uint8_t* filt = nullptr;    // [max_batch]   the row samples with truncation
  uint8_t* temp_nf = nullptr; // [max_batch]   the row samples without truncation
  int32_t* fk = nullptr;      // [max_batch]   effective top-k (0: none)
  float* fp = nullptr;        // [max_batch]   effective top-p (1: none)
};

// Target rows are reduced in chunks of kVChunk entries (16 per thread).
constexpr int kVChunk = 4096;
// Verification computes the target rows' log-sum-exp for the first kVRows1
// rows of every sampled sequence, and for the rest only where the accept scan
// got past them (marked kVMore in vpos).
constexpr int kVRows1 = 4;
constexpr int kVMore = -2;

}  // namespace xp

struct xp_timing_state {
  uint32_t mask = 0;
  int capacity = 0;
  std::vector<hipEvent_t> ev[XP_NSTAGES];   // 2 * capacity events per stage
  int n[XP_NSTAGES] = {0, 0, 0, 0, 0, 0};
};

struct xp_handle {
  int device = 0;
  int H = 0, r = 0, V = 0, B = 0, dtype = 0, max_batch = 0;
  const void *W_lm = nullptr, *W_h = nullptr, *W_g = nullptr, *W_e = nullptr, *W_in = nullptr,
             *L = nullptr, *W_1 = nullptr, *W_2 = nullptr, *W_r = nullptr;
  int ldS = 0, ntiles = 0;
  int cus = 0;
  int lm_chunks = 0;           // A1 stream workgroups along the vocabulary (= units)
  int lm_units_cur = 0;        // selection units of the last A1 launch (stream or GEMM)
  int read_wgs = 0;            // A7 workgroups along the vocabulary
  int read_units = 0;          // read_wgs * kReadWaves
  xp::Workspace ws;
  int last_batch = -1;         // batch of the last refine (verify state)
  bool state_valid = false;
  bool state_k0 = false;       // last refine ran K = 0 passes (q = softmax(s))
  bool state_temp = false;     // last refine was given sampling flags
  bool call_tempered = false;  // the current refine has sampled rows and a temperature array
  bool state_filtered = false; // last refine was given top-k / top-p arrays
  std::string err;
  xp_timing_state tm;
};

namespace xp {

// launchers (each returns hipGetLastError() of its launch)
hipError_t launch_fold(xp_handle* h, hipStream_t st);
hipError_t launch_prep(xp_handle* h, int batch, const void* hidden, const uint8_t* temp,
                       const float* temperature, hipStream_t st);
hipError_t launch_lmhead(xp_handle* h, int M, const void* hidden, const uint8_t* temp, hipStream_t st);
hipError_t launch_select(xp_handle* h, int batch, int pass, int K, uint32_t flags,
                         const int32_t* seed_ids, const uint8_t* temp, const float* u_draft,
                         int32_t* out_traj, int32_t* out_ids, int32_t* out_iters,
                         hipStream_t st, bool filtering);
// truncated sampling (xp_filter.hip)
hipError_t launch_filter_params(xp_handle* h, int batch, const uint8_t* temp, const int32_t* top_k,
                                const float* top_p, hipStream_t st);
hipError_t launch_fsample(xp_handle* h, int batch, int pass, uint32_t flags,
                          const int32_t* seed_ids, const float* u_draft, hipStream_t st);
hipError_t launch_vfilter(xp_handle* h, int batch, const int32_t* draft, const float* tl,
                          const float* racc, const float* ures, int32_t* out_n, int32_t* out_next,
                          hipStream_t st);
hipError_t launch_rspace(xp_handle* h, int batch, int pass, uint32_t flags, const int32_t* anchor,
                         bool front, hipStream_t st);
bool pass_fused_ok(const xp_handle* h, const uint8_t* temp);
int gemm_units(const xp_handle* h, int M);
// the context layer's projections for many positions (xp_lgemm.hip): tile
// size bn (128 or 256; 0: no plan) and S k splits; with S > 1 the launch
// writes S slabs of [M][N] fp32 partial products (Y, with R = Yb = NULL);
// the gate/up projections form the SwiGLU product (S = 1)
constexpr int kLayerSplitMax = 8;
constexpr size_t kLayerPartFloats = (size_t)16 << 20;   // slab values a layer holds (64 MB)
struct LayerPlan {
  int bn, S;
};
LayerPlan layer_plan(int n0, int n1, int N, int K, int M, bool glu, size_t part_floats);
hipError_t launch_layer_gemm(LayerPlan pl, const uint16_t* W0, const uint16_t* W1,
                             const uint16_t* W2, int n0, int n1, int N, int K, const uint16_t* X,
                             int M, const float* R, int ldr, float* Y, uint16_t* Yb, int ldy,
                             hipStream_t st);
hipError_t launch_layer_glu(LayerPlan pl, const uint16_t* Wg, const uint16_t* Wu, int F, int K,
                            const uint16_t* X, int M, uint16_t* act, int ldy, hipStream_t st);
int gemm_units_max(const xp_handle* h);
bool lmhead_gemm_ok(const xp_handle* h, int M);
hipError_t launch_lmhead_gemm(xp_handle* h, int M, const void* hidden, const uint8_t* temp,
                              hipStream_t st);
hipError_t launch_pass(xp_handle* h, int batch, int pass, uint32_t flags, const int32_t* seed_ids,
                       const int32_t* anchor, int32_t* out_traj, hipStream_t st);
int prep_ksp(int H);
hipError_t launch_read(xp_handle* h, int batch, int pass, uint32_t flags, const uint8_t* temp,
                       float* out_logits, hipStream_t st);
hipError_t launch_finish(xp_handle* h, int batch, int K, uint32_t flags, int32_t* out_ids,
                         int32_t* out_iters, float* out_logits, hipStream_t st, bool filtering);
hipError_t launch_verify(xp_handle* h, int batch, const int32_t* draft_ids, const uint8_t* temp,
                         const int32_t* target_ids, const float* target_logits,
                         const float* r_accept, const float* u_res, int32_t* out_n,
                         int32_t* out_next, hipStream_t st);

}  // namespace xp
