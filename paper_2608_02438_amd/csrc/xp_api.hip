// C ABI of the refine + verify path: argument validation, the handle and its
// workspace, and the launch sequence of one call.  No arithmetic of the method
// runs on the host.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <new>
#include <string>

#include "xp_internal.h"

namespace xp {
bool lm_split_ok(int H, int dtype);

__global__ void k_clear_err(uint32_t* err) {
  if (threadIdx.x == 0) *err = 0u;
}

}  // namespace xp

using namespace xp;

static thread_local std::string g_create_err;

static xp_status fail(xp_handle* h, xp_status s, const char* fmt, ...) __attribute__((format(printf, 3, 4)));
static xp_status fail(xp_handle* h, xp_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (h)
    h->err = buf;
  else
    g_create_err = buf;
  return s;
}

static size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

static void timing_free(xp_handle* h);

extern "C" const char* xp_status_string(xp_status s) {
  switch (s) {
    case XP_OK: return "XP_OK";
    case XP_EINVAL: return "XP_EINVAL";
    case XP_EUNSUPPORTED: return "XP_EUNSUPPORTED";
    case XP_EHIP: return "XP_EHIP";
    case XP_ENOMEM: return "XP_ENOMEM";
  }
  return "XP_UNKNOWN";
}

extern "C" const char* xp_last_error(const xp_handle* h) {
  return h ? h->err.c_str() : g_create_err.c_str();
}

extern "C" xp_status xp_create(const xp_weights* w, int32_t max_batch, xp_handle** out) {
  g_create_err.clear();
  if (!out) return fail(nullptr, XP_EINVAL, "out is NULL");
  *out = nullptr;
  if (!w) return fail(nullptr, XP_EINVAL, "weights is NULL");
  if (w->dtype != XP_F32 && w->dtype != XP_BF16)
    return fail(nullptr, XP_EINVAL, "dtype %d is not XP_F32 or XP_BF16", w->dtype);
  const void* ptrs[] = {w->W_lm, w->W_h, w->W_g, w->W_e, w->W_in, w->L, w->W_1, w->W_2, w->W_r};
  const char* names[] = {"W_lm", "W_h", "W_g", "W_e", "W_in", "L", "W_1", "W_2", "W_r"};
  for (int i = 0; i < 9; ++i)
    if (!ptrs[i]) return fail(nullptr, XP_EINVAL, "weight %s is NULL", names[i]);
  if (w->r <= 0 || w->H <= 0 || w->V <= 0 || w->B <= 0)
    return fail(nullptr, XP_EINVAL, "sizes must be positive (H=%d r=%d V=%d B=%d)", w->H, w->r,
                w->V, w->B);
  if (w->r != 256) return fail(nullptr, XP_EUNSUPPORTED, "r=%d: only r=256 is built", w->r);
  if (w->V < 16) return fail(nullptr, XP_EUNSUPPORTED, "V=%d: vocabularies below 16 are not built", w->V);
  if (w->B > 32) return fail(nullptr, XP_EUNSUPPORTED, "B=%d: blocks up to 32 are built", w->B);
  if (w->H % 256 != 0 || !lm_split_ok(w->H, w->dtype) ||
      (w->dtype == XP_F32 ? w->H > 4096 : w->H > 8192))
    return fail(nullptr, XP_EUNSUPPORTED,
                "H=%d: H must be a multiple of 256, at most 8192 (bf16) or 4096 (fp32)", w->H);
  if (max_batch < 1 || (int64_t)max_batch * w->B > 65536)
    return fail(nullptr, XP_EINVAL, "max_batch=%d out of range (1 .. 65536/B)", max_batch);

  xp_handle* h = new (std::nothrow) xp_handle();
  if (!h) return fail(nullptr, XP_ENOMEM, "host allocation failed");
  h->H = w->H;
  h->r = w->r;
  h->V = w->V;
  h->B = w->B;
  h->dtype = w->dtype;
  h->max_batch = max_batch;
  h->W_lm = w->W_lm;
  h->W_h = w->W_h;
  h->W_g = w->W_g;
  h->W_e = w->W_e;
  h->W_in = w->W_in;
  h->L = w->L;
  h->W_1 = w->W_1;
  h->W_2 = w->W_2;
  h->W_r = w->W_r;
  h->ldS = (w->V + 15) / 16 * 16;
  h->ntiles = h->ldS / 16;

  hipError_t e = hipGetDevice(&h->device);
  int cus = 0;
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device);
  if (e != hipSuccess) {
    delete h;
    return fail(nullptr, XP_EHIP, "device query failed: %s", hipGetErrorString(e));
  }
  h->cus = cus > 0 ? cus : 256;
  h->lm_chunks = h->ntiles < h->cus ? h->ntiles : h->cus;
  const int rw = (h->ntiles + kReadWaves - 1) / kReadWaves;
  h->read_wgs = rw < h->cus ? rw : h->cus;
  h->read_units = h->read_wgs * kReadWaves;
  // the temperature-1 selection scans at most 4096 units per position and
  // rescans Read units of at most 8 tiles
  if (h->read_units > 4096 || gemm_units_max(h) > 4096 || h->lm_chunks > 4096 ||
      (h->ntiles + h->read_units - 1) / h->read_units > 8) {
    const int V = w->V;
    delete h;
    return fail(nullptr, XP_EUNSUPPORTED, "V=%d: vocabularies above %d rows are not built", V,
                8 * 16 * 8 * 256);
  }

  // workspace layout: one allocation, 256-byte aligned slices
  const size_t es = w->dtype == XP_BF16 ? 2 : 4;
  const size_t Mmax = (size_t)max_batch * w->B;
  const size_t npairs = (size_t)w->B * (w->B - 1) / 2;
  size_t nk = (size_t)(h->lm_chunks > h->read_wgs ? h->lm_chunks : h->read_wgs);
  size_t nu = (size_t)(h->lm_chunks > h->read_units ? h->lm_chunks : h->read_units);
  const size_t ng = (size_t)gemm_units_max(h);          // the finest GEMM unit partition
  nk = nk > ng ? nk : ng;
  nu = nu > ng ? nu : ng;
  struct Slice {
    void** dst;
    size_t bytes;
  };
  Workspace& ws = h->ws;
  Slice sl[] = {
      {(void**)&ws.s, Mmax * h->ldS * 4},
      {(void**)&ws.T, (size_t)w->V * 256 * 4},
      {(void**)&ws.Fh, (size_t)256 * w->H * 4},
      {(void**)&ws.Fg, (size_t)256 * w->H * 4},
      {(void**)&ws.Lp, (npairs ? npairs : 1) * 256 * es},
      {(void**)&ws.ppart, (size_t)2 * prep_ksp(w->H) * Mmax * 256 * 4},
      {(void**)&ws.Pa, Mmax * 256 * 4},
      {(void**)&ws.c, Mmax * 256 * 4},
      {(void**)&ws.h1, Mmax * 512 * 4},
      {(void**)&ws.z, Mmax * 256 * es},
      {(void**)&ws.Y[0], Mmax * 4},
      {(void**)&ws.Y[1], Mmax * 4},
      {(void**)&ws.keys, nk * Mmax * 8},
      {(void**)&ws.stats, nu * Mmax * sizeof(Stat)},
      {(void**)&ws.lse, Mmax * 8},
      {(void**)&ws.invT, (size_t)max_batch * 4},
      {(void**)&ws.iters, (size_t)max_batch * 4},
      {(void**)&ws.ctrl, 16},
      {(void**)&ws.err, 16},
      {(void**)&ws.vstat, (size_t)max_batch * (w->B + 1) * 8},
      {(void**)&ws.vpos, (size_t)max_batch * 4},
      {(void**)&ws.vmass, (size_t)h->read_units * max_batch * 16},
      {(void**)&ws.vpart,
       (size_t)max_batch * (w->B + 1) * ((w->V + kVChunk - 1) / kVChunk) * 16},
      {(void**)&ws.lf, Mmax * w->V * 4},
      {(void**)&ws.fst, Mmax * sizeof(FState)},
      {(void**)&ws.tst, (size_t)max_batch * (w->B + 1) * sizeof(FState)},
      {(void**)&ws.filt, (size_t)max_batch},
      {(void**)&ws.temp_nf, (size_t)max_batch},
      {(void**)&ws.fk, (size_t)max_batch * 4},
      {(void**)&ws.fp, (size_t)max_batch * 4},
  };
  size_t total = 0;
  for (auto& s : sl) total += align_up(s.bytes, 256);
  char* base = nullptr;
  e = hipMalloc((void**)&base, total);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    delete h;
    return fail(nullptr, XP_ENOMEM, "workspace of %zu bytes: %s", total, hipGetErrorString(e));
  }
  size_t off = 0;
  for (auto& s : sl) {
    *s.dst = base + off;
    off += align_up(s.bytes, 256);
  }
  e = launch_fold(h, nullptr);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(k_clear_err, dim3(1), dim3(64), 0, nullptr, ws.err);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
  if (e != hipSuccess) {
    (void)hipFree(base);
    delete h;
    return fail(nullptr, XP_EHIP, "weight precompute failed: %s", hipGetErrorString(e));
  }
  *out = h;
  return XP_OK;
}

extern "C" void xp_destroy(xp_handle* h) {
  if (!h) return;
  (void)hipDeviceSynchronize();
  timing_free(h);
  (void)hipFree(h->ws.s);   // first slice = base of the allocation
  delete h;
}

#define XP_LAUNCH(call)                                                              \
  do {                                                                               \
    hipError_t e_ = (call);                                                          \
    if (e_ != hipSuccess)                                                            \
      return fail(h, XP_EHIP, "%s failed: %s", #call, hipGetErrorString(e_));        \
  } while (0)

// Event pair around one stage's launches when timing is on for that stage.
struct StageTimer {
  xp_handle* h;
  int stage;
  hipStream_t st;
  bool on;
  StageTimer(xp_handle* h_, int stage_, hipStream_t st_) : h(h_), stage(stage_), st(st_) {
    xp_timing_state& t = h->tm;
    on = (t.mask >> stage) & 1u && t.n[stage] < t.capacity;
    if (on) (void)hipEventRecord(t.ev[stage][2 * t.n[stage]], st);
  }
  ~StageTimer() {
    if (!on) return;
    xp_timing_state& t = h->tm;
    (void)hipEventRecord(t.ev[stage][2 * t.n[stage] + 1], st);
    ++t.n[stage];
  }
};

#define XP_TIMED(stage, call)                 \
  do {                                        \
    StageTimer tm_(h, (stage), st);           \
    XP_LAUNCH(call);                          \
  } while (0)

static void timing_free(xp_handle* h) {
  for (auto& v : h->tm.ev) {
    for (hipEvent_t e : v) (void)hipEventDestroy(e);
    v.clear();
  }
  h->tm = xp_timing_state();
}

extern "C" xp_status xp_timing_enable(xp_handle* h, uint32_t stage_mask, int32_t capacity) {
  if (!h) return XP_EINVAL;
  if (stage_mask >> XP_NSTAGES) return fail(h, XP_EINVAL, "unknown stage bits 0x%x", stage_mask);
  if (stage_mask && (capacity < 1 || capacity > (1 << 20)))
    return fail(h, XP_EINVAL, "capacity=%d out of range 1..2^20", capacity);
  XP_LAUNCH(hipDeviceSynchronize());
  timing_free(h);
  if (!stage_mask) return XP_OK;
  for (int s = 0; s < XP_NSTAGES; ++s) {
    if (!((stage_mask >> s) & 1u)) continue;
    h->tm.ev[s].resize(2 * (size_t)capacity);
    for (auto& e : h->tm.ev[s]) {
      hipError_t r = hipEventCreate(&e);
      if (r != hipSuccess) {
        e = nullptr;
        timing_free(h);
        return fail(h, XP_EHIP, "hipEventCreate: %s", hipGetErrorString(r));
      }
    }
  }
  h->tm.mask = stage_mask;
  h->tm.capacity = capacity;
  return XP_OK;
}

extern "C" xp_status xp_timing_read(xp_handle* h, float* ms_total, int32_t* pairs) {
  if (!h || !ms_total || !pairs) return XP_EINVAL;
  XP_LAUNCH(hipDeviceSynchronize());
  for (int s = 0; s < XP_NSTAGES; ++s) {
    float tot = 0.f;
    for (int i = 0; i < h->tm.n[s]; ++i) {
      float ms = 0.f;
      XP_LAUNCH(hipEventElapsedTime(&ms, h->tm.ev[s][2 * i], h->tm.ev[s][2 * i + 1]));
      tot += ms;
    }
    ms_total[s] = tot;
    pairs[s] = h->tm.n[s];
    h->tm.n[s] = 0;
  }
  return XP_OK;
}

extern "C" xp_status xp_refine_block(xp_handle* h, int32_t batch, const void* hidden,
                                     const int32_t* anchor, const int32_t* seed_ids,
                                     const uint8_t* temp, const float* temperature,
                                     const int32_t* top_k, const float* top_p,
                                     const float* u_draft, int32_t K,
                                     uint32_t flags, int32_t* out_ids, int32_t* out_iters,
                                     float* out_logits, int32_t* out_traj, void* stream) {
  if (!h) return XP_EINVAL;
  if (batch < 1 || batch > h->max_batch)
    return fail(h, XP_EINVAL, "batch=%d out of range 1..%d", batch, h->max_batch);
  if (!hidden || !anchor || !out_ids)
    return fail(h, XP_EINVAL, "hidden, anchor and out_ids are required");
  if (K < 0 || K > kMaxK) return fail(h, XP_EINVAL, "K=%d out of range 0..%d", K, kMaxK);
  if (flags & ~(XP_EARLY_EXIT | XP_WRITE_LOGITS))
    return fail(h, XP_EINVAL, "unknown flag bits 0x%x", flags);
  if (temp && !u_draft) return fail(h, XP_EINVAL, "u_draft is required when temp is given");
  if ((top_k || top_p) && !temp)
    return fail(h, XP_EINVAL, "top_k / top_p apply to sampled rows: temp is required");
  if ((flags & XP_WRITE_LOGITS) && !out_logits)
    return fail(h, XP_EINVAL, "XP_WRITE_LOGITS needs out_logits");
  if (!(flags & XP_WRITE_LOGITS) && out_logits)
    return fail(h, XP_EINVAL, "out_logits given without XP_WRITE_LOGITS");
  hipStream_t st = (hipStream_t)stream;
  h->state_valid = false;
  h->call_tempered = temp != nullptr && temperature != nullptr;
  const bool filtering = temp != nullptr && (top_k != nullptr || top_p != nullptr);
  // All-greedy batches run the selection of pass j-1, Fuse, Mix and the first
  // Trans product of pass j as one kernel; the others use separate kernels.
  XP_TIMED(XP_STAGE_PREP, launch_prep(h, batch, hidden, temp, temperature, st));
  if (filtering) XP_TIMED(XP_STAGE_PREP, launch_filter_params(h, batch, temp, top_k, top_p, st));
  XP_TIMED(XP_STAGE_LMHEAD, launch_lmhead(h, batch * h->B, hidden, temp, st));
  const bool fused = K > 0 && pass_fused_ok(h, temp);
  if (!fused)
    XP_TIMED(XP_STAGE_SELECT,
             launch_select(h, batch, -1, K, flags, seed_ids, temp, u_draft, out_traj,
                           K == 0 ? out_ids : nullptr, K == 0 ? out_iters : nullptr, st,
                           filtering));
  for (int j = 0; j < K; ++j) {
    if (fused) XP_TIMED(XP_STAGE_RSPACE, launch_pass(h, batch, j, flags, seed_ids, anchor, out_traj, st));
    XP_TIMED(XP_STAGE_RSPACE, launch_rspace(h, batch, j, flags, anchor, !fused, st));
    float* lout = filtering ? h->ws.lf : ((flags & XP_WRITE_LOGITS) ? out_logits : nullptr);
    XP_TIMED(XP_STAGE_READ, launch_read(h, batch, j, flags, temp, lout, st));
    const bool lastp = j == K - 1;
    if (!fused || lastp)
      XP_TIMED(XP_STAGE_SELECT,
               launch_select(h, batch, j, K, flags, nullptr, temp, u_draft, out_traj,
                             lastp ? out_ids : nullptr, lastp ? out_iters : nullptr, st,
                             filtering));
  }
  XP_LAUNCH(launch_finish(h, batch, K, flags, out_ids, out_iters, out_logits, st, filtering));
  h->last_batch = batch;
  h->state_k0 = (K == 0);
  h->state_temp = temp != nullptr;
  h->state_filtered = filtering;
  h->state_valid = true;
  return XP_OK;
}

extern "C" xp_status xp_verify_block(xp_handle* h, int32_t batch, const int32_t* draft_ids,
                                     const uint8_t* temp, const int32_t* target_ids,
                                     const float* target_logits, const float* r_accept,
                                     const float* u_resample, int32_t* out_accept_len,
                                     int32_t* out_next_token, void* stream) {
  if (!h) return XP_EINVAL;
  if (!h->state_valid)
    return fail(h, XP_EINVAL, "verify needs a preceding xp_refine_block on this handle");
  if (batch != h->last_batch)
    return fail(h, XP_EINVAL, "batch=%d differs from the refined batch %d", batch, h->last_batch);
  if (!draft_ids || !target_ids || !out_accept_len || !out_next_token)
    return fail(h, XP_EINVAL, "draft_ids, target_ids and both outputs are required");
  if (temp && !h->state_temp)
    return fail(h, XP_EINVAL, "temp given to verify but not to the preceding refine");
  if (temp && (!target_logits || !r_accept || !u_resample))
    return fail(h, XP_EINVAL, "sampled rows need target_logits, r_accept and u_resample");
  hipStream_t st = (hipStream_t)stream;
  XP_TIMED(XP_STAGE_VERIFY, launch_verify(h, batch, draft_ids, temp, target_ids, target_logits,
                                          r_accept, u_resample, out_accept_len, out_next_token,
                                          st));
  return XP_OK;
}

extern "C" xp_status xp_device_errors(xp_handle* h, uint32_t* out, void* stream) {
  if (!h || !out) return XP_EINVAL;
  hipStream_t st = (hipStream_t)stream;
  XP_LAUNCH(hipMemcpyAsync(out, h->ws.err, 4, hipMemcpyDeviceToHost, st));
  XP_LAUNCH(hipStreamSynchronize(st));
  hipLaunchKernelGGL(k_clear_err, dim3(1), dim3(64), 0, st, h->ws.err);
  XP_LAUNCH(hipGetLastError());
  return XP_OK;
}
