/*
 * xpress.h -- C ABI of the xPress refine + verify hot path on MI355X (gfx950).
 *
 * The path (paper sections 3.1 and 4):
 *   base readout   s_k = W_lm h_k                         (section 4.1, Fig. 2a)
 *   seed           Y0_k = select(s_k)                      (Algorithm 1, first step)
 *   K Jacobi passes of the refiner, each one
 *     Fuse  a_k = W_in [W_h h_k || W_g g || W_e[x_{k-1}]], g = mean_j h_j   (eq. fuse)
 *     Mix   c^(d) = (I + L^(d)) a^(d), L^(d) strictly lower-triangular       (eq. mix)
 *     Trans z_k = c_k + W_2 silu(W_1 c_k)                                      (eq. mlp)
 *     Read + Correct  l_k = s_k + W_r z_k                            (eqs. read, correct)
 *     select y_k = argmax_v l_k (greedy) or inverse-CDF sample of softmax(l_k)
 *     stop at the fixed point Y^(j+1) = Y^(j)             (Algorithm 1, Theorem 1)
 *   verification: greedy longest matching prefix plus bonus token, or
 *     speculative accept/reject with residual resampling (section 3.1)
 *
 * Conventions
 *   - Every pointer argument is a DEVICE pointer unless marked "host".  All
 *     buffers are caller-owned, row-major, densely packed.  Weight buffers
 *     must stay alive and unchanged for the life of the handle.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *     stream).  The host does argument validation only, before any HIP call;
 *     nothing is copied back to the host inside refine or verify.
 *   - A handle is not thread-safe.  Calls on one handle must be ordered on one
 *     stream (the handle's workspace is shared between calls).
 *   - On a non-XP_OK return nothing has been enqueued, except for XP_EHIP,
 *     after which outputs are unspecified.  xp_last_error() names the problem.
 *   - Token ids read from device memory (anchor, seed ids, draft ids, target
 *     ids) that fall outside [0, V) are replaced by 0 and recorded in the
 *     handle's device error word (XP_DEVERR_TOKEN); see xp_device_errors().
 */
#ifndef XPRESS_H
#define XPRESS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  XP_OK = 0,
  XP_EINVAL = -1,        /* bad argument (null pointer, size, flag combination)  */
  XP_EUNSUPPORTED = -2,  /* valid per the paper but not built here (e.g. r != 256) */
  XP_EHIP = -3,          /* a HIP runtime call failed                              */
  XP_ENOMEM = -4         /* device allocation of the workspace failed              */
} xp_status;

typedef enum { XP_F32 = 0, XP_BF16 = 1 } xp_dtype;

/* flags of xp_refine_block */
#define XP_EARLY_EXIT   1u  /* skip the remaining passes once every sequence is at its fixed point */
#define XP_WRITE_LOGITS 2u  /* write the refined logits l of the last executed pass to out_logits   */

/* bits of the device error word */
#define XP_DEVERR_TOKEN 1u  /* a token id outside [0, V) was read and replaced by 0 */
#define XP_DEVERR_TEMPERATURE 2u  /* a sampled row's temperature was not finite and > 0; 1 was used */
#define XP_DEVERR_FILTER 4u       /* a sampled row's top_k < 0 or top_p <= 0 (or NaN); not applied */

typedef struct xp_handle xp_handle;

/*
 * Weights (device pointers, element type `dtype`, row-major).  The paper's
 * shapes (section 4.1) with rows as output units:
 *   W_lm [V][H]   target LM head (base readout s_k = W_lm h_k)
 *   W_h  [r][H]   down-projection of h_k
 *   W_g  [r][H]   down-projection of g
 *   W_e  [V][r]   token embedding, one row per token (the paper's r x V W_e, transposed)
 *   W_in [r][3r]  fusion projection; column blocks [h | g | token] in eq. fuse order
 *   L    [r][B][B] per-channel mixer; entry [d][k][i] is read only for i < k
 *   W_1  [2r][r], W_2 [r][2r]   r-space MLP of eq. mlp
 *   W_r  [V][r]   readout head
 * Built: r = 256 (the paper's rank); H a multiple of 256, up to 8192 for bf16
 * and up to 4096 for fp32; 1 <= B <= 32; 16 <= V <= 262144 (the temperature
 * sampler scans at most 4096 vocabulary units of at most 8 tiles of 16 rows
 * on 256 CUs).  xp_create returns XP_EUNSUPPORTED outside these.
 */
typedef struct {
  int32_t H, r, V, B;
  int32_t dtype;                     /* xp_dtype */
  const void* W_lm;
  const void* W_h;
  const void* W_g;
  const void* W_e;
  const void* W_in;
  const void* L;
  const void* W_1;
  const void* W_2;
  const void* W_r;
} xp_weights;

/*
 * Create a handle for one weight set on the current HIP device.
 * Allocates the workspace for up to `max_batch` sequences (device memory, freed
 * by xp_destroy) and precomputes, once, weight-only products in fp32: the token
 * table T = W_e W_in[:, 2r:3r]^T ([V][r]) and the folded down-projections
 * W_in[:, 0:r] W_h and W_in[:, r:2r] W_g ([r][H] each); L is repacked to its
 * strictly lower part.  Synchronous (returns after the precompute finished).
 * Errors: XP_EINVAL (null, sizes), XP_EUNSUPPORTED (r != 256, H, B, dtype),
 * XP_ENOMEM, XP_EHIP.  *out is NULL on error.
 */
xp_status xp_create(const xp_weights* w, int32_t max_batch, xp_handle** out);

/*
 * The Toeplitz mixer (remark after Proposition 1, section 3): when L^(d)_{k,j}
 * depends only on the offset k - j, Mix is a causal depthwise conv1d of kernel
 * size B with taps [1, kappa_d[1], ..., kappa_d[B-1]].  Writes the full mixer
 *   L_out[d][k][j] = kappa[d][k - j] for j < k, 0 for j >= k
 * ([r][B][B], element type `dtype`, row-major) from
 *   kappa [r][B] (kappa[d][0] is never read: lag 0 is the identity of eq. mix)
 * for use as xp_weights.L, so a handle created from it runs the conv1d form.
 * Both are device pointers owned by the caller; L_out must not overlap kappa.
 * Asynchronous on `stream` (NULL = the default stream); no allocation.
 * Errors: XP_EINVAL (null pointer, r outside [1, 65536], B outside [1, 32],
 * unknown dtype), before any HIP call; XP_EHIP if the launch fails.
 */
xp_status xp_toeplitz_mixer(const void* kappa, int32_t r, int32_t B, int32_t dtype, void* L_out,
                            void* stream);

/* Free the handle and its workspace.  Waits for the device first.  NULL is a no-op. */
void xp_destroy(xp_handle* h);

/* Message for the last error on `h` (or of the last failed xp_create when h is NULL). */
const char* xp_last_error(const xp_handle* h);

/* Name of a status code. */
const char* xp_status_string(xp_status s);

/*
 * Refine a batch of draft blocks: base readout, seed, K Jacobi passes.
 *
 *   batch      number of sequences, 1 <= batch <= max_batch
 *   hidden     [batch][B][H] dtype     drafter hidden states h_{1:B}
 *   anchor     [batch] int32           x_0, the token before the block
 *   seed_ids   [batch][B] int32 or NULL  Y^(0); NULL: select from the base logits
 *   temp       [batch] uint8 or NULL   per sequence 0 = greedy (argmax, ties to the
 *              lowest index), nonzero = sampling; NULL = all greedy
 *   temperature [batch] float or NULL  the temperature T > 0 of each sampled
 *              sequence: it samples softmax(l / T) (greedy rows ignore it);
 *              NULL = 1 for every sampled row.  A value that is not finite and
 *              positive is replaced by 1 and sets XP_DEVERR_TEMPERATURE.
 *   top_k      [batch] int32 or NULL; top_p [batch] float or NULL: truncated
 *              sampling of each sampled sequence (seed, every pass, and the
 *              verification that follows): top-k keeps the tokens whose
 *              scaled logit l / T is at least the k-th largest (ties with it
 *              stay); top-p then keeps, of those ordered by logit descending
 *              (ties: lower index first), the shortest prefix whose softmax
 *              mass reaches p of theirs; sampling is from the kept tokens,
 *              renormalised.  k = 0 or k >= V and p >= 1 mean none; k < 0,
 *              p <= 0 or NaN set XP_DEVERR_FILTER and mean none.  Greedy rows
 *              ignore both.  Requires temp.  With either array given, every
 *              pass also writes its logits [batch][B][V] to the workspace
 *              (the truncation needs the whole row).
 *   u_draft    [batch][B] float in [0,1), required iff temp != NULL: the uniform of
 *              each position; a sampled position takes the smallest v whose
 *              cumulative softmax mass exceeds u (fixed across passes)
 *   K          number of Jacobi passes, 0 <= K <= 64 (K = 0 returns Y^(0))
 *   flags      XP_EARLY_EXIT | XP_WRITE_LOGITS
 *   out_ids    [batch][B] int32        refined block
 *   out_iters  [batch] int32 or NULL   passes until Y^(j+1) = Y^(j) held (K if never)
 *   out_logits [batch][B][V] float, required iff XP_WRITE_LOGITS: l of the last
 *              executed pass (s when K = 0)
 *   out_traj   [K+1][batch][B] int32 or NULL: Y^(0) .. Y^(K) (a skipped pass
 *              repeats the previous iterate)
 * The refined distributions of the last pass stay in the handle for a following
 * xp_verify_block on the same stream, until the next xp_refine_block.
 */
xp_status xp_refine_block(xp_handle* h, int32_t batch,
                          const void* hidden, const int32_t* anchor,
                          const int32_t* seed_ids, const uint8_t* temp,
                          const float* temperature,
                          const int32_t* top_k, const float* top_p,
                          const float* u_draft, int32_t K, uint32_t flags,
                          int32_t* out_ids, int32_t* out_iters,
                          float* out_logits, int32_t* out_traj, void* stream);

/*
 * Verify refined blocks against the target (section 3.1).
 *
 *   batch          must equal the batch of the preceding xp_refine_block
 *   draft_ids      [batch][B] int32, the block being verified (normally out_ids)
 *   temp           [batch] uint8 or NULL, as given to that refine
 *   target_ids     [batch][B+1] int32: greedy rows' target tokens t_1..t_{B+1}
 *                  (t_k is the target's choice after the draft prefix y_{<k});
 *                  always required (only greedy rows read it)
 *   target_logits  [batch][B+1][V] float: sampled rows' target logits after each
 *                  prefix; required iff temp != NULL
 *   r_accept       [batch][B] float in [0,1), required iff temp != NULL
 *   u_resample     [batch] float in [0,1), required iff temp != NULL
 *   out_accept_len [batch] int32 n in [0, B] (the paper's tau counts n + 1)
 *   out_next_token [batch] int32 correction token at the first rejection, or
 *                  the bonus token when all B are accepted
 * Greedy rows: n = longest prefix with y_i = t_i, next = t_{n+1}.
 * Sampled rows: accept y_k iff r_k q_k(y_k) <= p_k(y_k), q_k the refined
 * distribution of refine's last pass and p_k = softmax(target logits k / T),
 * T the row's temperature given to that refine (section 3.1 at T > 0), both
 * truncated by that refine's top_k / top_p (so the emitted tokens follow the
 * truncated target distribution); at the
 * first rejection next is the inverse-CDF sample at u_resample of max(0, p_k - q_k)
 * (of p_k if that has no mass); if all are accepted next samples p_{B+1}.
 */
xp_status xp_verify_block(xp_handle* h, int32_t batch,
                          const int32_t* draft_ids, const uint8_t* temp,
                          const int32_t* target_ids, const float* target_logits,
                          const float* r_accept, const float* u_resample,
                          int32_t* out_accept_len, int32_t* out_next_token,
                          void* stream);

/*
 * Stage timing with HIP events, for benchmarks.  While a stage's bit is set in
 * `stage_mask`, every call records one event pair on its stream around that
 * stage's kernels (up to `capacity` pairs per stage; later ones are not
 * recorded).  Stages: XP_STAGE_PREP (g and the static Fuse part), LMHEAD (base
 * readout s = W_lm h), SELECT (token selection of every pass), RSPACE (Fuse
 * gather, Mix, Trans), READ (Read + Correct stream), VERIFY.  A mask of 0
 * disables timing.  xp_timing_read synchronizes the device, writes the summed
 * milliseconds and the number of recorded pairs per stage (host arrays of
 * XP_NSTAGES entries) and clears the record.
 */
typedef enum {
  XP_STAGE_PREP = 0, XP_STAGE_LMHEAD = 1, XP_STAGE_SELECT = 2,
  XP_STAGE_RSPACE = 3, XP_STAGE_READ = 4, XP_STAGE_VERIFY = 5, XP_NSTAGES = 6
} xp_stage;

xp_status xp_timing_enable(xp_handle* h, uint32_t stage_mask, int32_t capacity);
xp_status xp_timing_read(xp_handle* h, float* ms_total, int32_t* pairs);

/*
 * Read and clear the handle's device error word (XP_DEVERR_* bits) into *out
 * (host).  Synchronizes `stream`.
 */
xp_status xp_device_errors(xp_handle* h, uint32_t* out, void* stream);

/*
 * The context layer: one Qwen3-8B-shaped decoder layer over the positions of
 * a drafted block, attending to each sequence's context KV.  The refiner does
 * not read the context (Proposition 1); such layers belong to the drafter and
 * the target (sections 3.1 and 5.1) and produce the hidden states h that the
 * base readout s_k = W_lm h_k (section 4.1) consumes.  Pre-norm, no biases:
 *   u  = RMSNorm(x) g_attn;  q = u Wq^T, k = u Wk^T, v = u Wv^T
 *   q, k: RMSNorm over head_dim per head (g_q, g_k), then rotate-half RoPE at
 *         position ctx_len[b] + i, angle pos * theta^(-2j/head_dim)
 *   attention: query head h reads KV head h / (n_heads / n_kv); scores
 *         q.k / sqrt(head_dim) over the context keys and the block's own keys
 *         (block key j visible to block query i iff j <= i when causal, always
 *         otherwise)
 *   x1 = x + attn Wo^T;  h = x1 + (silu(u2 Wg^T) * (u2 Wu^T)) Wd^T,
 *         u2 = RMSNorm(x1) g_mlp
 * RMSNorm: y = x / sqrt(mean(x^2) + eps) * g.
 *
 * Weights: device pointers, bf16, row-major, rows as output units:
 *   g_attn [H], Wq [n_heads*hd][H], Wk [n_kv*hd][H], Wv [n_kv*hd][H],
 *   g_q [hd], g_k [hd], Wo [H][n_heads*hd], g_mlp [H], Wg [ffn][H],
 *   Wu [ffn][H], Wd [H][ffn]
 * Built: head_dim 128; n_heads / n_kv in {1, 2, 4, 8}; H, n_heads*128 and ffn
 * multiples of 256; H <= 8192.  Every pointer 16-byte aligned (the kernels
 * read and write 16 bytes at a time).
 */
typedef struct {
  int32_t H, n_heads, n_kv, head_dim, ffn;
  float eps;                         /* RMSNorm epsilon (1e-6 for Qwen3) */
  float rope_theta;                  /* RoPE base (1e6 for Qwen3) */
  const void* g_attn;
  const void* Wq;
  const void* Wk;
  const void* Wv;
  const void* g_q;
  const void* g_k;
  const void* Wo;
  const void* g_mlp;
  const void* Wg;
  const void* Wu;
  const void* Wd;
} xp_layer_weights;

typedef struct xp_layer xp_layer;

/*
 * Create a layer for up to max_batch (<= 4096) blocks of up to max_B (<= 32)
 * positions and contexts of up to max_ctx (<= 2^20) keys on the current
 * device; allocates its workspace (freed by xp_layer_destroy).  Any later call
 * with batch <= max_batch and B <= max_B is served by that workspace.  The
 * weights are referenced, not copied: they must stay valid while the layer is
 * used.
 * Errors: XP_EINVAL (null or misaligned pointers, sizes), XP_EUNSUPPORTED
 * (shapes outside the built set, or max_batch * max_B * max(H, n_heads*128,
 * ffn) >= 2^31), XP_ENOMEM, XP_EHIP.  *out is NULL on error;
 * xp_layer_last_error(NULL) names the problem.
 */
xp_status xp_layer_create(const xp_layer_weights* w, int32_t max_batch, int32_t max_B,
                          int32_t max_ctx, xp_layer** out);

/*
 * One forward of the layer over `batch` blocks of B positions, asynchronous on
 * `stream`.  Device pointers:
 *   x        [batch][B][H] bf16   the block's input hidden states
 *   k_cache  [batch][C_max][n_kv][128] bf16  context keys (already normed and
 *            rotated, as a KV cache holds them); v_cache the same for values
 *   ctx_len  [batch] int32 in [0, C_max]: keys [0, ctx_len[b]) of sequence b
 *            are read, the rest never (values outside are clamped)
 *   h_f32    [batch][B][H] fp32 or NULL; h_bf16 [batch][B][H] bf16 or NULL:
 *            the layer output (h_bf16 is the input of the base readout)
 * causal: 1 = block key j visible to block query i iff j <= i; 0 = every block
 * key visible (the drafter's bidirectional block).
 * Calls on one layer share its workspace: issue them in stream order (one
 * stream, or streams synchronized between calls).
 * Every pointer 16-byte aligned.
 * Errors: XP_EINVAL (null handle or input, a misaligned pointer, batch, B or
 * C_max outside what the layer was created for), before any launch; XP_EHIP
 * if a launch fails (kernels already enqueued stay enqueued; h is then
 * unspecified).  xp_layer_last_error(L) names the problem.
 */
xp_status xp_layer_forward(xp_layer* L, int32_t batch, int32_t B, int32_t causal, const void* x,
                           const void* k_cache, const void* v_cache, int32_t C_max,
                           const int32_t* ctx_len, float* h_f32, void* h_bf16, void* stream);

/* Free the layer and its workspace (waits for the device first).  NULL is a no-op. */
void xp_layer_destroy(xp_layer* L);

/* Message for the last failed call on `L` (when L is NULL: of the last failed
 * xp_layer_create or xp_layer_forward_noalloc on this thread); "" if none
 * failed. */
const char* xp_layer_last_error(const xp_layer* L);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * forward as xp_layer_forward, without a layer handle and without any
 * allocation.  `w` is the weight set (as for xp_layer_create; only read
 * during the call); every other argument is as for xp_layer_forward.
 *
 * The intermediates live in a static device array of 64 MiB that every GPU
 * the library runs on holds until the process ends; its address is looked up
 * on the first call on each device.  Calls on one GPU share that array and it
 * keeps the last call's contents: calls that overlap in time on one GPU (two
 * streams, or two host threads) race and give undefined results; calls
 * ordered on one stream are safe.  Output equals xp_layer_forward's bit for
 * bit for calls of up to 64 positions whose attention partials fit beside
 * the other buffers at the default chunking.  Otherwise only the fp32
 * summation order differs: the context may be read in longer chunks (fewer
 * partials), and above 64 positions the projections run without the k
 * splits that xp_layer_forward may use.
 *
 * Limits: batch * B positions whose buffers (about 124 KB per position at
 * the Qwen3-8B shape, plus 1.5 MB of gate/up rows) fit in the array with at
 * least one attention partial per (sequence, position block, KV head, query
 * head); calls beyond that return XP_EINVAL before any HIP call.
 * Errors: XP_EINVAL (weights or arguments as for xp_layer_create and
 * xp_layer_forward, sizes beyond the array), XP_EUNSUPPORTED (shapes outside
 * the built set), before any HIP call; XP_EHIP if the address lookup or a
 * launch fails.  xp_layer_last_error(NULL) names the problem.
 */
xp_status xp_layer_forward_noalloc(const xp_layer_weights* w, int32_t batch, int32_t B,
                                   int32_t causal, const void* x, const void* k_cache,
                                   const void* v_cache, int32_t C_max, const int32_t* ctx_len,
                                   float* h_f32, void* h_bf16, void* stream);

/*
 * Measurement probes (not part of the method).  They give the measured peaks
 * that roofline fractions are also quoted against: the paper reports its
 * kernels' time on its own hardware (evaluation section, latency table), and a
 * fraction of a published peak says little without the attainable one.
 *
 * xp_probe_hbm_read: streams `bytes` (a multiple of 16) of the device buffer
 * `buf` (16-byte aligned) once with 16-byte non-temporal loads, `workgroups`
 * workgroups of 256 threads each taking a contiguous range, and writes the sum of its
 * 32-bit words modulo 2^32 to the device word *out_sum (cleared first by the
 * call).  Bandwidth = bytes / the launch's duration.
 *
 * xp_probe_mfma_bf16: `workgroups` workgroups of 4 waves; every wave runs 8
 * independent accumulator chains of `iters` v_mfma_f32_32x32x16_bf16
 * operations, chain j on the register operands operands[j][lane][0] (A, 16
 * bytes: 8 bf16 of row lane % 32, k = 8 (lane / 32) .. + 8) and
 * operands[j][lane][1] (B, the same for column lane % 32), i.e. a device
 * array of 8 x 64 x 2 x 16 bytes.  Wave w (global index) writes the sum of its
 * 8 accumulators to out[w][lane][16] (fp32; element i of lane l is
 * D[8 (i / 4) + 4 (l / 32) + i % 4][l % 32]), so out must hold workgroups x 4
 * x 64 x 16 floats.  Work = workgroups x 4 x iters x 8 x 32768 flops.
 *
 * Both return XP_EINVAL for null or misaligned pointers and out-of-range
 * sizes, before any HIP call, and XP_EHIP if the launch fails.
 */
xp_status xp_probe_hbm_read(const void* buf, size_t bytes, uint32_t* out_sum, int32_t workgroups,
                            void* stream);
xp_status xp_probe_mfma_bf16(const void* operands, int32_t workgroups, int32_t iters, float* out,
                             void* stream);

#ifdef __cplusplus
}
#endif

#endif /* XPRESS_H */
