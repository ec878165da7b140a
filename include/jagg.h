/*
 * JAGG group backward on one MI355X (gfx950) — C ABI.
 *
 * The library computes the parameter gradient of a DiT/MMDiT velocity network
 * over a window of W consecutive denoising steps in two ways:
 *
 *   JAGG:     g = J_0^T s_base + J_{W-1}^T s_corr, one backward pass over the
 *             batched endpoint pair (paper: JAGG, Phases 3 and 4; the
 *             Corollary of Theorem 1), with
 *             alpha_j = (t_0 - t_j) / (t_0 - t_{W-1})            (Eq. alpha)
 *             s_base = sum_j (1 - alpha_j) s_j, s_corr = sum_j alpha_j s_j
 *                                                      (Eq. s_base / s_corr)
 *   per step: g = sum_j J_j^T s_j, one backward per step   (the exact baseline
 *             with the same detach of z_j, Phase 2 remark)
 *
 * where J(z, t) = d v_theta(z, t) / d theta and s_j = dL_j / d v_j is the
 * per-step upstream gradient on the velocity output (given as input).
 *
 * Conventions for every call:
 *  - Status codes: 0 OK; 1 invalid argument (detected before any launch);
 *    2 out of memory; 3 device/launch error; 4 unsupported shape/dtype.
 *    jagg_last_error() returns a thread-local message for the last failure.
 *  - Ownership: the caller owns every buffer (parameters, gradients, inputs,
 *    saved activations, workspace).  The library never allocates device memory
 *    in these calls and never frees a caller pointer.  Pointers named "device"
 *    are device memory; "host" pointers are read before the call returns.
 *  - Streams: device work is enqueued on the context's HIP stream and the call
 *    returns without synchronising; results are valid after that stream is
 *    synchronised.  Calls on one context must not overlap from two threads.
 *  - Dtypes: JAGG_F32 or JAGG_BF16 (bf16 = raw uint16 bit pattern).  theta,
 *    the inputs, activations and s_j use cfg.act_dtype; dtheta uses
 *    cfg.grad_dtype.  All arithmetic accumulates in fp32.
 *  - Token rows ("stream-major"): for a batch of B samples the text rows of
 *    all samples come first (sample b's text tokens at rows b*n_txt ..), then
 *    the image rows (sample b's image tokens at rows B*n_txt + b*n_img ..).
 *    A block-only model takes and returns its token streams in this layout,
 *    [B*(n_txt+n_img)][hidden]; for B = 1 it is the joint sequence [text; image].
 */
#ifndef JAGG_H
#define JAGG_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { JAGG_OK = 0, JAGG_EINVAL = 1, JAGG_ENOMEM = 2, JAGG_EDEVICE = 3, JAGG_EUNSUPPORTED = 4 } jagg_status;
typedef enum { JAGG_F32 = 0, JAGG_BF16 = 1 } jagg_dtype;

/* Network shape.  The architecture is the MMDiT of the paper's experiments
 * (double-stream blocks with joint attention, then single-stream blocks),
 * written out in the oracle's module docstring: adaLN modulation from a
 * time-embedding MLP, LayerNorm without affine, q/k RMSNorm with a learned
 * gain, 2-D rotary embedding (text tokens at position (0,0)), tanh-GELU MLP.
 * block_only = 1: no patch/text embedding and no final layer; the model maps
 * the token streams (stream-major rows) to the token streams of the last
 * double block (n_single must be 0). */
typedef struct {
  int n_double, n_single;
  int hidden, heads, head_dim, mlp_hidden;
  int in_ch, patch, lat_h, lat_w; /* latent (B, in_ch, lat_h, lat_w); image tokens (lat_h/patch)*(lat_w/patch) */
  int n_txt, txt_dim;
  int t_freq_dim;                  /* sinusoidal timestep embedding width (even) */
  int block_only;
  int act_dtype;                   /* jagg_dtype of theta, inputs, activations, s_j */
  int grad_dtype;                  /* jagg_dtype of dtheta */
  int checkpoint;                  /* 1: save block inputs only, recompute each block in the VJP */
} dit_config;

typedef struct {
  char name[48];     /* e.g. "double.3.img.fc1.w" */
  size_t offset;     /* element offset in the flat theta / dtheta (multiple of 128) */
  size_t numel;
  int rows, cols;    /* weights [out][in]; vectors rows = numel, cols = 1 */
} jagg_tensor_desc;

typedef struct jagg_ctx jagg_ctx;

/* Thread-local message describing the last failure of any call (never NULL). */
const char* jagg_last_error(void);

/* Parameter layout of theta, the parameters of the velocity network
 * v_theta(z, t) whose gradient the method computes (problem statement of the
 * Method section; the block structure is the MMDiT described above).
 * *n_tensors receives the tensor count, *n_elems the flat length (padding
 * between tensors is never read or written).  If out != NULL it receives
 * min(cap, count) descriptors.  Host only; no device needed.  EINVAL on a null
 * pointer or an invalid config. */
jagg_status dit_param_layout(const dit_config* cfg, size_t* n_tensors, size_t* n_elems, jagg_tensor_desc* out,
                             size_t cap);

/* Create a context bound to `hip_stream` (a hipStream_t, or NULL for the null
 * stream) on the current device.  Validates the config.  Host only.  On its
 * first backward the context creates one more stream of its own (default
 * priority) for the double blocks' weight-gradient products; that work is
 * forked from and joined back into `hip_stream` with events inside each call,
 * so every call stays ordered on `hip_stream` alone. */
jagg_status jagg_ctx_create(const dit_config* cfg, void* hip_stream, jagg_ctx** out);
/* Release the context (and its own stream, after that stream's work is done). */
void jagg_ctx_destroy(jagg_ctx* ctx);

/* Bytes of the saved-activation buffer for a forward of `batch` samples, and
 * of the workspace needed by any call on `batch` samples.  Host only. */
jagg_status dit_saved_bytes(const jagg_ctx* ctx, int batch, size_t* bytes);
jagg_status dit_workspace_bytes(const jagg_ctx* ctx, int batch, size_t* bytes);
/* Bind a caller-owned device workspace (kept until replaced or the context is
 * destroyed; the caller frees it).  Calls check that it is large enough. */
jagg_status jagg_ctx_set_workspace(jagg_ctx* ctx, void* ws, size_t bytes);

/* Forward v = v_theta(z, t) for `batch` samples (1 <= batch <= 32).
 *   theta : device, flat parameters (act dtype)
 *   z     : device, latent (batch, in_ch, lat_h, lat_w); block-only: token rows
 *   t     : host, `batch` network-input timesteps
 *   txt   : device, text embeddings (batch, n_txt, txt_dim); NULL for block-only
 *   v_out : device, output with the shape of z
 *   saved : device, dit_saved_bytes(batch) bytes that the VJP reads; NULL runs
 *           without saving (the middle steps of a window: no graph).
 * Paper: JAGG Phase 1 (forward passes, graph only at the endpoints). */
jagg_status dit_forward_save(jagg_ctx* ctx, const void* theta, const void* z, const float* t, const void* txt,
                             void* v_out, void* saved, int batch);

/* Parameter VJP: dtheta = beta * dtheta + J^T s for the forward stored in
 * `saved` (same batch).  s: device, shape of v_out.  beta is 0 (overwrite) or
 * 1 (accumulate); padding entries of dtheta are left untouched.
 * Paper: one transformer backward ("Transformer bwd" column of the cost table). */
jagg_status dit_vjp(jagg_ctx* ctx, const void* theta, const void* saved, int batch, const void* s, void* dtheta,
                    float beta);

/* Eq. alpha on the host: alpha_j = (t_0 - t_j)/(t_0 - t_{W-1}) computed in fp64
 * and rounded to fp32 (alpha_0 = 0 and alpha_{W-1} = 1 exactly).  EINVAL if
 * W < 2, a pointer is NULL or t is not strictly decreasing (a window's steps
 * run from high to low noise; this includes t_0 == t_{W-1}). */
jagg_status jagg_alpha(const float* t, int W, float* alpha_out);

/* Eq. s_base / s_corr on the device: s_base = sum_j (1 - alpha_j) s_j,
 * s_corr = sum_j alpha_j s_j over n elements; fp32 accumulation in j order,
 * one rounding on store.  s: host array of W device pointers; t: host W
 * timesteps, strictly decreasing (the weights come from jagg_alpha).
 * s_base/s_corr: device, n elements of `dtype` (same as the inputs).
 * 2 <= W <= 64. */
jagg_status jagg_aggregate(jagg_ctx* ctx, const void* const* s, const float* t, int W, size_t n, int dtype,
                           void* s_base, void* s_corr);

/* Routing score of one window (high-noise vs low-noise scheduling: a window is
 * routed to JAGG while its score passes the cosine rule of the
 * gradient-quality appendix, cos >= 0.5).  The paper's cosine compares
 * gradients; this call scores any W per-step vectors the caller supplies
 * (per-step gradients, hidden states): the mean over the W(W-1)/2 pairs
 * (i < j) of cos(h_i, h_j) (n elements each, `dtype`), accumulated in fp64 in
 * a fixed order.  h: host array of W device pointers, 2 <= W <= 8.
 * score_out: host, receives the score (the call synchronises the stream).
 * Uses the head of the bound workspace; EINVAL if it is not bound or too
 * small, on a null pointer, n = 0 or an unknown dtype. */
jagg_status jagg_group_scores(jagg_ctx* ctx, const void* const* h, size_t n, int W, int dtype, double* score_out);

/* Allocation-free jagg_group_scores, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation): the same kernels and the same score, with their
 * partial sums in a static device array of the library (147,456 bytes per
 * device, held until the process ends) instead of the bound workspace, which
 * this call does not need.  score_dev: device, one double (8-byte aligned),
 * written on the context's stream; the call does not synchronise.  Calls
 * no allocator.  EINVAL on a null pointer, n = 0, an unknown dtype or W
 * outside 2..8 (W = 8 is the largest the static array holds).  Every call on
 * one device shares that array: calls that overlap on one device (on two
 * streams or threads) race and must be serialised by the caller. */
jagg_status jagg_group_scores_noalloc(jagg_ctx* ctx, const void* const* h, size_t n, int W, int dtype,
                                      double* score_dev);

/* Routing (high-noise vs low-noise scheduling; gradient-quality appendix).
 * Groups are ordered from high to low noise.  frac >= 0: the first
 * floor(frac * n_groups + 1e-6) groups use JAGG (static jagg_frac).  frac < 0:
 * scores (host, n_groups) decide: the longest prefix of groups whose score is
 * >= tau.  use_jagg_out: host, n_groups bytes (1 = JAGG, 0 = per-step);
 * frac_out: host, realised fraction (may be NULL).  Host only, bit-exact. */
jagg_status jagg_route(const double* scores, int n_groups, double tau, double frac, unsigned char* use_jagg_out,
                       double* frac_out);

/* JAGG group backward (Phases 3 and 4): aggregates the W upstream gradients
 * into the composite cotangent of the endpoint pair and runs ONE VJP over the
 * batched pair.  saved_pair: the forward of batch 2B on [z_0; z_{W-1}] with
 * t = [t_0 (B times); t_{W-1} (B times)] (block-only: stream-major rows of the
 * 2B samples, endpoint 0 first within each stream).  s: host array of W device
 * pointers, each with the shape of a batch-B output.  t: host W timesteps.
 * dtheta = beta * dtheta + g_jagg.  2 <= W <= 64. */
jagg_status jagg_group_backward(jagg_ctx* ctx, const void* theta, const void* saved_pair, int batch,
                                const void* const* s, const float* t, int W, void* dtheta, float beta);

/* Sequential-graph JAGG (appendix, sequential-graph variant): the backward of
 * ONE endpoint of the window, so that only that endpoint's saved activations
 * must exist at a time (the caller can run dit_forward_save for z_0, this call
 * with endpoint 0, then dit_forward_save for z_{W-1} into the same buffer and
 * this call with endpoint 1).  endpoint 0: dtheta = beta * dtheta +
 * J_0^T s_base; endpoint 1: dtheta = beta * dtheta + J_{W-1}^T s_corr, with the
 * composites of Eq. s_base / s_corr formed from the W upstream gradients (s:
 * host array of W device pointers, each a batch-B output; t: host W
 * timesteps).  saved: a batch-B forward of z_0 at t_0 (endpoint 0) or of
 * z_{W-1} at t_{W-1} (endpoint 1).  Endpoint 0 then endpoint 1 (beta 1) gives
 * the joint call's gradient up to fp32 summation order.  Workspace:
 * dit_workspace_bytes(batch).  2 <= W <= 64. */
jagg_status jagg_endpoint_backward(jagg_ctx* ctx, const void* theta, const void* saved, int batch, const void* const* s,
                                   const float* t, int W, int endpoint, void* dtheta, float beta);

/* Gradient quality (gradient-quality appendix: cos(g_jagg, g_exact) and the
 * norm ratio rho = |g_jagg| / |g_exact|) of two device vectors a, b of n
 * elements of `dtype` (16-byte aligned).  out (host, 5 doubles): out[0..2] the
 * fp64 sums a.b, a.a, b.b; out[3] = cos = a.b / sqrt(a.a b.b); out[4] = rho =
 * sqrt(a.a / b.b) (NaN where a norm is zero).  Every element of the n is
 * included: flat gradient buffers must hold zeros in their padding.
 * Deterministic (fixed block order).  Uses the head of the bound workspace;
 * synchronises the context's stream. */
jagg_status jagg_grad_compare(jagg_ctx* ctx, const void* a, const void* b, size_t n, int dtype, double* out);

/* Failure detection (no operation of the paper: a guard a caller runs on a
 * gradient before using it): the number of elements of the device vector x
 * (n elements of `dtype`, 16-byte aligned) that are NaN or +-Inf, i.e. whose
 * exponent bits are all ones.  count (host): one unsigned 64-bit value, exact.
 * Flat gradient buffers may be scanned whole: their zero padding counts as
 * finite.  Uses the head of the bound workspace; synchronises the context's
 * stream.  EINVAL for a null pointer, n == 0, an unknown dtype, a misaligned x
 * or a missing or too small workspace, before any launch. */
jagg_status jagg_count_nonfinite(jagg_ctx* ctx, const void* x, size_t n, int dtype, unsigned long long* count);

/* Gradient quality of one window (gradient-quality appendix, per-group
 * cos(g_jagg, g_exact) and rho; the endpoint-only ablation of the
 * experiments): runs the JAGG group backward into g_jagg, the per-step
 * backward into g_exact and the ablation J_0^T s_0 + J_{W-1}^T s_{W-1} (the
 * JAGG pass with the endpoint signals alone, weight one each) into g_ablate,
 * then compares them.  out (host, 4 doubles): cos(g_jagg, g_exact),
 * rho_jagg = |g_jagg| / |g_exact|, cos(g_ablate, g_exact), rho_ablate.
 *   saved_pair: batch-2B forward of the window's endpoint pair; saved_steps:
 *   host array of W device pointers, the batch-B forward of each step; s: host
 *   array of W device pointers; t: host, W timesteps (strictly decreasing);
 *   g_jagg, g_exact, g_ablate: device, dtheta-sized buffers of cfg.grad_dtype
 *   (16-byte aligned; their padding is never written and must hold zeros, so
 *   zero them once before the first call).
 * Workspace: dit_workspace_bytes(2 * batch).  Synchronises the stream. */
jagg_status jagg_window_quality(jagg_ctx* ctx, const void* theta, const void* saved_pair,
                                const void* const* saved_steps, int batch, const void* const* s, const float* t, int W,
                                void* g_jagg, void* g_exact, void* g_ablate, double* out);

/* Phase 2 of JAGG for a GRPO window on rectified flow (GRPO section: Eq.
 * grpo_loss, Eq. logprob and the Euler-step mean; hyperparameter appendix:
 * clip range, advantage clamp).  Per sample b and step j:
 *   mu_j = z_j + v_j (t_{j+1} - t_j)
 *   log pi_j = -|z_{j+1} - mu_j|^2 / (2 sigma_j^2) - n log(sqrt(2 pi) sigma_j)
 *              (n = elements per sample; squared norm over the sample)
 *   rho_j = exp(log pi_j - logp_old[j][b]), A = clamp(adv[b], -adv_clip, adv_clip)
 *   L_j = (1/W) max(-A rho_j, -A clip(rho_j, 1 - clip_eps, 1 + clip_eps))
 *   s_j = dL_j / dv_j = c_j (z_{j+1} - mu_j), c_j = dL_j/drho_j * rho_j *
 *         (t_{j+1} - t_j) / sigma_j^2, with dL_j/drho_j = 0 when the clipped
 *         term is strictly the larger (the PPO-clip remark's zero gradient)
 *         and -A/W otherwise.
 * The squared norms are accumulated in fp64 and the clip decision is taken
 * in fp64; the gradients are formed in fp32.  t_0 .. t_W must be strictly
 * decreasing.  All arrays use the batch-B
 * output layout of the model (block-only: stream-major token rows); every
 * per-sample segment must be a multiple of 8 elements. */
typedef struct {
  const void* const* v_hat; /* host array of W device pointers: model outputs v_j */
  const void* const* z;     /* host array of W+1 device pointers: z_0 .. z_W */
  const float* t;           /* host, W+1 timesteps t_0 .. t_W (t_W: the step after the window) */
  const float* sigma;       /* host, W: sigma_j > 0 */
  const double* logp_old;   /* device, W x batch, [j][b]: log pi_old(z_{j+1} | z_j) */
  const float* adv;         /* device, batch: advantages */
  float clip_eps;           /* PPO clip range (0.1 in the paper's runs) */
  float adv_clip;           /* advantage clamp (5.0 in the paper's runs) */
  int W;                    /* 2..8, 10, 12 or 16 */
  const int* v_batch;       /* host, W, or NULL: v_j holds samples v_index[j] .. v_index[j] + batch - 1 */
  const int* v_index;       /* of a batch-v_batch[j] array in the model's output layout (e.g. the output of */
                            /* the batch-2B endpoint-pair forward or of a batched no-grad middle forward); */
                            /* NULL: every v_j is a batch-B array.  v_batch[j] <= 64. */
} jagg_grpo_window;

/* Phases 2 and 3 fused: the composites s_base, s_corr (Eq. s_base / s_corr with
 * alpha from t_0 .. t_{W-1}) of the window's GRPO upstream gradients, without
 * materialising any s_j.  s_base, s_corr: device, batch-B output layout.
 * stats: device, W x batch x 3 doubles (log pi_j, rho_j, L_j) or NULL.  batch
 * 1..16.  Uses the bound workspace. */
jagg_status jagg_grpo_composites(jagg_ctx* ctx, const jagg_grpo_window* w, int batch, void* s_base, void* s_corr,
                                 double* stats);

/* Phase 2 alone: the W upstream gradients s_j (host array of W device
 * pointers, batch-B output layout), for the per-step baseline. */
jagg_status jagg_grpo_upstream(jagg_ctx* ctx, const jagg_grpo_window* w, int batch, void* const* s_out,
                               double* stats);

/* Phases 2-4: the fused composites written straight into the endpoint pair's
 * cotangent, then one VJP over the batch-2B pair (as jagg_group_backward).
 * dtheta = beta * dtheta + g_jagg. */
jagg_status jagg_grpo_group_backward(jagg_ctx* ctx, const void* theta, const void* saved_pair, int batch,
                                     const jagg_grpo_window* w, void* dtheta, float beta, double* stats);

/* Per-step baseline: W VJPs, one per step, accumulated into dtheta
 * (dtheta = beta * dtheta + sum_j J_j^T s_j).  saved: host array of W device
 * pointers, each a batch-B forward. */
jagg_status perstep_group_backward(jagg_ctx* ctx, const void* theta, const void* const* saved, int batch,
                                   const void* const* s, int W, void* dtheta, float beta);

/* Whole-trajectory gradient (high-noise vs low-noise scheduling; gradient
 * accumulation over groups).  The T steps, in sampling order (t strictly
 * decreasing: high noise first), form n = floor(T / W) full windows (window g
 * = steps gW .. gW + W - 1) and a tail of T mod W steps.  Window g takes the
 * JAGG backward (as jagg_group_backward) when use_jagg[g] = 1 and the per-step
 * backward (as perstep_group_backward) when it is 0; the tail always takes the
 * per-step backward.  dtheta = beta * dtheta + the sum of all windows'
 * gradients.
 *   saved_pairs: host array of n device pointers; entry g is the batch-2B
 *                forward of window g's endpoint pair (read only where
 *                use_jagg[g] = 1; may be NULL elsewhere, or the array NULL
 *                if no window takes JAGG)
 *   saved_steps: host array of T device pointers; entry k is the batch-B
 *                forward of step k (read only for the steps of per-step
 *                windows and of the tail; may be NULL for the others)
 *   s:           host array of T device pointers, batch-B outputs s_k
 *   t:           host, T timesteps
 *   use_jagg:    host, n bytes 0/1 (e.g. from jagg_route); may be NULL if n = 0
 * Workspace: dit_workspace_bytes(2 * batch) if any window takes JAGG, else
 * dit_workspace_bytes(batch).  2 <= W <= 64, T >= 1, batch 1..16 (1..32 if no
 * window takes JAGG).  EINVAL before any launch on a null pointer that would
 * be read, a mask byte other than 0/1, t not strictly decreasing or a size out
 * of range. */
jagg_status jagg_trajectory_backward(jagg_ctx* ctx, const void* theta, int T, int W, int batch,
                                     const void* const* saved_pairs, const void* const* saved_steps,
                                     const void* const* s, const float* t, const unsigned char* use_jagg,
                                     void* dtheta, float beta);

/* One product of a linear layer's backward, the kernel the VJP issues for every
 * projection of a block (backward-cost appendix: the backward of a linear map
 * is two products, the input gradient and the weight gradient).  Weights are
 * stored [n_out][n_in]; dY, X, W and pre are bf16 (JAGG_BF16), row-major,
 * densely packed, device, 16-byte aligned; accumulation is fp32.
 *   JAGG_DGRAD:      result[rows][n_in]  = dY[rows][n_out] W[n_out][n_in]
 *                    (result_dtype JAGG_F32 or JAGG_BF16; beta must be 0)
 *   JAGG_DGRAD_GELU: result[rows][n_in]  = (dY W) * gelu'(pre[rows][n_in])
 *                    (tanh-GELU derivative; result bf16; beta must be 0)
 *   JAGG_WGRAD:      result[n_out][n_in] = beta * result + dY^T X[rows][n_in]
 *                    (result_dtype JAGG_F32 or JAGG_BF16; beta 0 or 1)
 * `other` is W for the two input-gradient kinds and X for JAGG_WGRAD; `pre`
 * is read only by JAGG_DGRAD_GELU.  rows, n_out, n_in >= 1.  Enqueued on the
 * context's stream; needs no workspace.  EINVAL on a null or unaligned
 * pointer, a bad kind, dtype or beta, or a size out of range. */
typedef enum { JAGG_DGRAD = 0, JAGG_DGRAD_GELU = 1, JAGG_WGRAD = 2 } jagg_linear_kind;
jagg_status jagg_linear_grad(jagg_ctx* ctx, int kind, const void* dY, const void* other, const void* pre, int rows,
                             int n_out, int n_in, void* result, int result_dtype, float beta);

/* Measurement hook (no effect on results).  jagg_prof_begin(cls) arms one
 * kernel class for this process; every later launch of that class, on any
 * context, is bracketed by a pair of HIP events on its stream.
 * jagg_prof_end synchronises those events, returns the launch count, the
 * summed kernel time in ms and the summed algorithmic work of the launches
 * (FLOPs: 2 per multiply-add of the defining products; bytes for the
 * aggregation: W reads + 2 writes per element), and disarms.
 * Classes: 1 forward GEMM (Y = X W^T), 2 input-gradient GEMM (dX = dY W),
 * 3 weight-gradient GEMM (dW = dY^T X), 4 attention forward (work: the QK^T
 * and PV products), 5 attention backward dK/dV kernel (work: the dV, dP and
 * dK products; the score recompute is not counted), 6 attention backward dQ
 * kernel (work: the dQ product), 7 aggregation, 8 gradient comparison (work:
 * bytes read), 9 GRPO upstream gradients and their composites (work: bytes). */
jagg_status jagg_prof_begin(int cls);
jagg_status jagg_prof_end(long* launches, double* total_ms, double* total_work);

#ifdef __cplusplus
}
#endif

#endif /* JAGG_H */
