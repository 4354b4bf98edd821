/*
 * track.h -- C ABI of the TRACK denoising hot path for AMD MI355X (gfx950).
 *
 * TRACK (trajectory-aware capacity routing via top-K selection) runs, at each
 * denoising step, either a large or a small video-DiT denoiser on the shared
 * latent, guides it with classifier-free guidance (Eq. 1) and advances the
 * latent with the scheduler (Eq. 2).  An offline calibration rolls out the
 * all-large trajectory, probes both models at every step (Sec. "Reference-
 * Trajectory Calibration"), scores them with the relative disagreement of
 * Eq. 4, averages over samples (Eq. 5) and routes the K lowest-scoring steps
 * to the small model (Sec. "Constrained Trajectory Divergence Minimization
 * using Top-K Switching"); inference then follows that policy (Eq. 3).
 *
 * Conventions for every call:
 *  - Returns TRACK_OK (0) or a TRACK_E_* code; the message of the last failure
 *    on the calling thread is available from track_last_error().  Nothing
 *    aborts and no C++ exception crosses this interface.  Outputs are
 *    unspecified when a call fails.
 *  - "dev" pointers are HIP device pointers on the current device; "host"
 *    pointers are ordinary host memory.  The caller owns every buffer; the
 *    library never allocates device memory on the compute path (the caller
 *    provides the workspace) and never frees caller memory.
 *  - stream is a hipStream_t passed as void* (NULL = the default stream).
 *    Calls marked "asynchronous" only enqueue work on that stream.
 *  - The latent is C x F x H x W float32, contiguous (the layout of the
 *    paper's Preliminaries).  Text embeddings are [text_len, text_dim] in the
 *    model's dtype (float32 or bfloat16), contiguous.
 *  - Determinism: identical inputs on one device give identical bits.  The
 *    large-model evaluations and latent updates of track_calibrate are
 *    bit-identical to track_sample with an all-large policy.
 */
#ifndef TRACK_H
#define TRACK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t track_status;
#define TRACK_OK             0
#define TRACK_E_INVALID      1  /* null pointer, bad enum, out-of-range scalar */
#define TRACK_E_SHAPE        2  /* shapes inconsistent with the model or each other */
#define TRACK_E_INCOMPATIBLE 3  /* large/small pair does not share latent, conditioning and dtype */
#define TRACK_E_DEVICE       4  /* a HIP runtime call failed */
#define TRACK_E_NOMEM        5  /* workspace missing or too small */
#define TRACK_E_UNSUPPORTED  6  /* valid request this build does not implement */

#define TRACK_DTYPE_F32  0
#define TRACK_DTYPE_BF16 1

/* Shape of a Wan-2.1-style video DiT denoiser f_m(x, t, c). */
typedef struct track_dit_config {
  int32_t blocks;     /* transformer blocks */
  int32_t dim;        /* hidden width d = heads * head_dim */
  int32_t heads;
  int32_t head_dim;   /* even; the bfloat16 path requires 128 */
  int32_t ffn_dim;    /* MLP hidden width */
  int32_t in_ch;      /* latent channels C (also the output channels) */
  int32_t patch_t, patch_h, patch_w;
  int32_t text_dim;   /* width of the text embedding */
  int32_t freq_dim;   /* sinusoidal timestep features (even) */
  int32_t dtype;      /* TRACK_DTYPE_F32 or TRACK_DTYPE_BF16: weights, text and activations */
} track_dit_config;

/* Latent C x F x H x W and text context length. */
typedef struct track_latent_shape {
  int32_t channels, frames, height, width;
  int32_t text_len;
} track_latent_shape;

/* Flow-matching sampler (Eq. 2) on the table sigma_i = s u/(1+(s-1)u),
 * u = 1 - i/N (sigma_0 = 1, sigma_N = 0), model timestep t_i = 1000 sigma_i.
 *   TRACK_SOLVER_EULER  x += (sigma_{i+1} - sigma_i) p.
 *   TRACK_SOLVER_UNIPC  UniPC (Zhao et al., 2023) of order 1..3 in its
 *     data-prediction form with B(h) = e^h - 1 on alpha = 1 - sigma,
 *     lambda = log(alpha / sigma), m = x - sigma p: a corrector from step 1
 *     on (reusing the model output at the predicted point), a predictor of
 *     order min(order, i + 1, N - i), history entries at sigma = 1 left out,
 *     rho = 1/2 for the order-2 predictor and the order-1 corrector.  The
 *     scheduler history h_i is kept across model switches. */
#define TRACK_SOLVER_EULER 0
#define TRACK_SOLVER_UNIPC 1
typedef struct track_sampler_config {
  int32_t steps;      /* N >= 1 */
  int32_t use_cfg;    /* 1: Eq. 1 guidance with the negative prompt; 0: conditional prediction only */
  double  shift;      /* s > 0 */
  double  guidance;   /* w of Eq. 1 */
  double  eps;        /* epsilon of Eq. 4 (> 0) */
  int32_t solver;     /* TRACK_SOLVER_EULER or TRACK_SOLVER_UNIPC */
  int32_t order;      /* UniPC order, 1..3 (ignored by Euler) */
} track_sampler_config;

typedef struct track_model_t* track_model;

/* ---------------------------------------------------------------- weights
 * Weights live in one caller-owned device buffer of track_weights_bytes(cfg)
 * bytes.  Tensor i sits at byte offset track_weight_info(...).offset, dense
 * row-major, elements of the config's dtype; every offset is 256-byte
 * aligned.  Linear weights are [out_features, in_features].  The tensor list
 * (names and shapes) is:
 *   patch.w [d, C*pt*ph*pw], patch.b [d], time.w1 [d, freq], time.b1 [d],
 *   time.w2 [d, d], time.b2 [d], mod.w [6d, d], mod.b [6d],
 *   text.w1 [d, text_dim], text.b1 [d], text.w2 [d, d], text.b2 [d],
 *   then per block b: blk<b>.mod [6, d] (shift1, scale1, gate1, shift2,
 *   scale2, gate2 offsets added to the shared modulation), qkv.w [3d, d],
 *   qkv.b [3d], norm_q [d], norm_k [d], o.w [d, d], o.b [d], cq.w [d, d],
 *   cq.b [d], ckv.w [2d, d], ckv.b [2d], norm_cq [d], norm_ck [d],
 *   co.w [d, d], co.b [d], ffn1.w [ffn, d], ffn1.b [ffn], ffn2.w [d, ffn],
 *   ffn2.b [d]; then head.mod [2, d] (shift, scale), head.w [C*pt*ph*pw, d],
 *   head.b [C*pt*ph*pw]. */
int32_t track_weight_count(const track_dit_config* cfg);            /* < 0 on an invalid config */
size_t  track_weights_bytes(const track_dit_config* cfg);           /* 0 on an invalid config */
track_status track_weight_info(const track_dit_config* cfg, int32_t index, const char** name /* static string */,
                               int32_t* ndim, int64_t shape[2], size_t* offset_bytes);

/* ---------------------------------------------------------------- models
 * A model is a non-owning view of a weight buffer plus the workspace the
 * caller attaches.  The buffers must outlive the handle.  dev_weights must be
 * 256-byte aligned and hold track_weights_bytes(cfg) bytes. */
track_status track_model_create(const track_dit_config* cfg, const void* dev_weights, size_t bytes, track_model* out);
void         track_model_destroy(track_model m);   /* NULL is a no-op */

/* Workspace (activations for one guided prediction of `batch` = 2 with
 * guidance, 1 without, plus trajectory state) for the given latent shape.
 * Returns 0 when the shape is invalid for the model. */
size_t       track_workspace_bytes(track_model m, const track_latent_shape* shape, int32_t batch);
/* Attach a caller-owned, 256-byte aligned device workspace; calls that use
 * the model must not overlap on the GPU while they share it. */
track_status track_model_set_workspace(track_model m, void* dev_ws, size_t bytes);

/* ---------------------------------------------------------------- the four calls
 * One guided prediction p_m(x_t, t) (Eq. 1): the denoiser on cond and, when
 * uncond != NULL, on uncond, combined as f(null) + w (f(cond) - f(null)).
 * uncond == NULL gives the conditional prediction f(x_t, t, cond).
 * t is the model timestep (1000 sigma).  x_t, p_out: dev C x F x H x W float32
 * (may not alias).  Needs a workspace for batch 2 (1 without uncond).
 * Asynchronous. */
track_status track_dit_forward(track_model m, const track_latent_shape* shape, const float* x_t, double t,
                               const void* cond, const void* uncond, float guidance_scale, float* p_out,
                               void* stream);

/* Reference-trajectory calibration (Sec. "Reference-Trajectory Calibration"):
 * for every sample j < M start at x_T[j] (dev latent), at each step k evaluate
 * p_L and p_S on the same latent, timestep, cond[j], uncond and guidance,
 * record r[j*N + k] (Eq. 4, Frobenius norms over the whole latent, float64),
 * then advance with p_L.  q[k] is the mean over j in sample order (Eq. 5).
 * x_T, cond: host arrays of M device pointers; uncond NULL iff !use_cfg.
 * r_out (host, M*N) and q_out (host, N) may be NULL.  x0_out, if not NULL,
 * is a host array of M device latents that receive each sample's all-large
 * endpoint (the reference trajectory's x after N steps).  The pair must be
 * compatible (same in_ch, patch, text_dim, dtype; "Compatible model pairs").
 * Uses the large model's workspace for the trajectory state.  Synchronises
 * the stream before returning. */
track_status track_calibrate(track_model large, track_model small, const track_latent_shape* shape, int32_t M,
                             const float* const* x_T, const void* const* cond, const void* uncond,
                             const track_sampler_config* scfg, double* r_out, double* q_out, float* const* x0_out,
                             void* stream);

/* Calibration with the frequency-band decomposition of the disagreement
 * (Sec. "Frequency Analysis"): everything track_calibrate does, and at each
 * step k of sample j the guided difference d = p_S - p_L on the C x F x H x W
 * latent is transformed with orthonormal DFTs, spatially over (H, W) for every
 * (c, f) and temporally over F for every (c, h, w).  Frequency index k of an
 * axis of length n has normalised frequency nu = 2 min(k, n - k) / n (1 at
 * Nyquist); the spatial nu is sqrt(nu_h^2 + nu_w^2).  Bands: low nu < 1/3,
 * mid 1/3 <= nu < 2/3, high nu >= 2/3.  band_r_out[(j*N + k)*6 + b] (host,
 * M*N*6, may be NULL) receives ||P_b d||_2 / max(||p_L||_2, eps) for b =
 * spatial low, mid, high, temporal low, mid, high (each triple's squares sum
 * to r^2 of Eq. 4); band_q_out[k*6 + b] (host, N*6, may be NULL) their mean
 * over the samples (Eq. 5 per band).  Needs W <= 1024, H <= 256, F <= 64.
 * Synchronises the stream before returning. */
track_status track_calibrate_bands(track_model large, track_model small, const track_latent_shape* shape, int32_t M,
                                   const float* const* x_T, const void* const* cond, const void* uncond,
                                   const track_sampler_config* scfg, double* r_out, double* q_out,
                                   double* band_r_out, double* band_q_out, float* const* x0_out, void* stream);

/* Top-K routing (Sec. "Constrained Trajectory Divergence Minimization using
 * Top-K Switching"): the K steps with the lowest q go to the small model;
 * equal scores go to the lower step index.  q: host [N]; small_idx: host [K],
 * written in ascending order.  0 <= K <= N.  Host only, synchronous. */
track_status track_route_policy(const double* q, int32_t N, int32_t K, int32_t* small_idx);

/* Eqs. 6-7 in the C_0 form (Sec. "Constrained Trajectory Divergence
 * Minimization"): with W_k = q_k^2, step k goes to the small model iff
 * W_k < C0; at W_k == C0 (where any beta is optimal) it stays on the large
 * model.  q: host [N], no NaN; small_idx: host, room for N indices, receives
 * the selected steps in ascending order; *K_out receives their count.  A C0
 * strictly between the K-th and (K+1)-th smallest W_k selects exactly the
 * steps track_route_policy picks for K.  Host only, synchronous. */
track_status track_route_threshold(const double* q, int32_t N, double C0, int32_t* small_idx, int32_t* K_out);

/* Equal-budget baseline policies (Sec. "Equal-Budget Policy Ablations"):
 * exactly K of N steps go to the small model.
 *   TRACK_POLICY_FIRST_K   steps 0 .. K-1
 *   TRACK_POLICY_LAST_K    steps N-K .. N-1
 *   TRACK_POLICY_RANDOM_K  step k draws the k-th output of a SplitMix64
 *                          generator started at `seed` (state += 0x9E3779B97F4A7C15
 *                          per output, then the generator's two xor-shift-
 *                          multiply rounds); the K smallest outputs win, equal
 *                          outputs going to the lower step.
 * `seed` is ignored by the first two.  small_idx: host [K], ascending.
 * 0 <= K <= N.  Host only, synchronous. */
#define TRACK_POLICY_FIRST_K 0
#define TRACK_POLICY_LAST_K 1
#define TRACK_POLICY_RANDOM_K 2
track_status track_route_baseline(int32_t kind, int32_t N, int32_t K, uint64_t seed, int32_t* small_idx);

/* Routed sampling (Eq. 3): x = x_T; for i < N, x += (sigma_{i+1} - sigma_i)
 * p_{pi(i)}(x, t_i) with pi(i) = small iff use_small[i] != 0.  use_small:
 * host [N].  x_T, x0_out: dev latents (may alias).  Uses the large model's
 * workspace for the trajectory state.  Asynchronous. */
track_status track_sample(track_model large, track_model small, const uint8_t* use_small,
                          const track_latent_shape* shape, const track_sampler_config* scfg, const float* x_T,
                          const void* cond, const void* uncond, float* x0_out, void* stream);

/* Message of the last failed call on this thread ("" if none). */
const char* track_last_error(void);

/* Progress of the long-running calls.  When a callback is set (process
 * wide), track_calibrate and track_sample synchronise the stream after every
 * denoising step and then call fn(user, sample, step, steps) with the sample
 * index (-1 for track_sample) and the step just completed.  NULL (the
 * default) disables it and the per-step synchronisation. */
typedef void (*track_progress_fn)(void* user, int32_t sample, int32_t step, int32_t steps);
track_status track_set_progress(track_progress_fn fn, void* user);

/* ---------------------------------------------------------------- component entry points
 * The individual kernels of the denoiser step, exposed so that each can be
 * checked and timed on its own at full size.  All asynchronous on `stream`;
 * dtype selects float32 or bfloat16 activations and weights. */

/* out = epilogue(A W^T + bias): A dev [M, K] (row stride lda elements),
 * W dev [N, K], bias dev [N] (dtype).  epilogue: 0 bias -> out dtype [M, N];
 * 1 bias + tanh-GELU -> out dtype; 2 resid[M, N] float32 += gate[N] (float32)
 * * (acc + bias); 3 resid += acc + bias; 4 bias -> out float32.
 * out (or resid) row stride ldo elements. */
#define TRACK_EPI_BIAS       0
#define TRACK_EPI_BIAS_GELU  1
#define TRACK_EPI_GATE_RESID 2
#define TRACK_EPI_RESID      3
#define TRACK_EPI_BIAS_F32   4
track_status track_op_linear(int32_t dtype, int32_t epilogue, int64_t M, int64_t N, int64_t K, const void* A,
                             int64_t lda, const void* W, const void* bias, const float* gate, void* out, int64_t ldo,
                             void* stream);

/* The V projection of self-attention with V^T written from the epilogue:
 * y = A W^T + bias (bfloat16, float32 accumulation) stored transposed per
 * batch of L rows, vt[((m / L) * N + n) * ldv + m % L] -- the V^T layout
 * track_op_attention reads, with N = heads * head_dim.  Columns [L, ldv) of
 * vt are not written.  Requires dtype bfloat16, N % 256 == 0, K % 64 == 0,
 * M % L == 0, L >= 128, L, ldv and lda multiples of 8, ldv >= L,
 * lda < 2^22 and 16-byte aligned buffers; otherwise TRACK_E_UNSUPPORTED
 * (shape limits), TRACK_E_SHAPE or TRACK_E_INVALID. */
track_status track_op_linear_vt(int32_t dtype, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                                const void* W, const void* bias, int64_t L, void* vt, int64_t ldv, void* stream);

/* Non-causal scaled dot-product attention, softmax(q k^T / sqrt(head_dim)) v,
 * per batch b and head h.  Row r of q for batch b is q[(b*Lq + r)*ldq +
 * h*head_dim + c]; likewise k with Lk, ldk.  v is given transposed:
 * vt[((b*H + h)*head_dim + c)*ldv + key], ldv >= Lk, entries at key >= Lk
 * finite (the library writes zeros there).  out[(b*Lq + r)*ldo + h*head_dim + c].
 * bfloat16 requires head_dim 128, ldv % 8 == 0, ldq, ldk % 8 == 0 and 16-byte
 * aligned base pointers.  Lq == 0 is a no-op;
 * Lk == 0 is an error (the softmax is undefined). */
track_status track_op_attention(int32_t dtype, int32_t B, int32_t H, int32_t head_dim, int64_t Lq, int64_t Lk,
                                const void* q, int64_t ldq, const void* k, int64_t ldk, const void* vt, int64_t ldv,
                                void* out, int64_t ldo, void* stream);

/* The same attention with q given already multiplied by the softmax scale in
 * base 2, q' = q log2(e) / sqrt(head_dim) (bfloat16 only; the form in which
 * the forward's q RMSNorm writes q, the factor taken inside its one rounding):
 * softmax(q' k^T ln 2) v.  The logits then come out of the matrix cores in
 * log2 units and each probability is one exp2, with no per-element scale.
 * Arguments, layout and errors as track_op_attention; TRACK_E_INVALID for
 * float32. */
track_status track_op_attention_log2q(int32_t dtype, int32_t B, int32_t H, int32_t head_dim, int64_t Lq, int64_t Lk,
                                      const void* q, int64_t ldq, const void* k, int64_t ldk, const void* vt,
                                      int64_t ldv, void* out, int64_t ldo, void* stream);

/* y[r, :] = LN(x[r, :]) * (1 + scale) + shift over width d (biased variance,
 * eps 1e-6, no affine).  x float32 [rows, d]; y dtype [rows, d]; scale,
 * shift float32 [d] or NULL (NULL = plain LN).  d < 1: TRACK_E_SHAPE;
 * d % 4 != 0 or d > 8192: TRACK_E_UNSUPPORTED; rows <= 0 is a no-op. */
track_status track_op_layernorm(int32_t dtype, int64_t rows, int32_t d, const float* x, const float* scale,
                                const float* shift, void* y, void* stream);

/* In place on buf rows (row stride ld elements, segment at column col0, width
 * d = heads*head_dim): RMSNorm with gain g [d] (dtype), eps 1e-6, then, if
 * grid != NULL, 3D RoPE per head with token r % L at (f, h, w) of grid
 * {F', H', W'} (L = F'H'W'), sections head_dim - 4*(head_dim/6), 2*(head_dim/6),
 * 2*(head_dim/6), pairs (2i, 2i+1), angle pos * 10000^(-2i/width).  With RoPE,
 * rope_ws is caller-owned device scratch of 2 * track_rope_table_len(head_dim,
 * grid) floats that receives the cos/sin tables (float64 cast to float32).
 * head_dim % 4 == 0 and d <= 8192, else TRACK_E_UNSUPPORTED; rows <= 0 is a
 * no-op. */
int64_t      track_rope_table_len(int32_t head_dim, const int32_t* grid);   /* -1 on bad input */
track_status track_op_rmsnorm_rope(int32_t dtype, int64_t rows, int32_t heads, int32_t head_dim, void* buf,
                                   int64_t ld, int64_t col0, const void* g, const int32_t* grid, float* rope_ws,
                                   void* stream);

/* The same on the q and k segments of each row at once, as the denoiser's
 * self-attention runs it: columns col0 .. col0 + d with gain g_q and
 * col0 + d .. col0 + 2d with gain g_k (d = heads*head_dim, ld >= col0 + 2d),
 * both rotated with the row's RoPE angles; results equal two
 * track_op_rmsnorm_rope calls bit for bit. */
track_status track_op_rmsnorm_rope_qk(int32_t dtype, int64_t rows, int32_t heads, int32_t head_dim, void* buf,
                                      int64_t ld, int64_t col0, const void* g_q, const void* g_k, const int32_t* grid,
                                      float* rope_ws, void* stream);

/* Step kernels on token-layout velocities vel [B, n] float32 (B = 2: cond
 * then uncond; B = 1: no guidance).  Guided p = u + w (c - u) (Eq. 1).
 * Sample mode: x[n] += dsigma * p.  Calibration mode also takes the small
 * model's velocities and accumulates ||p_S - p_L||^2 and ||p_L||^2, writing
 * r = sqrt(num) / max(sqrt(den), eps) (Eq. 4) to r_out[0] (dev float64), and
 * advances x with p_L.  partial: dev float64 scratch of
 * track_step_partial_count(n) * 2 entries. */
int64_t      track_step_partial_count(int64_t n);
track_status track_op_step(int64_t n, int32_t B, float guidance, float dsigma, const float* vel_L, const float* vel_S,
                           float* x, double* partial, double eps, double* r_out, void* stream);

/* track_op_step without the partial buffer, for callers that cannot allocate
 * device memory (code under HIP graph capture, allocation-free serving
 * loops): the calibration partials live in a static device array of 2048
 * doubles (16 KiB, held on each GPU the library runs on until the process
 * ends), which covers every n (the step kernels use at most 1024 blocks; a
 * larger requirement is rejected with TRACK_E_UNSUPPORTED).  Same arguments
 * and results as track_op_step, bit for bit; allocates nothing.  The array
 * is shared by every call on a GPU, so calls that overlap on one GPU (on
 * different streams or threads) race; calls ordered on one stream do not. */
track_status track_op_step_noalloc(int64_t n, int32_t B, float guidance, float dsigma, const float* vel_L,
                                   const float* vel_S, float* x, double eps, double* r_out, void* stream);

/* Band energies of the guided difference of two token-layout velocity
 * buffers, the kernels of track_calibrate_bands.  vel_large, vel_small:
 * device [batch][L][P] float32 in patch-token layout (L = (F/pt)(H/ph)(W/pw)
 * tokens, P = C pt ph pw entries; entry ((c pt + f%pt) ph + h%ph) pw + w%pw of
 * token ((f/pt)(H/ph) + h/ph)(W/pw) + w/pw holds latent (c, f, h, w));
 * batch 2 applies Eq. 1 with `guidance` (branch 0 conditional, 1 negative
 * prompt), batch 1 takes the conditional branch.  energy_out (host [6])
 * receives ||P_b (p_S - p_L)||_2^2 for b = spatial low, mid, high, temporal
 * low, mid, high (bands as in track_calibrate_bands).  workspace: device,
 * 256-byte aligned, track_band_workspace_bytes(shape, pt, ph, pw) bytes (0 for
 * unsupported shapes).  Synchronous. */
size_t track_band_workspace_bytes(const track_latent_shape* shape, int32_t patch_t, int32_t patch_h, int32_t patch_w);
track_status track_op_band_energy(const track_latent_shape* shape, int32_t patch_t, int32_t patch_h, int32_t patch_w,
                                  int32_t batch, float guidance, const float* vel_large, const float* vel_small,
                                  void* workspace, size_t workspace_bytes, double* energy_out, void* stream);

/* One UniPC step as the kernels apply it, for tests and external drivers.
 * track_unipc_coefficients (host only) fills coef[12] for step `step` of an
 * N-step table of the given shift and order: coef[0] cx, [1] c_m0, [2] c_h1,
 * [3] c_h2, [4] c_new, [5] corrector on (0/1), [6] corrector history terms
 * (0..2), [7] px, [8] p_m, [9] p_h1, [10] p_h2, [11] predictor history terms
 * (0..2).  With m = x - sigma_step p (p the guided velocity, Eq. 1):
 *   x^c    = corrector ? cx x_last + c_m0 h0 + c_h1 h1 + c_h2 h2 + c_new m : x
 *   x_next = px x^c + p_m m + p_h1 h0 + p_h2 h1
 * where h0, h1, h2 are m of the three previous steps (terms beyond the
 * stated counts are absent).  track_op_unipc_step applies this to n floats
 * (n % 4 == 0): x <- x_next, x_last <- x^c, m_out <- m; vel_L [batch][n]
 * gives p; with vel_S it also writes the Eq. 4 partials and r_out like
 * track_op_step.  h0 / h1 / h2 may be NULL when their terms are absent.
 * All device buffers distinct.  Asynchronous on the stream. */
track_status track_unipc_coefficients(int32_t N, double shift, int32_t order, int32_t step, double* coef);
track_status track_op_unipc_step(int64_t n, int32_t batch, float guidance, float sigma, const double* coef,
                                 const float* vel_L, const float* vel_S, float* x, float* x_last, const float* h0,
                                 const float* h1, const float* h2, float* m_out, double* partial, double eps,
                                 double* r_out, void* stream);

/* ---------------------------------------------------------------- profiling
 * For each kernel class whose bit (1 << kind) is set in the mask given to
 * track_profile_enable, the library brackets every launch of that class with
 * HIP events on the launch stream (0 disables).  track_profile_read
 * synchronises the device and returns the launch count and the summed
 * milliseconds since the last track_profile_reset. */
/* Plain HBM streams, the practical bandwidth ceiling the memory-bound
 * kernels are measured against: kind 0 copies `bytes` from src to dst, 1
 * reads src (dst: a device word the kernel may write), 2 fills dst.  bytes
 * must be a positive multiple of 16384; buffers 16-byte aligned.  A copy may
 * run in place (src == dst, the ceiling for in-place kernels); partially
 * overlapping buffers are not allowed.
 * Asynchronous.  Launches count as TRACK_PROF_OTHER below. */
#define TRACK_HBM_COPY  0
#define TRACK_HBM_READ  1
#define TRACK_HBM_WRITE 2
track_status track_hbm_stream(int32_t kind, const void* src, void* dst, int64_t bytes, void* stream);

/* Plain matrix-core stream, the sustained MFMA ceiling the MFMA-bound kernels
 * are measured against beside the published peak: one 4-wave workgroup per
 * compute unit, every wave running 8 independent chains of
 * v_mfma_f32_32x32x16_bf16 for `iters` loop iterations on operands it reads
 * once from `operands` (device, 65536 bytes = 32768 bf16 values, 16-byte
 * aligned; the caller's data, since the clock the chip holds under matrix
 * work depends on the operand bits).  `sink` is a device float the kernel
 * writes only for one planted sum value; *flop (host) receives the launch's
 * floating-point operation count, CUs x 4 x iters x 8 x 32768.
 * iters in [1, 2^31).  Asynchronous.  Launches count as TRACK_PROF_OTHER. */
track_status track_mfma_stream(const void* operands, int64_t iters, float* sink, int64_t* flop, void* stream);

#define TRACK_PROF_ATTN_SELF  0
#define TRACK_PROF_ATTN_CROSS 1
#define TRACK_PROF_GEMM       2
#define TRACK_PROF_NORM       3
#define TRACK_PROF_STEP       4
#define TRACK_PROF_OTHER      5
#define TRACK_PROF_KINDS      6
track_status track_profile_enable(int32_t kind_mask);
track_status track_profile_reset(void);
track_status track_profile_read(int32_t kind, int64_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif
#endif /* TRACK_H */
