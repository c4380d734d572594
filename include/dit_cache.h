/*
 * dit_cache.h -- C ABI of the budget-aware cached DiT sampler for MI355X (gfx950).
 *
 * One call of dit_cache_sample runs one sample of T Euler flow-matching steps.
 * At every step the library
 *   1. forms the first block's adaLN-modulated image-token input m_t (the
 *      trajectory tensor of Eq. 3; DIT_INDICATOR_PATCH selects the paper's
 *      post-patch-embedding tensor instead),
 *   2. reduces it against the previous step's and the last computed step's
 *      copies into relative-L1 distances (Eq. 3, trajectory state),
 *   3. evaluates the gate of Eq. 1 on the budget and trajectory state and
 *      applies the two budget rules of Alg. 2 (spend the remainder; stop
 *      when the budget is spent), so exactly B steps are computed and step 0
 *      always is (Sec. 3.1),
 *   4. runs the full block stack and refreshes the cached residual
 *      r = h_out - h, or reuses it: h_out = h + r (plain residual reuse,
 *      Sec. 3.1 and App. A.1; under guidance both branches share the
 *      decision, each keeps its own residual),
 *   5. applies the final layer, the guidance combine and the Euler update
 *      x_{t+1} = x_t + (sigma_{t+1} - sigma_t) v.
 * All of this runs in hand-written HIP kernels, except the 8-feature gate
 * and the pacing rule, which run on the host in double precision between
 * two kernel launches (one 32-byte device->host read per step).
 *
 * Conventions
 *   - Every function returns a dit_status; DIT_OK is 0, errors are < 0 and
 *     dit_cache_last_error() gives a message.  On error, the latent is
 *     unspecified and *out holds the steps completed so far.
 *   - The caller owns every buffer it passes; the library never frees them.
 *     The library owns its device copy of the weights and its workspace.
 *   - Device buffers are plain device pointers (e.g. torch tensor
 *     data_ptr()).  Work is enqueued on the stream given at create time and
 *     every call returns after that stream has drained.
 *   - A handle is not thread-safe: use one handle per host thread.
 */
#ifndef DIT_CACHE_H
#define DIT_CACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DIT_ABI_VERSION 4
#define DIT_N_FEATURES 8

typedef enum dit_status {
  DIT_OK = 0,
  DIT_EINVAL = -1,      /* null pointer, bad enum, bad gate blob, bad forced mask  */
  DIT_ENOMEM = -2,      /* device or pinned host allocation failed                 */
  DIT_EHIP = -3,        /* a HIP runtime call failed                               */
  DIT_ESHAPE = -4,      /* config sizes inconsistent or blob size mismatch         */
  DIT_EBUDGET = -5,     /* T < 1, B < 1 or B > T                                   */
  DIT_ENONFINITE = -6   /* an indicator sum is not finite (NaN/Inf in the latent)  */
} dit_status;

enum { DIT_DTYPE_F32 = 0, DIT_DTYPE_BF16 = 1 };
enum { DIT_INDICATOR_MODULATED = 0, DIT_INDICATOR_PATCH = 1 };

/* Model shape.  Exactly one family: n_double/n_single (MMDiT: double-stream
 * blocks followed by single-stream blocks on [txt; img]) or n_cross (video
 * blocks: self-attention, cross-attention to the text, FFN).
 * Requirements: hidden = heads * head_dim; bf16 needs head_dim == 128 and
 * hidden, mlp_hidden, ctx_dim, in_channels, time_dim multiples of 8; f32
 * needs head_dim <= 128 and a multiple of 4. */
typedef struct dit_model_config {
  int32_t abi_version;   /* DIT_ABI_VERSION                                  */
  int32_t dtype;         /* storage dtype S: DIT_DTYPE_F32 or DIT_DTYPE_BF16  */
  int32_t n_double, n_single, n_cross;
  int32_t hidden;        /* H */
  int32_t heads, head_dim;
  int32_t mlp_hidden;    /* F */
  int32_t in_channels;   /* C: latent channels per token */
  int32_t ctx_dim;       /* text embedding width */
  int32_t time_dim;      /* sinusoidal timestep embedding width (256) */
  int32_t n_img;         /* N image / video tokens */
  int32_t n_txt;         /* N_t text tokens */
  int32_t batch;         /* 1, or 2 = (conditional, unconditional) guidance pair */
  int32_t pooled_text;   /* 1: vec also adds an MLP of the mean text token */
} dit_model_config;

/* Weight blob (host memory, copied at create; elements of the storage
 * dtype: bf16 bit patterns or f32).  Tensors are concatenated in this
 * order, each row-major, linear weights as [out, in] (mod width
 * M = 12H*n_double + 3H*n_single + 6H*(n_cross > 0) + 2H):
 *   img_in.w [H,C] img_in.b [H]  txt_in.w [H,ctx] txt_in.b [H]
 *   time_in.0.w [H,time_dim] .0.b [H]  time_in.2.w [H,H] .2.b [H]
 *   (pooled_text) pool_in.0.w [H,ctx] .0.b [H] pool_in.2.w [H,H] .2.b [H]
 *   mod.w [M,H] mod.b [M]
 *   per double block i, stream img then txt:
 *     qkv.w [3H,H] qkv.b [3H] o.w [H,H] o.b [H] mlp0.w [F,H] mlp0.b [F] mlp1.w [H,F] mlp1.b [H]
 *   per single block i: l1.w [3H+F,H] l1.b [3H+F] l2.w [H,H+F] l2.b [H]
 *   per cross block i: mod_offset [6H] qkv.w [3H,H] qkv.b o.w [H,H] o.b xq.w [H,H] xq.b
 *     xkv.w [2H,H] xkv.b xo.w [H,H] xo.b ffn0.w [F,H] ffn0.b ffn1.w [H,F] ffn1.b
 *   final.w [C,H] final.b [C]
 * Modulation chunks inside one step's M-wide vector: double block i at
 * 12H*i: img (shift1, scale1, gate1, shift2, scale2, gate2) then txt; single
 * block i at 12H*n_double + 3H*i: (shift, scale, gate); video blocks: one
 * shared 6H chunk plus each block's mod_offset; final layer: the last 2H
 * (shift, scale). */

/* Per-call sampler parameters. */
/* Decision policies (Sec. 3 states the three paradigms on one cost model:
 * every policy runs the same kernels and records the same features).
 *   GATE       Alg. 2: the gate's vote z_t > ln(tau/(1-tau)), overridden by
 *              the budget rules; realised NFE = B.
 *   STATIC     m = mu(B, T), fixed before sampling: computed steps at
 *              t_i = floor(i T / B), i = 0..B-1; realised NFE = B.  The
 *              gate blob is not read (may be NULL).
 *   THRESHOLD  online rule m_t = [q_t > delta], q_t = relative-L1 change of
 *              the indicator accumulated since the last computed step
 *              (feature f7); t = 0 computes; no budget rule, so the realised
 *              NFE is whatever the rule spends (B enters only the features).
 *              The gate blob is not read (may be NULL). */
enum { DIT_POLICY_GATE = 0, DIT_POLICY_STATIC = 1, DIT_POLICY_THRESHOLD = 2 };

/* Step rule applied to the network's velocity v_t at every step.
 *   EULER  x_{t+1} = x_t + (sigma_{t+1} - sigma_t) v_t.
 *   UNIPC  UniPC-2 predictor-corrector (Zhao et al. 2023; the Wan sampler of
 *          Sec. 4.1) on the data prediction m_t = x_t - sigma_t v_t with
 *          B(h) = e^h - 1, lambda = log((1 - sigma) / sigma): the network sees
 *          x_t, the corrector then refines x_t with m_t, and the predictor
 *          steps from the corrected sample.  Orders: min(2, i + 1, T - i) for
 *          the predictor of step i; the corrector of step i uses step i-1's. */
enum { DIT_SOLVER_EULER = 0, DIT_SOLVER_UNIPC = 1 };

typedef struct dit_sample_params {
  int32_t T;                    /* steps, >= 1 */
  int32_t B;                    /* full evaluations, 1 <= B <= T */
  const double* sigmas;         /* host [T+1] in [0, 1], strictly decreasing (the default schedule
                                   runs from sigma_0 = 1 to sigma_T = 0), or NULL; else DIT_EINVAL */
  double shift;                 /* used when sigmas == NULL: sigma_i = s u / (1 + (s-1) u), u = 1 - i/T */
  double tau;                   /* cutoff on sigma(z), in (0, 1); the paper uses 0.5 */
  double guidance;              /* guidance scale g, used when batch == 2 */
  const uint8_t* forced_mask;   /* host [T] replay mask (m_0 = 1; exactly B ones unless the
                                   policy is DIT_POLICY_THRESHOLD) or NULL */
  int32_t indicator;            /* DIT_INDICATOR_MODULATED (default) or DIT_INDICATOR_PATCH */
  int32_t policy;               /* DIT_POLICY_GATE (default), _STATIC or _THRESHOLD */
  double delta;                 /* DIT_POLICY_THRESHOLD's cutoff on q_t */
  int32_t solver;               /* DIT_SOLVER_EULER (default) or DIT_SOLVER_UNIPC */
} dit_sample_params;

/* Per-step record, host arrays owned by the caller (each may be NULL
 * except `full`). */
typedef struct dit_schedule {
  uint8_t* full;       /* [T] 1 = network evaluated and cache refreshed, 0 = residual reused */
  float* logit;        /* [T] gate logit z_t (THRESHOLD: q_t; NaN at t = 0 and under STATIC) */
  uint8_t* forced;     /* [T] 1 where a budget rule (or t = 0) fixed the decision */
  double* features;    /* [T * 8] gate inputs f0..f7 (NaN row at t = 0) */
  double* sums;        /* [T * 4] sum|m_t-m_{t-1}|, sum|m_{t-1}|, sum|m_t-m_last|, sum|m_last| */
  int32_t nfe;         /* out: computed steps (== B on success unless THRESHOLD) */
  int32_t steps_done;  /* out: steps completed */
} dit_schedule;

typedef struct dit_cache dit_cache;

/* Validate the config, allocate device weights + workspace, copy the blob
 * (host pointer, nbytes must equal the layout above) on `hip_stream` (a
 * hipStream_t, or NULL for the null stream).  *out receives the handle. */
dit_status dit_cache_create(const dit_model_config* cfg, const void* weights, size_t nbytes,
                            void* hip_stream, dit_cache** out);

/* One sample with the paper's defaults (tau = 0.5, guidance 1, shift 1,
 * modulated indicator, gated decisions).
 *   latent   device, f32 [n_img, in_channels]: x_0 in, x_T out (in place)
 *   text_emb device, storage dtype [batch, n_txt, ctx_dim] (conditional first)
 *   gate_weights host f32 blob: [k, d_0..d_{k-1}, zflag, (mu[d_0], sd[d_0]),
 *                W_1, b_1, ..., W_{k-1}, b_{k-1}], W_l row-major [d_l, d_{l-1}],
 *                ReLU between layers, d_{k-1} = 1, d_0 <= 8 (reads f0..f_{d_0-1}) */
dit_status dit_cache_sample(dit_cache* h, float* latent, const void* text_emb, int32_t T, int32_t B,
                            const float* gate_weights, size_t gate_len, dit_schedule* out);

/* Same with explicit parameters (sigma schedule or shift, tau, guidance,
 * replay mask, indicator tensor). */
dit_status dit_cache_sample_ex(dit_cache* h, float* latent, const void* text_emb,
                               const float* gate_weights, size_t gate_len,
                               const dit_sample_params* p, dit_schedule* out);

/* n_samples independent samples (one prompt each) advanced in lockstep, each
 * with its own schedule (Sec. 3.1 poses the problem per prompt p): at
 * every step the library forms and reduces every sample's indicator, waits
 * once for all their sums, decides per sample (Alg. 2 with that sample's
 * own budget state), reuses the cached residuals of the samples that skip,
 * and runs the block stack of the samples that compute together: every
 * linear layer is one GEMM launch over all their rows, attention one launch
 * over all their sequences.  Sample j's result is the result of
 * dit_cache_sample_ex on its own inputs, up to the rounding of the stacked
 * launches.
 *   latents   device, f32 [n_samples, n_img, in_channels]: x_0 in, x_T out
 *   text_emb  device, storage dtype [n_samples, batch, n_txt, ctx_dim]
 *   p         shared by all samples; p->forced_mask, if not NULL, is host
 *             [n_samples, T] (one replay mask per sample)
 *   out       host array of n_samples schedules, one per sample
 * Workspace for n_samples is allocated on first use and kept (per sample
 * about 6 [n_img, hidden] tensors plus, for the stacked block stack, the
 * rows of every sequence).  On error every latent is unspecified and each
 * out[j].steps_done holds the steps that sample completed. */
dit_status dit_cache_sample_batch(dit_cache* h, int32_t n_samples, float* latents, const void* text_emb,
                                  const float* gate_weights, size_t gate_len,
                                  const dit_sample_params* p, dit_schedule* out);

/* The gate of Eq. 1 alone, on the host in double precision: *logit =
 * z = g_theta(f) for one 8-feature state f (features[0..7], the layout of
 * dit_schedule.features; a gate with d_0 < 8 inputs reads f_0..f_{d_0-1}),
 * from the same self-describing blob dit_cache_sample takes (plain MLP or
 * the branched form of App. A.2, optional z-scoring).  Alg. 2 computes when
 * z > ln(tau / (1 - tau)).  Needs no device.  Errors: DIT_EINVAL (null
 * pointer or malformed blob; the message via dit_cache_last_error(NULL)). */
dit_status dit_gate_logit(const float* gate_weights, size_t gate_len, const double* features, double* logit);

void dit_cache_destroy(dit_cache* h);

/* Last error message of this handle ("" if none).  With h == NULL: the last
 * error of a failed dit_cache_create on this thread. */
const char* dit_cache_last_error(const dit_cache* h);

/* ---- measurement ------------------------------------------------------ */

/* Kernel classes timed with HIP events on the handle's stream when
 * profiling is on. */
enum {
  DIT_K_GEMM = 0,       /* block-stack GEMMs (MFMA)                             */
  DIT_K_ATTN = 1,       /* block-stack attention (MFMA)                          */
  DIT_K_INDICATOR = 2,  /* patch embed + modulated indicator + reduction         */
  DIT_K_REUSE = 3,      /* reuse step: residual add, final layer, Euler          */
  DIT_K_FULL_OTHER = 4, /* full step: LN-modulate, transposes, refresh, final    */
  DIT_K_ONCE = 5,       /* once per sample: text, vec and modulation table       */
  DIT_K_COUNT = 6
};

typedef struct dit_stats {
  double ms[DIT_K_COUNT];        /* summed event time per class               */
  double work[DIT_K_COUNT];      /* algorithmic FLOPs (GEMM, ATTN) or bytes   */
  int64_t launches[DIT_K_COUNT];
  double host_gate_ms;           /* host time from sums ready to decision     */
  double sample_ms;              /* wall time of dit_cache_sample calls       */
  int64_t samples, full_steps, reuse_steps;
} dit_stats;

dit_status dit_cache_set_profiling(dit_cache* h, int32_t enable);
dit_status dit_cache_get_stats(const dit_cache* h, dit_stats* out);
dit_status dit_cache_reset_stats(dit_cache* h);

#ifdef __cplusplus
}
#endif
#endif /* DIT_CACHE_H */
