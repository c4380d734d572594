/*
 * dit_kernels.h -- component entry points of the cached DiT sampler's
 * full-step kernels (gfx950), for callers that drive single operations:
 * parity tests at full workload shapes and kernel microbenchmarks.
 * Same conventions as dit_cache.h (status codes, caller-owned device
 * buffers, the call returns after the stream has drained).
 */
#ifndef DIT_KERNELS_H
#define DIT_KERNELS_H

#include <stddef.h>
#include <stdint.h>

#include "dit_cache.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Epilogue flags of the bf16 GEMM. */
enum {
  DIT_EPI_STORE = 0,      /* C = S(acc + bias)                                   */
  DIT_EPI_F32 = 1,        /* C (f32) = acc + bias                                */
  DIT_EPI_GATED_RES = 2,  /* C = S(C + gate[n] * (acc + bias)), in place         */
  DIT_EPI_SILU = 4        /* C = S(SiLU(acc + bias))                             */
};

/* C = epilogue(A . W^T + bias): the linear layers of the blocks (QKV with
 * per-head RMS norm of q and k, out-projection and MLP-down with the
 * adaLN-gated residual, MLP-up with GELU-tanh).  bf16 operands, f32
 * accumulation on MFMA, S = round to bf16 (nearest even).
 *   A    device bf16 [M, K], row stride lda elements (lda >= K, K % 8 == 0)
 *   W    device bf16 [N, K], row stride ldw (torch nn.Linear layout)
 *   bias device bf16 [N] or NULL
 *   C    device bf16 (f32 with DIT_EPI_F32) [M, *], row stride ldc (>= N,
 *        plus gap when gap_at < N; else DIT_ESHAPE)
 *   gate device f32 [N], DIT_EPI_GATED_RES only
 *   rms_cols  columns n < rms_cols are normalised per 128-wide head
 *             (RMS, eps 1e-6, unit gain) before rounding; 0 = none;
 *             must be a multiple of 128
 *   gelu_from columns n >= gelu_from get GELU-tanh; >= N = none
 *   gap_at, gap  output column = n + gap for n >= gap_at (writes the MLP
 *             half of a fused projection next to a hole for the attention
 *             output); gap = 0 = none
 * Errors: DIT_EINVAL (null pointers, bad flags), DIT_ESHAPE (K % 8, lda or
 * ldw < K, ldc too small, gap < 0, rms_cols not a multiple of 128), DIT_EHIP. */
typedef struct dit_gemm_desc {
  const void* A; int64_t lda;
  const void* W; int64_t ldw;
  const void* bias;
  void* C; int64_t ldc;
  int32_t M, N, K;
  int32_t flags;
  const float* gate;
  int32_t rms_cols;
  int32_t gelu_from;
  int32_t gap_at, gap;
} dit_gemm_desc;

dit_status dit_gemm_bf16(const dit_gemm_desc* d, void* hip_stream);

/* Attention flags. */
enum {
  /* The caller guarantees |q . k| <= 128 per head (e.g. q and k RMS-normalised
   * with unit gain), so every logit is at most sqrt(128) and a fixed shift
   * replaces the running maximum of the softmax (same result). */
  DIT_ATTN_BOUNDED_LOGITS = 1
};

/* o = softmax(q k^T / sqrt(128)) v per head (non-causal), bf16 in and out,
 * f32 softmax and accumulation on MFMA.  q [Lq, heads*128] (row stride
 * ldq), k and v [Lk, heads*128] (ldk, ldv), o [Lq, heads*128] (ldo);
 * head h occupies columns [128h, 128h + 128).  flags: 0 or
 * DIT_ATTN_BOUNDED_LOGITS.  vt_ws is a device workspace of heads * 128 *
 * round_up(Lk, 64) bf16 elements that receives v transposed per head.
 * Errors: DIT_EINVAL, DIT_ESHAPE (Lq, Lk < 1), DIT_EHIP. */
dit_status dit_attention_bf16(const void* q, int64_t ldq, const void* k, int64_t ldk,
                              const void* v, int64_t ldv, void* o, int64_t ldo,
                              int32_t Lq, int32_t Lk, int32_t heads, int32_t flags, void* vt_ws,
                              void* hip_stream);

/* Largest v-transpose the allocation-free attention holds: heads * 128 *
 * round_up(Lk, 64) bf16 elements (32 MiB; e.g. 24 heads at up to 5440 keys). */
#define DIT_NOALLOC_VT_MAX_ELEMS (16 * 1024 * 1024)

/* dit_attention_bf16 without the vt_ws workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  The transposed values go to a
 * fixed device array of DIT_NOALLOC_VT_MAX_ELEMS bf16 elements inside the
 * library, one per GPU, held until the process ends; the call allocates
 * nothing (no hipMalloc / hipFree, no allocating library routine).  The
 * array's device address is looked up once per device, on the first call
 * made with that device current.  Same arguments, kernels and result bits
 * as dit_attention_bf16.  Every call on one GPU shares that GPU's array:
 * calls that overlap on one GPU (other streams or host threads) race and
 * must be serialised by the caller.  Errors: as dit_attention_bf16, plus
 * DIT_ESHAPE when heads * 128 * round_up(Lk, 64) > DIT_NOALLOC_VT_MAX_ELEMS
 * (nothing is launched). */
dit_status dit_attention_bf16_noalloc(const void* q, int64_t ldq, const void* k, int64_t ldk,
                                      const void* v, int64_t ldv, void* o, int64_t ldo,
                                      int32_t Lq, int32_t Lk, int32_t heads, int32_t flags,
                                      void* hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* DIT_KERNELS_H */
