// Internal launchers of the gfx950 kernels (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/dit_kernels.h"

namespace dit {

struct GemmArgs {
  const void* A; int64_t lda;
  const void* W; int64_t ldw;
  const void* bias;
  void* C; int64_t ldc;
  const float* gate;
  int M, N, K;
  int flags;
  int rms_cols = 0;
  int gelu_from = 0x7fffffff;
  int gap_at = 0x7fffffff;
  int gap = 0;
  // Gated residual with one gate vector per segment of gseg rows: row m uses
  // gate + (m / gseg) * gstride.  gseg = 0: one vector; else a multiple of 32.
  int gseg = 0;
  int64_t gstride = 0;
  // Values transposed for attention (vt != nullptr): output columns
  // [vt_col0, vt_col0 + 128 vt_heads) are not stored in C but written, with
  // bias and bf16 rounding as usual, as vt[z][head][d][key] with row stride
  // vt_ld and the key order of launch_transpose_v_bf16 (permuted inside
  // 16-key groups).  Output row m (m < vt_split: segment 0, else segment 1
  // with m - vt_split) of a segment with R rows per sequence and key offset
  // k0 goes to sequence m / R, key k0 + m % R.
  void* vt = nullptr;
  int vt_col0 = 0, vt_heads = 0, vt_ld = 0;
  int vt_split = 0x7fffffff;
  int vt_rows0 = 1, vt_key0 = 0, vt_rows1 = 1, vt_key1 = 0;
};

// bf16 MFMA GEMM; n = 1 or 2 independent problems in one launch.  Invalid
// arguments (no tile configuration admits the problem) return an error.
hipError_t launch_gemm_bf16(const GemmArgs* g, int n, hipStream_t s, int n_cu);
// Whether launch_gemm_bf16 can write the transposed values of these problems
// itself (the vt fields set): 128-column head groups, 32-row aligned segments
// and the 256 x 256 kernel.  Otherwise the caller leaves vt unset and
// transposes the values with launch_transpose_v_bf16.
bool gemm_bf16_fuses_vt(const GemmArgs* g, int n, int n_cu);
// v = A W^T + bias for N <= 128 (multiple of 16), K % 32 == 0, f32 output; with
// x != nullptr the result goes into the Euler update x += alpha * v instead.
hipError_t launch_proj_small_n(const void* A, int64_t lda, const void* W, int64_t ldw, const void* bias,
                               float* out, int64_t ldo, float* x, int64_t ldx, float alpha, int M, int N,
                               int K, hipStream_t s);
// f32 GEMM (small f32 workloads); bias f32; rms_cols handled by rms_heads_f32.
hipError_t launch_gemm_f32(const GemmArgs* g, int n, hipStream_t s);

// Flash attention, bf16, head_dim 128. vt = v transposed per head:
// [heads][128][ldvt], ldvt = round_up(Lk, 64), zero padded.  Rows r >= split
// of q, k, v and o are stored gap rows further down (a joint sequence split
// over a buffer of stacked sequences); split = INT_MAX for one contiguous
// piece.  nseq independent sequences in one launch: sequence z's rows start
// z * zs rows down, its gap is gap + z * gz, its vt block is the z-th
// [heads][128][ldvt] block.
hipError_t launch_transpose_v_bf16(const void* v, int64_t ldv, void* vt, int Lk, int heads,
                                   hipStream_t s, int split = 0x7fffffff, int64_t gap = 0, int nseq = 1,
                                   int64_t zs = 0, int64_t gz = 0);
hipError_t launch_flash_attn_bf16(const void* q, int64_t ldq, const void* k, int64_t ldk,
                                  const void* vt, int ldvt, void* o, int64_t ldo, int Lq,
                                  int Lk, int heads, bool bounded_logits, hipStream_t s,
                                  int split = 0x7fffffff, int64_t gap = 0, int nseq = 1, int64_t zs = 0,
                                  int64_t gz = 0);
// f32 attention, head_dim <= 128 (multiple of 4).
hipError_t launch_attn_f32(const float* q, int64_t ldq, const float* k, int64_t ldk,
                           const float* v, int64_t ldv, float* o, int64_t ldo, int Lq, int Lk,
                           int heads, int head_dim, hipStream_t s);

// ---- streaming kernels, templated on the storage type (float or bf16) ----
// out = S(LN(x) * (1 + scale) + shift) per row; rows < split use (sh0, sc0),
// the others (sh1, sc1); mod vectors are f32.  scale == nullptr: plain LN.
// Several sequences stacked by rows: row r < split takes its vectors
// (r / seg0) * mstride floats further on, row r >= split (r - split) / seg1.
template <typename T>
hipError_t launch_ln_mod(const T* x, int64_t ldx, T* out, int64_t ldo, int rows, int H, int split,
                         const float* sh0, const float* sc0, const float* sh1, const float* sc1,
                         hipStream_t s, int seg0 = 0x7fffffff, int seg1 = 0x7fffffff, int64_t mstride = 0);
// Indicator: m = S(LN(h)(1+sc)+sh) (or m = h when sc == nullptr), written
// to m_out; with partials != nullptr the relative-L1 sums |m-mp|, |mp|,
// |m-ml|, |ml| are reduced in a fixed order into out[4] (f64, host-mapped)
// through `partials` (indicator_partials(rows) 4-vectors).
template <typename T>
hipError_t launch_indicator(const T* h, T* m_out, const T* m_prev, const T* m_last, int rows,
                            int H, const float* sh, const float* sc, double* partials, double* out,
                            hipStream_t s);
int indicator_partials(int rows);
// out[0..3] = fixed-order float64 sum of n partial 4-vectors (out host-mapped).
hipError_t launch_reduce_partials(const double* partials, int n, double* out, hipStream_t s);

// Fused streaming kernels (bf16; C in {32, 64, 128}, H % 32 == 0): the
// patch embedding h = S(S(x) W_in^T + b_in) is recomputed in LDS.
bool reuse_fused_fits(int C, int H);
int reuse_indicator_partials(int rows);
// m_out = S(LN(h)(1 + sc) + sh) (m_out = h when sc == nullptr) and, with
// partials != nullptr, the four relative-L1 sums against m_prev / m_last into
// out[4]; with h_out != nullptr only h is written (to h_out).
hipError_t launch_reuse_indicator(const float* x, int C, const void* W_in, const void* b_in, void* m_out,
                                  const void* m_prev, const void* m_last, int rows, int H, const float* sh,
                                  const float* sc, double* partials, double* out, void* h_out, hipStream_t s);
// Reuse step of nb (1 or 2) branches: h_out = S(h + r_b), y = S(LN(h_out)(1 +
// scale) + shift) with (shift, scale) = mod_b[0..H), mod_b[H..2H), v_b = y
// W_out^T + b_out, v = v_0 (nb = 1) or v_1 + guidance (v_0 - v_1), x += dsig v.
// With vout != nullptr the combined v is written there (f32 [rows, C]) and x
// is left unchanged (the step rule runs afterwards).
hipError_t launch_reuse_final(float* x, int C, const void* W_in, const void* b_in, const void* r, int nb,
                              const void* W_out, const void* b_out, const float* mod0, const float* mod1,
                              float dsig, float guidance, int rows, int H, float* vout, hipStream_t s);
// One step's streaming work fused (bf16, C = 64): the embedding once in LDS;
// with m_out != nullptr m_t and (with m_prev != nullptr, partials !=
// nullptr) the four relative-L1 sums into out[4]; with r != nullptr also the
// reuse candidate of nb branches: x + dsig v into x_spec (x is not
// modified), or v into v_spec when v_spec != nullptr; with h_out != nullptr
// the embedding h itself.  mf_b = the branch's final (shift, scale), [2H] f32.
bool step_fused_fits(int C, int H, int nb);
int step_fused_partials(int rows, int H, int nb);
hipError_t launch_step_fused(const float* x, int C, const void* W_in, const void* b_in, void* m_out,
                             const void* m_prev, const void* m_last, int rows, int H, const float* sh0,
                             const float* sc0, double* partials, double* out, const void* r, int nb,
                             const void* W_out, const void* b_out, const float* mf0, const float* mf1, float dsig,
                             float guidance, float* x_spec, float* v_spec, void* h_out, hipStream_t s);
// Column-sliced form of the fused step (bf16, C = 64, H % 256 == 0): one
// launch writes m_t (with partials != nullptr its sum |m| into mag[i_new]
// and, with m_prev != nullptr, the four relative-L1 sums into out[4], the
// magnitudes of m_prev and m_last read from mag[i_prev], mag[i_last]), h
// (h_out != nullptr) and, with r != nullptr, per column slice the
// reuse candidate's projection partials into `cand`; a second launch adds
// the slices in a fixed order, applies the factored final LN, the guidance
// combine and the Euler update (x + dsig v into x_spec, x unchanged) or
// writes v into v_spec, and reduces the indicator partials.  The LN
// statistics of h come from S(x) and the statistics matrix st_hi + st_lo
// (step_stream_stats); fc_b = [A | B] of the branch (launch_final_consts).
struct StepStreamDesc {
  const float* x = nullptr; int rows = 0, H = 0;
  const void* W_in = nullptr; const void* b_in = nullptr;
  const void* st_hi = nullptr; const void* st_lo = nullptr; float bbar = 0.f, b2 = 0.f;
  void* m_out = nullptr; const void* m_prev = nullptr; const void* m_last = nullptr;
  const float* sh0 = nullptr; const float* sc0 = nullptr;
  double* partials = nullptr; double* out = nullptr;
  // sum |m| of each of the lane's three indicator buffers (device f64 [3]):
  // the buffer written (i_new) and the two compared (i_prev, i_last)
  double* mag = nullptr; int i_new = 0, i_prev = -1, i_last = -1;
  const void* r = nullptr; int nb = 1;
  const void* W_out = nullptr; const float* mf0 = nullptr; const float* mf1 = nullptr;
  const float* fc0 = nullptr; const float* fc1 = nullptr;
  float* cand = nullptr;
  float dsig = 0.f, guidance = 1.f;
  float* x_spec = nullptr; float* v_spec = nullptr;
  void* h_out = nullptr;
};
bool step_stream_fits(int C, int H, int nb);
// indicator partial 4-vectors and candidate partial floats one launch needs
int step_stream_partials(int rows, int H);
size_t step_stream_cand_floats(int rows, int H, int nb);
// host: the [80][64] statistics matrix (centred Gram matrix of W_in's rows,
// their mean, the bias-row cross term, zero rows) as bf16 hi + lo parts, the
// bias mean and the bias's centred sum of squares; W_in [H][64], b_in [H] bf16.
void step_stream_stats(const uint16_t* W_in, const uint16_t* b_in, int H, uint16_t* hi, uint16_t* lo, float* bbar,
                       float* b2);
hipError_t launch_step_stream(const StepStreamDesc& d, hipStream_t s);
// out[row] = [A_c (64) | B_c (64)] for nrows rows of a modulation table
// (shift at row * ld + off, scale H further): A_c = sum_k (1 + scale_k)
// W_out[c, k], B_c = sum_k shift_k W_out[c, k] + b_out[c]; W_out [64][H] bf16.
hipError_t launch_final_consts(const float* mod, int64_t ld, int off, int nrows, const void* W_out,
                               const void* b_out, int H, float* out, hipStream_t s);
// y = S(LN(S(a + b))(1+sc)+sh) per row (reuse-step final-layer input).
template <typename T>
hipError_t launch_add_ln_mod(const T* a, const T* b, T* out, int rows, int H, const float* sh,
                             const float* sc, hipStream_t s);
// r = S(a - b) (refresh) or r = S(a + b) (reuse), n elements.
template <typename T>
hipError_t launch_add(const T* a, const T* b, T* out, int64_t n, float sign, hipStream_t s);
// x += dsigma * v (batch 1) or x += dsigma * (v_u + g (v_c - v_u)).
// Coefficients of one UniPC step (corrector of x_t, predictor of x_{t+1}).
struct UniCoef {
  int corr;
  float cx, cs, cp, ct;  // x_c = cx x_last + cs m_{t-1} + cp m_{t-2} + ct m_t
  float px, pt, pp;      // x_{t+1} = px x_c + pt m_t + pp m_{t-1}
};
hipError_t launch_unipc(float* x, const float* v_c, const float* v_u, float g, float sig_t, float* x_last,
                        const float* m_s, const float* m_p, float* m_t, const UniCoef& k, int64_t n,
                        hipStream_t s);
hipError_t launch_euler(float* x, const float* v_c, const float* v_u, float g, float dsigma,
                        int64_t n, hipStream_t s);
// latent f32 -> storage type.
template <typename T>
hipError_t launch_cast_from_f32(const float* x, T* out, int64_t n, hipStream_t s);
// Per-head RMS norm in place on columns [0, cols) of rows x ld (f32 path).
hipError_t launch_rms_heads_f32(float* x, int64_t ld, int rows, int cols, int head_dim,
                                hipStream_t s);
// temb[t][k] = S(cos / sin(1000 sigma_t f_k)), f_k = 10000^(-k/half).
template <typename T>
hipError_t launch_time_embed(const double* sigmas, T* out, int T_, int dim, hipStream_t s);
// out[c] = S(mean over rows of x[:, c]).
template <typename T>
hipError_t launch_mean_rows(const T* x, int rows, int cols, T* out, hipStream_t s);
// out[t][c] = S(SiLU(S(a[t][c] + (b ? b[c] : 0)))) with a f32 [rows, cols], b f32 [cols].
template <typename T>
hipError_t launch_vec_silu(const float* a, const float* b, T* out, int rows, int cols,
                           hipStream_t s);
// mod_blk[t][c] = mod[t][base + c] + offset[c] (video blocks), f32.
template <typename T>
hipError_t launch_add_offset(const float* mod, int64_t ld, int base, const T* offset, float* out,
                             int rows, int cols, hipStream_t s);

}  // namespace dit
