// Column-sliced streaming kernels of one sampler step (bf16, 64 latent
// channels, gfx950).
//
// One step of the cached sampler (Eq. 3, Alg. 2) needs, for every image
// token, the patch embedding h = S(S(x) W_in^T + b_in), the first block's
// modulated input m_t = S(LN(h)(1 + scale0) + shift0) with its relative-L1
// sums against m_{t-1} and m_{t_last}, and, should the step be reused, the
// result of the cached residual path: u_b = S(h + r_b), y_b = S(LN(u_b)(1 +
// scale_f,b) + shift_f,b), v_b = y_b W_out^T + b_out, the guidance combine
// and the Euler update.  Every row-wide statistic is what keeps a kernel
// from tiling the hidden dimension, and a work-group that holds whole rows
// must read all of W_in and W_out (two [H, 64] matrices) for a handful of
// tokens.  Here a work-group owns 32 tokens x (128 NW) columns instead:
//
//  * LN statistics of h follow from S(x) alone.  With z_j = s . w_j + b_j
//    (s = S(x), w_j = row j of W_in), sum_j z_j = H (s . wbar + bbar) and
//    sum_j (z_j - zbar)^2 = s^T G s + 2 s . g + B2 with the centred Gram
//    matrix G = sum_j (w_j - wbar)(w_j - wbar)^T, g = sum_j (b_j - bbar)
//    (w_j - wbar) and B2 = sum_j (b_j - bbar)^2, all formed once from the
//    weights (in double, stored as bf16 hi + lo pairs so the MFMA products
//    keep about 16 bits).  The statistics are those of z rather than of its
//    bf16 rounding h; the two differ far below the indicator's tolerance.
//  * The candidate's LN statistics and its projection are additive over
//    columns once factored:  with d_k = u_k - c (c = the token's mean of h,
//    a shift against cancellation), mu_u = c + D1 / H, var_u = D2 / H -
//    (D1 / H)^2 (D1 = sum d_k, D2 = sum d_k^2), and
//      v_c = rho (P_c - (D1 / H) A_c) + B_c,
//      P_c = sum_k S(d_k (1 + scale_k)) W_out[c, k],
//      A_c = sum_k (1 + scale_k) W_out[c, k],  B_c = sum_k shift_k W_out[c, k] + b_out[c],
//    rho = 1 / sqrt(var_u + eps).  Each work-group writes (P, D1, D2) of its
//    column slice; the combine kernel adds the slices in a fixed order.
//    The bf16 operand S(d (1 + scale)) takes the place of the stored y.
//
// Wave layout (16x16x32 bf16 MFMAs): a wave owns two 16-token groups and 128
// columns as four 32-column pairs of MFMA tiles.  The W_in rows of a pair are
// permuted so that lane (lr, lq) of both tiles ends with
// h[token lr][col + 8 lq + 0..7]: one 16-byte chunk of a row, which is the
// layout of the streamed rows (m_{t-1}, m_last, r, m_t) and, as the B operand
// of the projection, exactly what the lane already holds.
#include <math.h>
#include <string.h>

#include <type_traits>
#include <vector>

#include "common.h"
#include "kernels.h"

namespace dit {
namespace {

constexpr int SS_TOK = 32;    // tokens per work-group (two 16-token MFMA groups)
constexpr int SS_COLS = 128;  // h columns per wave (four 32-column tile pairs)
constexpr int SS_C = 64;      // latent channels
constexpr int SS_PART = 66;   // floats per token and slice in the candidate partials: P[64], D1, D2

struct StepStreamArgs {
  const float* x; int rows, H;
  const bf16_t* W_in; const bf16_t* b_in;
  const bf16_t* st_hi; const bf16_t* st_lo;  // [80][64]: G, wbar, g, zero rows
  float bbar, b2;
  bf16_t* m_out; const bf16_t* m_prev; const bf16_t* m_last;
  const float* sh0; const float* sc0;
  double* ind_part;
  const bf16_t* r;
  const bf16_t* W_out;
  const float* mf0; const float* mf1;
  float* cand;
  bf16_t* h_out;
};

// A row of the statistics matrix read by lane row m of statistics tile j:
// tiles 0..3 hold G's rows permuted so that output (lq, i) of tile j is row
// 32 (j / 2) + 8 lq + 4 (j % 2) + i, the column of s the lane holds as element
// 4 (j % 2) + i of its k-block j / 2; tile 4 holds wbar and g (rows 64, 65)
// and zero rows.
__device__ __forceinline__ int stat_row(int j, int m) {
  return j < 4 ? 32 * (j >> 1) + 8 * (m >> 2) + 4 * (j & 1) + (m & 3) : 64 + m;
}

// Sum of the 16 lanes of each row (lanes 16 r .. 16 r + 15) with DPP moves,
// left in every lane of the row: a fixed order, no LDS traffic.
__device__ __forceinline__ float row16_sum(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x141, 0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x140, 0xF, 0xF, false));
  return v;
}

// MODE 0: every part switched by its arguments; MODE 1 / 2: the reuse-candidate
// step with m_t, its sums against m_{t-1} and modulation known at compile
// time (2: m_last is m_{t-1}), so the streamed loads carry no branches.
//
// Two register layouts meet through a per-wave LDS tile of 32 tokens x 128
// columns (rows padded by 16 bytes, which keeps both access patterns free of
// bank conflicts):
//  * MFMA layout: lane (lr, lq) holds columns 32 p + 8 lq .. + 7 of tokens lr
//    and 16 + lr: the embedding's output and the projection's B operand;
//  * streaming layout: lane (sc, sq) = (lane & 15, lane >> 4) holds columns
//    8 sc .. 8 sc + 7 of tokens 4 j + sq, j = 0..7: each load or store
//    instruction covers 256 contiguous bytes of 4 rows (16-row, 64-byte
//    pieces, the MFMA layout's own, stream at about two thirds of the rate).
// h goes from the first layout to the second, the candidate's operand
// S(d (1 + scale_f)) back; the tile then holds the wave's partials.
//
// Indicator sums: a work-group adds |m_t - m_{t-1}|, |m_t| and |m_t - m_last|
// over its tokens; sum |m_{t-1}| and sum |m_last| are the |m| sums of earlier
// steps, kept per indicator buffer by the reduction.
template <int NW, int NB, int MODE>
__global__ __launch_bounds__(64 * NW, (NB == 1 && NW == 4) ? 3 : 2) void step_stream_kernel(StepStreamArgs a) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lq = lane >> 4;  // MFMA layout
  const int sc = lane & 15, sq = lane >> 4;  // streaming layout
  const int H = a.H, rows = a.rows;
  const float invH = 1.f / (float)H;
  const int nsl = H / (SS_COLS * NW);
  const int tile = blockIdx.x / nsl, slice = blockIdx.x - tile * nsl;
  const int row0 = tile * SS_TOK;
  const int lcol = SS_COLS * wave;               // first column of this wave in the slice
  const int colw = slice * SS_COLS * NW + lcol;  // ... in the row
  const bool mpass = MODE ? true : a.m_out != nullptr;
  const bool mod = MODE ? true : a.sc0 != nullptr;
  const bool sums = MODE ? true : a.ind_part != nullptr;
  const bool diffs = MODE ? true : a.m_prev != nullptr;
  const bool spec = MODE ? true : a.r != nullptr;
  const bool same = MODE ? MODE == 2 : a.m_prev == a.m_last;
  const bool stats = mpass || spec;

  constexpr int TRW = SS_COLS + 8;  // bf16 per LDS tile row (272 bytes)
  constexpr int TRB = SS_TOK * TRW * 2;
  static_assert(SS_TOK * SS_PART * 4 <= TRB, "the partials fit the tile");
  __shared__ float vec[2 + NB][SS_COLS * NW];  // 1 + scale0, shift0, then 1 + scale_f of each branch
  __shared__ __attribute__((aligned(16))) float stl[SS_TOK][8];  // per token: four Gram partials, s . wbar, s . g
  __shared__ float red[NW][4];
  constexpr int XSW = SS_C + 8;  // bf16 per row of the S(x) tile (144 bytes: conflict-free fragment reads)
  __shared__ __attribute__((aligned(16))) bf16_t xs[SS_TOK * XSW];
  __shared__ __attribute__((aligned(16))) char trb[NW][TRB];
  bf16_t* tr = (bf16_t*)trb[wave];
  float* cred = (float*)trb[wave];  // [SS_TOK][SS_PART] once the tile is done with
  auto crow = [&](int t) { return (int64_t)min(t, rows - 1); };

  // Load order.  Vector loads return in issue order, so anything loaded after
  // the streamed rows would wait for them, and the compiler, left alone,
  // interleaves loads and waits to save registers.  Scheduling barriers pin
  // the phases: (1) the L2-resident operands of the MFMA work (x once per
  // work-group, W_in and b_in, then, once S(x) is staged in LDS, the
  // statistics tiles and vectors);
  // (2) the embedding and the statistics on MFMAs; (3) the indicator rows;
  // the residual rows follow as the first indicator rows are consumed, and
  // W_out once the candidate's operand is formed.
  // x of the 32 tokens, read once per work-group: 8-float chunks, chunk c =
  // token c / 8, columns 8 (c % 8) .. + 7
  constexpr int XC = SS_TOK * SS_C / 8 / (64 * NW);
  float xr[XC][8];
#pragma unroll
  for (int u = 0; u < XC; ++u) {
    const int c = threadIdx.x + 64 * NW * u;
    load_f8(a.x + crow(row0 + (c >> 3)) * SS_C + 8 * (c & 7), xr[u]);
  }
  uint4 wi[4][2][2];  // W_in rows of the four tile pairs [pair][tile][k-block]
  uint4 bi[4];        // b_in of the lane's columns
#pragma unroll
  for (int p = 0; p < 4; ++p) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16_t* wp = a.W_in + (int64_t)(colw + 32 * p + 8 * (lr >> 2) + 4 * t + (lr & 3)) * SS_C + 8 * lq;
#pragma unroll
      for (int s = 0; s < 2; ++s) wi[p][t][s] = *(const uint4*)(wp + 32 * s);
    }
    bi[p] = *(const uint4*)(a.b_in + colw + 32 * p + 8 * lq);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int u = 0; u < XC; ++u) {  // S(x) into LDS (waits for x only)
    const int c = threadIdx.x + 64 * NW * u;
    *(uint4*)(xs + (c >> 3) * XSW + 8 * (c & 7)) = pack8(xr[u]);
  }
  __builtin_amdgcn_sched_barrier(0);
  // statistics tiles of this wave (w, w + NW, ... < 5), hi and lo parts
  constexpr int NJ = (5 + NW - 1) / NW;
  uint4 sth[NJ][2], stlo[NJ][2];
  if (stats)
#pragma unroll
    for (int u = 0; u < NJ; ++u) {
      const int j = min(wave + NW * u, 4);
      const int64_t so = (int64_t)stat_row(j, lr) * SS_C + 8 * lq;
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        sth[u][s] = *(const uint4*)(a.st_hi + so + 32 * s);
        stlo[u][s] = *(const uint4*)(a.st_lo + so + 32 * s);
      }
    }
  // modulation vectors of the work-group's columns (two elements per thread)
  constexpr int VW = SS_COLS * NW;
  float vk[2][2 + NB];
  if (stats)
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int c = slice * VW + threadIdx.x + 64 * NW * e;
      if (mod) {
        vk[e][0] = a.sc0[c];
        vk[e][1] = a.sh0[c];
      }
      if (spec)
#pragma unroll
        for (int b = 0; b < NB; ++b) vk[e][2 + b] = (b ? a.mf1 : a.mf0)[H + c];
    }
  __builtin_amdgcn_sched_barrier(0);

  lds_barrier();  // the work-group's S(x) tile is in LDS
  uint4 xf[2][2];  // S(x) fragments: the B operand of every MFMA below
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int s = 0; s < 2; ++s) xf[g][s] = *(const uint4*)(xs + (16 * g + lr) * XSW + 32 * s + 8 * lq);
  {
    // the embedding h = S(S(x) W_in^T + b_in): lane (lr, lq) of pair p ends
    // with h[token 16 g + lr][colw + 32 p + 8 lq + 0..7], stored to the tile
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      float bb[8];
      unpack8(bi[p], bb);
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        f32x4_t d0 = {0.f, 0.f, 0.f, 0.f}, d1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          const bf16x8_t xb = __builtin_bit_cast(bf16x8_t, xf[g][s]);
          d0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wi[p][0][s]), xb, d0, 0, 0, 0);
          d1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wi[p][1][s]), xb, d1, 0, 0, 0);
        }
        const float hvals[8] = {d0[0] + bb[0], d0[1] + bb[1], d0[2] + bb[2], d0[3] + bb[3],
                                d1[0] + bb[4], d1[1] + bb[5], d1[2] + bb[6], d1[3] + bb[7]};
        *(uint4*)(tr + (16 * g + lr) * TRW + 32 * p + 8 * lq) = pack8(hvals);
      }
    }
    // LN statistics of the 32 tokens from the statistics tiles
    if (stats)
#pragma unroll
      for (int u = 0; u < NJ; ++u) {
        const int j = wave + NW * u;
        if (j >= 5) break;
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          f32x4_t d = {0.f, 0.f, 0.f, 0.f};
          const bf16x8_t b0 = __builtin_bit_cast(bf16x8_t, xf[g][0]), b1 = __builtin_bit_cast(bf16x8_t, xf[g][1]);
          d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, sth[u][0]), b0, d, 0, 0, 0);
          d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, sth[u][1]), b1, d, 0, 0, 0);
          d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, stlo[u][0]), b0, d, 0, 0, 0);
          d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, stlo[u][1]), b1, d, 0, 0, 0);
          if (j < 4) {
            float sv[8];
            unpack8((j & 2) ? xf[g][1] : xf[g][0], sv);
            const bool hi = (j & 1) != 0;
            float q = ((hi ? sv[4] : sv[0]) * d[0] + (hi ? sv[5] : sv[1]) * d[1]) +
                      ((hi ? sv[6] : sv[2]) * d[2] + (hi ? sv[7] : sv[3]) * d[3]);
            q += __shfl_xor(q, 16, 64);
            q += __shfl_xor(q, 32, 64);
            if (lq == 0) stl[16 * g + lr][j] = q;
          } else if (lq == 0) {
            stl[16 * g + lr][4] = d[0];
            stl[16 * g + lr][5] = d[1];
          }
        }
      }
  }
  __builtin_amdgcn_sched_barrier(0);

  // the indicator rows (streaming layout): m_{t-1} and m_last
  uint4 pv[8], lv[8], rv[8];
  if (diffs)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t o = crow(row0 + 4 * j + sq) * H + colw + 8 * sc;
      pv[j] = ld_stream(a.m_prev + o);
      if (!same) lv[j] = ld_stream(a.m_last + o);
    }
  __builtin_amdgcn_sched_barrier(0);

  if (stats)
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int i = threadIdx.x + 64 * NW * e;
      if (mod) {
        vec[0][i] = 1.f + vk[e][0];
        vec[1][i] = vk[e][1];
      }
      if (spec)
#pragma unroll
        for (int b = 0; b < NB; ++b) vec[2 + b][i] = 1.f + vk[e][2 + b];
    }
  if (stats) lds_barrier();  // statistics, vectors and this wave's h tile are in LDS; the rows stay in flight
  else __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's h tile is in LDS

  uint4 hs[8];  // h in the streaming layout
#pragma unroll
  for (int j = 0; j < 8; ++j) hs[j] = *(const uint4*)(tr + (4 * j + sq) * TRW + 8 * sc);
  if (a.h_out)  // the block stack's input of a computed step
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (row0 + 4 * j + sq < rows) *(uint4*)(a.h_out + (int64_t)(row0 + 4 * j + sq) * H + colw + 8 * sc) = hs[j];
  if (!stats) return;

  const int ntile = gridDim.x / nsl;
  // LN of h for token 4 j + sq of the streaming layout: h ra + rb (mean for the candidate)
  auto tok_stats = [&](int j, float& mean, float& ra, float& rb) {
    const float4 s4 = *(const float4*)&stl[4 * j + sq][0];
    const float2 s2 = *(const float2*)&stl[4 * j + sq][4];
    const float q = ((s4.x + s4.y) + (s4.z + s4.w)) + 2.f * s2.y + a.b2;
    mean = s2.x + a.bbar;
    ra = rsqrtf(fmaxf(q, 0.f) * invH + DIT_LN_EPS);
    rb = -mean * ra;
  };
  const int vc = lcol + 8 * sc;  // the lane's columns in the work-group's vectors
  auto load_r = [&](int b, int j) {
    rv[j] = ld_stream(a.r + (int64_t)b * rows * H + crow(row0 + 4 * j + sq) * H + colw + 8 * sc);
  };

  // (a1, a2) m_t and the relative-L1 sums; the residual rows of branch 0 are
  // requested as soon as the first half of the indicator rows is consumed
  float s0 = 0.f, s1 = 0.f, s2 = 0.f;
  if (mpass) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int t = row0 + 4 * j + sq;
      float mean, ra, rb;
      tok_stats(j, mean, ra, rb);
      float y[8];
      unpack8(hs[j], y);
      if (mod) {
        float k[8], dsh[8];  // read per row: fewer live registers
        load_f8(&vec[0][vc], k);
        load_f8(&vec[1][vc], dsh);
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = fmaf(fmaf(y[e], ra, rb), k[e], dsh[e]);
      }
      const uint4 mt = pack8(y);
      if (t < rows) {
        st_stream(a.m_out + (int64_t)t * H + colw + 8 * sc, mt);
        if (sums) {
          float mv[8];
          unpack8(mt, mv);
          if (diffs) {
            float pp[8], ll[8];
            unpack8(pv[j], pp);
            if (same) {
#pragma unroll
              for (int e = 0; e < 8; ++e) ll[e] = pp[e];
            } else {
              unpack8(lv[j], ll);
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              s0 += fabsf(mv[e] - pp[e]);
              s2 += fabsf(mv[e] - ll[e]);
            }
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) s1 += fabsf(mv[e]);
        }
      }
      if (spec && (j == 4 || j == 7))  // residual rows as the indicator rows are consumed
#pragma unroll
        for (int i = (j == 4 ? 0 : 4); i < (j == 4 ? 4 : 8); ++i) load_r(0, i);
    }
  } else if (spec) {
#pragma unroll
    for (int i = 0; i < 8; ++i) load_r(0, i);
  }

  // (a4, a5) the candidate, one branch at a time: d = S(h + r) - mean summed
  // (d1) and squared (d2) per token, S(d (1 + scale_f)) back into the tile in
  // place of h, then the tile in the MFMA layout projected on W_out
  f32x4_t acc[2][4];
  uint4 wo[4][4];  // W_out[16 ct + lr][colw + 32 p + 8 lq + 0..7] (MFMA layout)
  auto pass = [&](auto bc) {
    constexpr int b = decltype(bc)::value;
    float kf[8];
    load_f8(&vec[2 + b][vc], kf);
    float d1[8], d2[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float mean, ra, rb;
      tok_stats(j, mean, ra, rb);
      float hf[8], rf[8], u[8], dk[8];
      unpack8(hs[j], hf);
      unpack8(rv[j], rf);
#pragma unroll
      for (int e = 0; e < 8; ++e) u[e] = hf[e] + rf[e];
      unpack8(pack8(u), u);  // u = S(h + r)
      float q1 = 0.f, q2 = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = u[e] - mean;
        q1 += d;
        q2 = fmaf(d, d, q2);
        dk[e] = d * kf[e];
      }
      d1[j] = q1;
      d2[j] = q2;
      *(uint4*)(tr + (4 * j + sq) * TRW + 8 * sc) = pack8(dk);
      if (b + 1 < NB) load_r(b + 1, j);  // the next branch's rows into the freed registers
    }
#pragma unroll
    for (int p = 0; p < 4; ++p)
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
        wo[p][ct] = *(const uint4*)(a.W_out + (int64_t)(16 * ct + lr) * H + colw + 32 * p + 8 * lq);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      d1[j] = row16_sum(d1[j]);
      d2[j] = row16_sum(d2[j]);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the operand tile is written
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) acc[g][ct] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < 4; ++p)
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const uint4 ub = *(const uint4*)(tr + (16 * g + lr) * TRW + 32 * p + 8 * lq);
#pragma unroll
        for (int ct = 0; ct < 4; ++ct)
          acc[g][ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wo[p][ct]),
                                                               __builtin_bit_cast(bf16x8_t, ub), acc[g][ct], 0, 0, 0);
      }
    // the wave's partials into its tile: lane (lr, lq) holds P[token 16 g + lr][16 ct + 4 lq + i]
    __builtin_amdgcn_s_waitcnt(0xc07f);  // the operand reads of this wave are done
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
#pragma unroll
        for (int i = 0; i < 4; ++i) cred[(16 * g + lr) * SS_PART + 16 * ct + 4 * lq + i] = acc[g][ct][i];
    if (sc == 0)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        cred[(4 * j + sq) * SS_PART + 64] = d1[j];
        cred[(4 * j + sq) * SS_PART + 65] = d2[j];
      }
  };
  // the work-group's sum over its waves, in wave order, to the slice's partials
  auto from_lds = [&](int b) {
    float* out = a.cand + (((int64_t)b * nsl + slice) * ntile * SS_TOK + row0) * SS_PART;
    for (int i = threadIdx.x; i < SS_TOK * SS_PART; i += 64 * NW) {
      float v = ((const float*)trb[0])[i];
#pragma unroll
      for (int w = 1; w < NW; ++w) v += ((const float*)trb[w])[i];
      out[i] = v;
    }
  };

  if (spec) {
    pass(std::integral_constant<int, 0>());
    if (NB == 2) {
      lds_barrier();
      from_lds(0);
      lds_barrier();  // every thread has read branch 0's partials before the tiles are reused
      pass(std::integral_constant<int, NB - 1>());
    }
  }
  if (sums) {
    s0 = warp_sum(s0); s1 = warp_sum(s1); s2 = warp_sum(s2);
    if (lane == 0) { red[wave][0] = s0; red[wave][1] = s1; red[wave][2] = s2; }
  }
  if (!spec && !sums) return;
  lds_barrier();
  if (spec) from_lds(NB - 1);
  if (sums && threadIdx.x < 4) {
    double t = 0.0;
    if (threadIdx.x < 3)
#pragma unroll
      for (int w = 0; w < NW; ++w) t += (double)red[w][threadIdx.x];
    a.ind_part[(int64_t)blockIdx.x * 4 + threadIdx.x] = t;
  }
}

struct CombineArgs {
  const float* cand; int rows, nsl, ntile, H, nb;
  const float* fc0; const float* fc1;  // [2][64]: A_c, B_c of each branch
  const float* x; float* x_spec; float* v_spec; float dsig, guidance;
  const double* ind_part; int n_ind; double* ind_out;
  double* mag; int i_new, i_prev, i_last;  // sum |m| of each indicator buffer; out only with i_prev >= 0
  int cand_blocks;  // work-groups that combine candidates (the last one, if any more, reduces the sums)
};

// Candidate combine (one work-group per 32 tokens: 8 threads per token, 8
// output channels each; a token's slice partials are 264 contiguous bytes)
// and the fixed-order reduction of the indicator partials into host-mapped
// memory (the last work-group).  Both read their inputs in groups whose loads
// are all issued before the first add (CB_SL slices, RD_U entries per
// thread), clamped to the last valid index and discarded by a select; the
// additions keep one thread's sequential order, so the result does not depend
// on the group sizes.
constexpr int CB_TOK = 32;
constexpr int CB_SL = 6;
constexpr int RD_U = 8;
__global__ __launch_bounds__(256) void step_combine_kernel(CombineArgs a) {
  if ((int)blockIdx.x == a.cand_blocks) {
    __shared__ double sred[4][256];
    double acc[4] = {0, 0, 0, 0};
    for (int i0 = threadIdx.x; i0 < a.n_ind; i0 += 256 * RD_U) {
      double v[RD_U][4];
#pragma unroll
      for (int u = 0; u < RD_U; ++u) {
        const double* q = a.ind_part + (int64_t)min(i0 + 256 * u, a.n_ind - 1) * 4;
#pragma unroll
        for (int c = 0; c < 4; ++c) v[u][c] = q[c];
      }
#pragma unroll
      for (int u = 0; u < RD_U; ++u) {
        const bool ok = i0 + 256 * u < a.n_ind;
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c] = ok ? acc[c] + v[u][c] : acc[c];
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) sred[c][threadIdx.x] = acc[c];
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if ((int)threadIdx.x < w)
#pragma unroll
        for (int c = 0; c < 4; ++c) sred[c][threadIdx.x] += sred[c][threadIdx.x + w];
      __syncthreads();
    }
    // raw sums |m_t - m_{t-1}|, |m_t|, |m_t - m_last|; the magnitudes of the
    // older tensors were recorded when they were written
    if (threadIdx.x == 0) {
      const double m_new = sred[1][0];
      if (a.i_prev >= 0) {
        a.ind_out[0] = sred[0][0];
        a.ind_out[1] = a.mag[a.i_prev];
        a.ind_out[2] = sred[2][0];
        a.ind_out[3] = a.mag[a.i_last];
      }
      a.mag[a.i_new] = m_new;
    }
    __threadfence_system();
    return;
  }
  const int tl = threadIdx.x >> 3, c0 = 8 * (threadIdx.x & 7);
  const int tok = blockIdx.x * CB_TOK + tl;
  if (tok >= a.rows) return;
  const int64_t o = (int64_t)tok * SS_C + c0;
  float xv[8];
  if (!a.v_spec) load_f8(a.x + o, xv);
  const float invH = 1.f / (float)a.H;
  const int64_t sstride = (int64_t)a.ntile * SS_TOK * SS_PART;
  float vres[8];
  for (int b = 0; b < a.nb; ++b) {
    const float* base = a.cand + ((int64_t)b * a.nsl * a.ntile * SS_TOK + tok) * SS_PART;
    const float* fc = b ? a.fc1 : a.fc0;
    float A[8], B[8];
    load_f8(fc + c0, A);
    load_f8(fc + SS_C + c0, B);
    float P[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    float D1 = 0.f, D2 = 0.f;
    for (int s0 = 0; s0 < a.nsl; s0 += CB_SL) {
      float v[CB_SL][8];
      float2 dd[CB_SL];
#pragma unroll
      for (int u = 0; u < CB_SL; ++u) {
        const float* q = base + min(s0 + u, a.nsl - 1) * sstride;
        load_f8(q + c0, v[u]);
        dd[u] = *(const float2*)(q + 64);
      }
#pragma unroll
      for (int u = 0; u < CB_SL; ++u) {
        const bool ok = s0 + u < a.nsl;
#pragma unroll
        for (int e = 0; e < 8; ++e) P[e] = ok ? P[e] + v[u][e] : P[e];
        D1 = ok ? D1 + dd[u].x : D1;
        D2 = ok ? D2 + dd[u].y : D2;
      }
    }
    const float dm = D1 * invH;
    const float rho = rsqrtf(fmaxf(D2 * invH - dm * dm, 0.f) + DIT_LN_EPS);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float v = rho * (P[e] - dm * A[e]) + B[e];
      // guidance: v = v_u + g (v_c - v_u), branch 0 conditional, branch 1 unconditional
      vres[e] = b == 0 ? v : v + a.guidance * (vres[e] - v);
    }
  }
  if (a.v_spec) {
    *(float4*)(a.v_spec + o) = make_float4(vres[0], vres[1], vres[2], vres[3]);
    *(float4*)(a.v_spec + o + 4) = make_float4(vres[4], vres[5], vres[6], vres[7]);
  } else {
    *(float4*)(a.x_spec + o) = make_float4(xv[0] + a.dsig * vres[0], xv[1] + a.dsig * vres[1],
                                           xv[2] + a.dsig * vres[2], xv[3] + a.dsig * vres[3]);
    *(float4*)(a.x_spec + o + 4) = make_float4(xv[4] + a.dsig * vres[4], xv[5] + a.dsig * vres[5],
                                               xv[6] + a.dsig * vres[6], xv[7] + a.dsig * vres[7]);
  }
}

// A_c = sum_k (1 + scale_k) W_out[c, k], B_c = sum_k shift_k W_out[c, k] + b_out[c]
// for every row of the modulation table (shift at mod + off, scale H further);
// one work-group per table row, each wave 16 output channels.
__global__ __launch_bounds__(256) void final_consts_kernel(const float* __restrict__ mod, int64_t ld, int off,
                                                           const bf16_t* __restrict__ W, const bf16_t* __restrict__ bo,
                                                           int H, float* __restrict__ out) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* sh = mod + (int64_t)blockIdx.x * ld + off;
  const float* sc = sh + H;
  for (int c = wave * 16; c < wave * 16 + 16; ++c) {
    float sa = 0.f, sb = 0.f;
    for (int k = 8 * lane; k < H; k += 512) {
      float w[8], k1[8], k2[8];
      unpack8(*(const uint4*)(W + (int64_t)c * H + k), w);
      load_f8(sc + k, k1);
      load_f8(sh + k, k2);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sa += (1.f + k1[e]) * w[e];
        sb += k2[e] * w[e];
      }
    }
    sa = warp_sum(sa);
    sb = warp_sum(sb);
    if (lane == 0) {
      out[(int64_t)blockIdx.x * 2 * SS_C + c] = sa;
      out[(int64_t)blockIdx.x * 2 * SS_C + SS_C + c] = sb + bf16_to_f32(bo[c]);
    }
  }
}

// Waves per work-group: 4 (512 columns) where they divide H, else 2.
int stream_waves(int H) {
  if (H < 2 * SS_COLS || H % (2 * SS_COLS)) return 0;
  return (H / SS_COLS) % 4 == 0 ? 4 : 2;
}

}  // namespace

bool step_stream_fits(int C, int H, int nb) { return C == SS_C && stream_waves(H) > 0 && nb >= 1 && nb <= 2; }

int step_stream_partials(int rows, int H) {
  const int nw = stream_waves(H);
  return nw ? (rows + SS_TOK - 1) / SS_TOK * (H / (SS_COLS * nw)) : 0;
}

size_t step_stream_cand_floats(int rows, int H, int nb) {
  const int nw = stream_waves(H);
  if (!nw) return 0;
  return (size_t)nb * (H / (SS_COLS * nw)) * ((rows + SS_TOK - 1) / SS_TOK) * SS_TOK * SS_PART;
}

void step_stream_stats(const uint16_t* W_in, const uint16_t* b_in, int H, uint16_t* hi, uint16_t* lo, float* bbar,
                       float* b2) {
  auto f = [](uint16_t u) {
    uint32_t v = (uint32_t)u << 16;
    float r;
    memcpy(&r, &v, 4);
    return (double)r;
  };
  auto rne = [](float v) -> uint16_t {
    uint32_t u;
    memcpy(&u, &v, 4);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
  };
  auto back = [](uint16_t u) {
    uint32_t v = (uint32_t)u << 16;
    float r;
    memcpy(&r, &v, 4);
    return r;
  };
  constexpr int C = SS_C;
  std::vector<double> wbar(C, 0.0), g(C, 0.0), G((size_t)C * C, 0.0), wc(C);
  double bsum = 0.0;
  for (int j = 0; j < H; ++j) {
    bsum += f(b_in[j]);
    for (int k = 0; k < C; ++k) wbar[k] += f(W_in[(size_t)j * C + k]);
  }
  const double bm = bsum / H;
  for (double& v : wbar) v /= H;
  double bb2 = 0.0;
  for (int j = 0; j < H; ++j) {
    const double bc = f(b_in[j]) - bm;
    bb2 += bc * bc;
    for (int k = 0; k < C; ++k) wc[k] = f(W_in[(size_t)j * C + k]) - wbar[k];
    for (int k = 0; k < C; ++k) g[k] += bc * wc[k];
    for (int n = 0; n < C; ++n)
      for (int k = 0; k < C; ++k) G[(size_t)n * C + k] += wc[n] * wc[k];
  }
  std::vector<double> m((size_t)80 * C, 0.0);
  for (size_t i = 0; i < (size_t)C * C; ++i) m[i] = G[i];
  for (int k = 0; k < C; ++k) {
    m[(size_t)64 * C + k] = wbar[k];
    m[(size_t)65 * C + k] = g[k];
  }
  for (size_t i = 0; i < m.size(); ++i) {
    hi[i] = rne((float)m[i]);
    lo[i] = rne((float)(m[i] - (double)back(hi[i])));
  }
  *bbar = (float)bm;
  *b2 = (float)bb2;
}

hipError_t launch_step_stream(const StepStreamDesc& d, hipStream_t s) {
  const int nw = stream_waves(d.H);
  if (!step_stream_fits(SS_C, d.H, d.nb) || d.rows < 1) return hipErrorInvalidValue;
  // the embedding runs on every launch; the modulation is a shift and a scale together
  if (!d.x || !d.W_in || !d.b_in || (d.sh0 == nullptr) != (d.sc0 == nullptr) || (d.m_prev && !d.m_last))
    return hipErrorInvalidValue;
  // sums need m_t and the magnitude record; differences need the sums and the host-mapped output
  if ((d.partials && (!d.m_out || !d.mag || d.i_new < 0 || d.i_new > 2)) ||
      (d.m_prev && (!d.partials || !d.out || d.i_prev < 0 || d.i_prev > 2 || d.i_last < 0 || d.i_last > 2)))
    return hipErrorInvalidValue;
  if (d.r && (!d.cand || !d.W_out || !d.fc0 || (d.nb == 2 && (!d.fc1 || !d.mf1)) || !d.mf0 || (!d.x_spec && !d.v_spec)))
    return hipErrorInvalidValue;
  if ((d.m_out || d.r) && (!d.st_hi || !d.st_lo)) return hipErrorInvalidValue;
  const int nsl = d.H / (SS_COLS * nw), ntile = (d.rows + SS_TOK - 1) / SS_TOK;
  StepStreamArgs a{d.x, d.rows, d.H, (const bf16_t*)d.W_in, (const bf16_t*)d.b_in, (const bf16_t*)d.st_hi,
                   (const bf16_t*)d.st_lo, d.bbar, d.b2, (bf16_t*)d.m_out, (const bf16_t*)d.m_prev,
                   (const bf16_t*)d.m_last, d.sh0, d.sc0, d.partials, (const bf16_t*)d.r, (const bf16_t*)d.W_out,
                   d.mf0, d.mf1, d.cand, (bf16_t*)d.h_out};
  const dim3 grid(ntile * nsl);
  const bool two = d.r && d.nb == 2;
  // the reuse-candidate step with modulated m_t and sums takes the branch-free instances
  const int mode = (d.r && d.m_out && d.sc0 && d.partials && d.m_prev) ? (d.m_prev == d.m_last ? 2 : 1) : 0;
  auto go = [&](auto nw, auto nbc) {
    constexpr int NW = decltype(nw)::value, NB = decltype(nbc)::value;
    if (mode == 1) hipLaunchKernelGGL((step_stream_kernel<NW, NB, 1>), grid, dim3(64 * NW), 0, s, a);
    else if (mode == 2) hipLaunchKernelGGL((step_stream_kernel<NW, NB, 2>), grid, dim3(64 * NW), 0, s, a);
    else hipLaunchKernelGGL((step_stream_kernel<NW, NB, 0>), grid, dim3(64 * NW), 0, s, a);
  };
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I4 = std::integral_constant<int, 4>;
  if (nw == 4) { if (two) go(I4(), I2()); else go(I4(), I1()); }
  else { if (two) go(I2(), I2()); else go(I2(), I1()); }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int cb = d.r ? (d.rows + CB_TOK - 1) / CB_TOK : 0;
  if (cb == 0 && !d.partials) return hipSuccess;
  CombineArgs c{d.cand, d.rows, nsl, ntile, d.H, d.nb, d.fc0, d.fc1, d.x, d.x_spec, d.v_spec, d.dsig,
                d.guidance, d.partials, ntile * nsl, d.out, d.mag, d.i_new, d.m_prev ? d.i_prev : -1, d.i_last, cb};
  hipLaunchKernelGGL(step_combine_kernel, dim3(cb + (d.partials ? 1 : 0)), dim3(256), 0, s, c);
  return hipGetLastError();
}

hipError_t launch_final_consts(const float* mod, int64_t ld, int off, int nrows, const void* W_out,
                               const void* b_out, int H, float* out, hipStream_t s) {
  if (H % 8) return hipErrorInvalidValue;
  if (nrows < 1) return hipSuccess;
  hipLaunchKernelGGL(final_consts_kernel, dim3(nrows), dim3(256), 0, s, mod, ld, off, (const bf16_t*)W_out,
                     (const bf16_t*)b_out, H, out);
  return hipGetLastError();
}

}  // namespace dit
