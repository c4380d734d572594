// Fused per-step kernels of the cached sampler's streaming path (bf16,
// gfx950): the patch embedding is recomputed inside each kernel instead of
// being stored, so a reuse step moves only what the method needs.
//
//  * reuse_indicator_kernel  (a1 + a2 of every step)
//      h = S(S(x) W_in^T + b_in) for a tile of RR token rows, on MFMA into
//      LDS; then per row m_t = S(LN(h)(1 + scale0) + shift0) is written and
//      the relative-L1 sums against m_{t-1} and m_{t_last} accumulated
//      (f64 partials per workgroup, reduced in a fixed order afterwards).
//      With h_out != nullptr it writes h instead (the full step's block-stack
//      input, bit-identical to the h the indicator saw).
//  * reuse_final_kernel  (a4 reuse + a5)
//      per branch: h_out = S(h + r), y = S(LN(h_out)(1 + scale_f) + shift_f)
//      into LDS, v = y W_out^T + b_out on MFMA, guidance combine, and the
//      Euler update x += dsigma v in place.
// HBM traffic of a reuse step: read m_{t-1}, m_{t_last} (once if equal) and
// r, write m_t, plus the latent (N x C f32) and the L2-resident embedding /
// projection weights.
#include <math.h>

#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace dit {
namespace {

constexpr int RR = 16;  // token rows per workgroup (the MFMA's 16 token lanes)
constexpr int RW = 8;   // waves per workgroup
constexpr int LPAD = 8; // bf16 elements of padding per LDS row (16 bytes)
#ifndef EMBED_EB
#define EMBED_EB 8
#endif

// Copies n16 16-byte vectors global -> LDS with the whole workgroup; every
// thread issues its loads (up to 8 in flight) before its stores.
__device__ __forceinline__ void stage(const void* src, void* dst, int n16) {
  constexpr int NT = 64 * RW, U = 4;
  for (int i0 = threadIdx.x; i0 < n16; i0 += NT * U) {
    uint4 v[U];
    // indices clamped instead of tested: no branches, so all loads issue
    // before the first store (clamped duplicates store the same value twice)
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = ((const uint4*)src)[min(i0 + u * NT, n16 - 1)];
#pragma unroll
    for (int u = 0; u < U; ++u) ((uint4*)dst)[min(i0 + u * NT, n16 - 1)] = v[u];
  }
}

// h rows row0 .. row0 + RR - 1 into LDS (row stride ldl): the transposed
// product h^T = W_in S(x)^T on 16x16x32 MFMAs, 16 h-columns per tile (bias
// b_in read from its LDS copy bl); the
// operand's 16 token lanes cover the RR rows (lanes past them repeat the
// last valid row and are not stored).  Lane (lr, lq) ends with
// h[row lr][16 j + 4 lq + i], i = 0..3: one 8-byte LDS store.
template <int CK, int EB, int TR = RR>
__device__ __forceinline__ void embed_to_lds(const float* __restrict__ x, int C, const bf16_t* __restrict__ W,
                                             const bf16_t* bl, int row0, int rows, int H, bf16_t* hl, int ldl,
                                             int wave, int lane) {
  static_assert(TR <= 16, "the MFMA has 16 token lanes");
  const int lr = lane & 15, lq = lane >> 4;
  const int xr = min(row0 + min(lr, TR - 1), rows - 1);
  bf16x8_t xf[CK];
#pragma unroll
  for (int s = 0; s < CK; ++s) {
    float v[8];
    load_f8(x + (int64_t)xr * C + 32 * s + 8 * lq, v);
    xf[s] = __builtin_bit_cast(bf16x8_t, pack8(v));
  }
  const bool store = lr < TR && row0 + lr < rows;
  // W_in tiles stream from L2 in batches of EB, the next batch in flight
  // while the current one is multiplied and stored
  // Each wave takes a contiguous run of tiles when they divide evenly (its
  // W_in rows then spread over every L2 channel), else tiles wave + RW u.
  const int ntile = H / 16;
  const bool contig = ntile % RW == 0;
  const int nu = contig ? ntile / RW : (ntile - wave + RW - 1) / RW;
  uint4 wcur[EB][CK], wnxt[EB][CK];
  // every workgroup walks its tiles from a different start, so the CUs of an
  // XCD do not all request the same L2 lines at the same time
  const int rot = blockIdx.x % nu;
  auto tile_of = [&](int u) {
    const int v = u + rot, w = v < nu ? v : v - nu;
    return contig ? wave * nu + w : wave + RW * w;
  };
  auto load_batch = [&](int u0, uint4 (&w)[EB][CK]) {
#pragma unroll
    for (int e = 0; e < EB; ++e) {
      const int u = min(u0 + e, nu - 1);
      const bf16_t* wp = W + (int64_t)(16 * tile_of(u) + lr) * C + 8 * lq;
#pragma unroll
      for (int s = 0; s < CK; ++s) w[e][s] = *(const uint4*)(wp + 32 * s);
    }
  };
  load_batch(0, wcur);
  for (int u0 = 0; u0 < nu; u0 += EB) {
    if (u0 + EB < nu) load_batch(u0 + EB, wnxt);
#pragma unroll
    for (int e = 0; e < EB; ++e) {
      if (u0 + e >= nu) break;
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < CK; ++s)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wcur[e][s]), xf[s], acc, 0, 0, 0);
      if (store) {
        const int n = 16 * tile_of(u0 + e) + 4 * lq;
        const uint2 bb = *(const uint2*)(bl + n);
        const float b0 = __uint_as_float(bb.x << 16), b1 = __uint_as_float(bb.x & 0xffff0000u);
        const float b2 = __uint_as_float(bb.y << 16), b3 = __uint_as_float(bb.y & 0xffff0000u);
        *(uint2*)(hl + lr * ldl + n) =
            make_uint2(pack_bf16x2(acc[0] + b0, acc[1] + b1), pack_bf16x2(acc[2] + b2, acc[3] + b3));
      }
    }
#pragma unroll
    for (int e = 0; e < EB; ++e)
#pragma unroll
      for (int s = 0; s < CK; ++s) wcur[e][s] = wnxt[e][s];
  }
}

// LN statistics of one row held as MAXC 8-value chunks per lane (chunks
// c = lane + 64 j < nch); two passes over registers, f32.
template <int MAXC>
__device__ __forceinline__ void row_stats(const float (&v)[MAXC][8], int nch, int H, int lane, float& mean,
                                          float& rstd) {
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < MAXC; ++j)
#pragma unroll
    for (int e = 0; e < 8; ++e) s += v[j][e];
  mean = warp_sum(s) / (float)H;
  float q = 0.f;
#pragma unroll
  for (int j = 0; j < MAXC; ++j) {
    if (lane + 64 * j < nch)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = v[j][e] - mean;
        q += d * d;
      }
  }
  rstd = rsqrtf(warp_sum(q) / (float)H + DIT_LN_EPS);
}

template <int CK, int MAXC>
__global__ __launch_bounds__(64 * RW) void reuse_indicator_kernel(
    const float* __restrict__ x, int C, const bf16_t* __restrict__ W_in, const bf16_t* __restrict__ b_in,
    bf16_t* __restrict__ m_out, const bf16_t* __restrict__ m_prev, const bf16_t* __restrict__ m_last,
    int rows, int H, const float* __restrict__ sh, const float* __restrict__ sc, double* __restrict__ partials,
    bf16_t* __restrict__ h_out) {
  // dynamic LDS: h tile [RR][H + LPAD] bf16, then b_in [H] bf16, then scale / shift [H] f32
  extern __shared__ __attribute__((aligned(16))) bf16_t hl[];
  __shared__ float red[RW][4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row0 = blockIdx.x * RR;
  const int ldl = H + LPAD, nch = H / 8;
  constexpr int RPW = RR / RW;  // rows per wave
  const bool sums = partials != nullptr && h_out == nullptr;
  bf16_t* bl = hl + RR * ldl;
  float* scl = (float*)(bl + H);
  float* shl = scl + H;
  stage(b_in, bl, H / 8);
  if (sc && !h_out) {
    stage(sc, scl, H / 4);
    stage(sh, shl, H / 4);
  }
  const bool same = m_prev == m_last;
  lds_barrier();
  embed_to_lds<CK, EMBED_EB>(x, C, W_in, bl, row0, rows, H, hl, ldl, wave, lane);

  // The previous indicator rows are requested only now: vector loads retire
  // in issue order, so had they been issued before the embedding, its first
  // wait for W_in would have waited for them too.  They stream in while m_t
  // is computed and stored (addresses clamped into the tensors so every load
  // is unconditional and they all issue back to back; out-of-range chunks
  // and rows are not used).
  uint4 pv[RPW][MAXC], lv[RPW][MAXC];
  if (sums) {
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
      const int row = min(row0 + wave + RW * q, rows - 1);
#pragma unroll
      for (int j = 0; j < MAXC; ++j) {
        const int c = min(lane + 64 * j, nch - 1);
        pv[q][j] = ld_stream(m_prev + (int64_t)row * H + 8 * c);
        if (!same) lv[q][j] = ld_stream(m_last + (int64_t)row * H + 8 * c);
      }
    }
  }
  lds_barrier();  // the h tile is complete; the row loads stay in flight

  // pass 1: m_t rows (or h rows on a full step), values kept for the sums
  uint4 mt[RPW][MAXC];
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const int rr = wave + RW * q, row = row0 + rr;
    const bf16_t* src = hl + rr * ldl;
    if (h_out) {  // block-stack input of a full step
      if (row >= rows) continue;
#pragma unroll
      for (int j = 0; j < MAXC; ++j) {
        const int c = lane + 64 * j;
        if (c < nch) *(uint4*)(h_out + (int64_t)row * H + 8 * c) = *(const uint4*)(src + 8 * c);
      }
      continue;
    }
    float v[MAXC][8];
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = lane + 64 * j;
      unpack8(*(const uint4*)(src + 8 * min(c, nch - 1)), v[j]);
      if (c >= nch)
#pragma unroll
        for (int e = 0; e < 8; ++e) v[j][e] = 0.f;
    }
    float mean = 0.f, rstd = 1.f;
    if (sc) row_stats<MAXC>(v, nch, H, lane, mean, rstd);
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = lane + 64 * j;
      float y[8];
      if (sc) {
        float a[8], bsh[8];
        load_f8(scl + 8 * min(c, nch - 1), a);
        load_f8(shl + 8 * min(c, nch - 1), bsh);
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = (v[j][e] - mean) * rstd * (1.f + a[e]) + bsh[e];
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = v[j][e];
      }
      mt[q][j] = pack8(y);
      if (c < nch && row < rows) st_stream(m_out + (int64_t)row * H + 8 * c, mt[q][j]);
    }
  }
  if (!sums) return;
  // pass 2: relative-L1 sums against the stored (rounded) m_t
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const int row = row0 + wave + RW * q;
    if (row >= rows) break;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = lane + 64 * j;
      if (c >= nch) continue;
      float mv[8], p[8], l[8];
      unpack8(mt[q][j], mv);
      unpack8(pv[q][j], p);
      if (same) {
#pragma unroll
        for (int e = 0; e < 8; ++e) l[e] = p[e];
      } else {
        unpack8(lv[q][j], l);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        a0 += fabsf(mv[e] - p[e]);
        a1 += fabsf(p[e]);
        a2 += fabsf(mv[e] - l[e]);
        a3 += fabsf(l[e]);
      }
    }
  }
  a0 = warp_sum(a0); a1 = warp_sum(a1); a2 = warp_sum(a2); a3 = warp_sum(a3);
  if (lane == 0) { red[wave][0] = a0; red[wave][1] = a1; red[wave][2] = a2; red[wave][3] = a3; }
  __syncthreads();
  if (threadIdx.x < 4) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < RW; ++w) s += (double)red[w][threadIdx.x];
    partials[(int64_t)blockIdx.x * 4 + threadIdx.x] = s;
  }
}

template <int CK, int MAXC, int NT>
__global__ __launch_bounds__(64 * RW) void reuse_final_kernel(
    float* __restrict__ x, int C, const bf16_t* __restrict__ W_in, const bf16_t* __restrict__ b_in,
    const bf16_t* __restrict__ r, int nb, const bf16_t* __restrict__ W_out, const bf16_t* __restrict__ b_out,
    const float* mod0, const float* mod1, float dsig, float guidance, int rows, int H, float* __restrict__ vout) {
  // dynamic LDS: h / y tile [RR][H + LPAD] bf16, then b_in [H] bf16, then scale / shift [H] f32
  extern __shared__ __attribute__((aligned(16))) bf16_t hl[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lq = lane >> 4;
  const int row0 = blockIdx.x * RR;
  const int ldl = H + LPAD, nch = H / 8;
  bf16_t* bl = hl + RR * ldl;
  float* scl = (float*)(bl + H);
  float* shl = scl + H;
  constexpr int RPW = RR / RW;
  static_assert(RW % NT == 0, "projection tiles divide the waves");
  constexpr int KS = RW / NT;  // waves per projection tile
  __shared__ float vpart[RW][64][4];
  float vres[4] = {0.f, 0.f, 0.f, 0.f};

  for (int b = 0; b < nb; ++b) {
    const bf16_t* rb = r + (int64_t)b * rows * H;
    const float* mod = b ? mod1 : mod0;
    uint4 rv[RPW][MAXC];  // clamped, unconditional loads (see the indicator kernel)
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
      const int row = min(row0 + wave + RW * q, rows - 1);
#pragma unroll
      for (int j = 0; j < MAXC; ++j) rv[q][j] = ld_stream(rb + (int64_t)row * H + 8 * min(lane + 64 * j, nch - 1));
    }
    if (b) lds_barrier();  // the previous branch's projection is done with the tile
    if (b == 0) stage(b_in, bl, H / 8);
    stage(mod + H, scl, H / 4);
    stage(mod, shl, H / 4);
    lds_barrier();
    embed_to_lds<CK, 4>(x, C, W_in, bl, row0, rows, H, hl, ldl, wave, lane);
    lds_barrier();
    // h_out = S(h + r), y = S(LN(h_out)(1 + sc) + sh), in place
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
      const int rr = wave + RW * q, row = row0 + rr;
      if (row >= rows) break;
      bf16_t* src = hl + rr * ldl;
      float v[MAXC][8];
#pragma unroll
      for (int j = 0; j < MAXC; ++j) {
        const int c = lane + 64 * j;
        float hv[8], rvv[8];
        unpack8(*(const uint4*)(src + 8 * min(c, nch - 1)), hv);
        unpack8(rv[q][j], rvv);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[j][e] = c < nch ? St<bf16_t>::rd(hv[e] + rvv[e]) : 0.f;
      }
      float mean, rstd;
      row_stats<MAXC>(v, nch, H, lane, mean, rstd);
#pragma unroll
      for (int j = 0; j < MAXC; ++j) {
        const int c = lane + 64 * j;
        if (c >= nch) continue;
        float a[8], bsh[8], y[8];
        load_f8(scl + 8 * c, a);
        load_f8(shl + 8 * c, bsh);
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = (v[j][e] - mean) * rstd * (1.f + a[e]) + bsh[e];
        *(uint4*)(src + 8 * c) = pack8(y);
      }
    }
    lds_barrier();
    // v^T = W_out y^T: lane (lr, lq) of tile j ends with v[row lr][16 j + 4 lq + i].
    // KS waves share a tile, each a contiguous K range; partial sums meet in
    // LDS and are added in wave order.
    {
      const int j = wave % NT, part = wave / NT;
      const int ks = H / 32, per = ks / KS;  // H % (32 KS) == 0 (checked on the host)
      const int s0 = part * per;
      const int rot = (blockIdx.x * 8) % per;  // staggered start, as in the embedding
      auto ks_of = [&](int q) { const int v = q + rot; return s0 + (v < per ? v : v - per); };
      const bf16_t* wp = W_out + (int64_t)(16 * j + lr) * H + 8 * lq;
      const bf16_t* yp = hl + lr * ldl + 8 * lq;
      f32x4_t acc[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[u] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      constexpr int PB = 8;  // k-steps per batch of W_out loads
      uint4 wb[PB], wn[PB];
#pragma unroll
      for (int u = 0; u < PB; ++u) wb[u] = *(const uint4*)(wp + 32 * ks_of(min(u, per - 1)));
      for (int s = 0; s < per; s += PB) {
        if (s + PB < per)
#pragma unroll
          for (int u = 0; u < PB; ++u) wn[u] = *(const uint4*)(wp + 32 * ks_of(min(s + PB + u, per - 1)));
#pragma unroll
        for (int u = 0; u < PB; ++u) {
          if (s + u >= per) break;
          acc[u & 3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8_t, wb[u]), __builtin_bit_cast(bf16x8_t, *(const uint4*)(yp + 32 * ks_of(s + u))),
              acc[u & 3], 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < PB; ++u) wb[u] = wn[u];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) vpart[wave][lane][i] = (acc[0][i] + acc[1][i]) + (acc[2][i] + acc[3][i]);
    }
    lds_barrier();
    if (wave < NT) {
      const uint2 bb = *(const uint2*)(b_out + 16 * wave + 4 * lq);
      const float bias[4] = {__uint_as_float(bb.x << 16), __uint_as_float(bb.x & 0xffff0000u),
                             __uint_as_float(bb.y << 16), __uint_as_float(bb.y & 0xffff0000u)};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float vb = vpart[wave][lane][i];
#pragma unroll
        for (int p = 1; p < KS; ++p) vb += vpart[wave + NT * p][lane][i];
        vb += bias[i];
        // guidance: v = v_u + g (v_c - v_u), branch 0 conditional, branch 1 unconditional
        vres[i] = b == 0 ? vb : vb + guidance * (vres[i] - vb);
      }
    }
  }
  // Euler update in place, or v handed to the step rule
  if (wave < NT && row0 + lr < rows && vout) {
    *(float4*)(vout + (int64_t)(row0 + lr) * C + 16 * wave + 4 * lq) = make_float4(vres[0], vres[1], vres[2], vres[3]);
  } else if (wave < NT && row0 + lr < rows) {
    float4* xp = (float4*)(x + (int64_t)(row0 + lr) * C + 16 * wave + 4 * lq);
    float4 xv = *xp;
    xv.x += dsig * vres[0];
    xv.y += dsig * vres[1];
    xv.z += dsig * vres[2];
    xv.w += dsig * vres[3];
    *xp = xv;
  }
}

// One step's streaming work on a tile of TR token rows, fused and
// speculative.  The patch embedding is computed once into LDS; from it
//   (a1, a2) m_t = S(LN(h)(1 + scale0) + shift0) is written and the four
//            relative-L1 sums against m_{t-1} and m_{t_last} accumulated, and
//   (a4, a5) the reuse step's result is formed as if the step were reused:
//            per branch h_out = S(h + r_b), y = S(LN(h_out)(1 + scale_f) +
//            shift_f) (in place of h in the tile), v_b = y W_out^T + b_out,
//            guidance combine, then x + dsigma v into x_spec (Euler) or v into
//            v_spec (the step rule runs after the decision).
// The decision is taken afterwards on the host; a reused step then costs
// no further pass over HBM, a computed one discards the candidate.  Every
// row load is issued before the first value it feeds is needed: the
// indicator rows and branch 0's residual rows right after the embedding,
// branch 1's residual rows while branch 0's projection runs.
struct StepFusedArgs {
  const float* x; int C;
  const bf16_t* W_in; const bf16_t* b_in;
  bf16_t* m_out; const bf16_t* m_prev; const bf16_t* m_last;
  int rows, H;
  const float* sh0; const float* sc0;  // nullptr: m_t = h (the paper's tensor)
  double* partials;                    // nullptr: no sums (t = 0)
  const bf16_t* r; int nb;             // nullptr: no reuse candidate
  const bf16_t* W_out; const bf16_t* b_out;
  const float* mf0; const float* mf1;  // final (shift, scale) of each branch, [2H] f32
  float dsig, guidance;
  float* x_spec; float* v_spec;
  bf16_t* h_out;                       // non-null: h rows are stored too (block-stack input)
};

template <int CK, int MAXC, int TR, int NT, int NB>
__global__ __launch_bounds__(64 * RW) void step_fused_kernel(StepFusedArgs a) {
  // dynamic LDS: tile [TR][H + LPAD] bf16, b_in [H] bf16, vectors [2H] f32 (scale | shift)
  extern __shared__ __attribute__((aligned(16))) bf16_t hl[];
  __shared__ float red[RW][4];
  __shared__ float vpart[RW][64][4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lq = lane >> 4;
  const int row0 = blockIdx.x * TR;
  const int H = a.H, rows = a.rows, C = a.C;
  const int ldl = H + LPAD, nch = H / 8;
  constexpr int RPW = (TR + RW - 1) / RW;  // rows per wave
  static_assert(RW % NT == 0, "projection tiles divide the waves");
  constexpr int KS = RW / NT;              // waves per projection tile
  bf16_t* bl = hl + TR * ldl;
  float* scl = (float*)(bl + H);
  float* shl = scl + H;
  const bool mod = a.sc0 != nullptr;
  const bool mpass = a.m_out != nullptr;
  const bool sums = a.partials != nullptr;
  const bool spec = a.r != nullptr;
  const bool same = a.m_prev == a.m_last;
  auto row_of = [&](int q) { return wave + RW * q; };            // tile row of this wave's q-th row
  auto valid = [&](int q) { return row_of(q) < TR && row0 + row_of(q) < rows; };
  auto grow = [&](int q) { return min(row0 + min(row_of(q), TR - 1), rows - 1); };  // clamped global row

  stage(a.b_in, bl, H / 8);
  if (mod) {
    stage(a.sc0, scl, H / 4);
    stage(a.sh0, shl, H / 4);
  }
  lds_barrier();
  embed_to_lds<CK, EMBED_EB, TR>(a.x, C, a.W_in, bl, row0, rows, H, hl, ldl, wave, lane);

  // indicator rows of all this wave's rows: unconditional loads with clamped
  // addresses, all in flight together; branch 0's residual rows follow row
  // by row as the indicator registers free up
  uint4 pv[RPW][MAXC], lv[RPW][MAXC], rv[RPW][MAXC];
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const int64_t base = (int64_t)grow(q) * H;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = min(lane + 64 * j, nch - 1);
      if (sums) {
        pv[q][j] = ld_stream(a.m_prev + base + 8 * c);
        if (!same) lv[q][j] = ld_stream(a.m_last + base + 8 * c);
      }
    }
  }
  auto load_r = [&](const bf16_t* rb, int q) {
    const int64_t base = (int64_t)grow(q) * H;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) rv[q][j] = ld_stream(rb + base + 8 * min(lane + 64 * j, nch - 1));
  };
  if (spec && !sums)
#pragma unroll
    for (int q = 0; q < RPW; ++q) load_r(a.r, q);
  lds_barrier();  // the h tile is complete; the row loads stay in flight

  if (a.h_out)  // the block stack's input, bit-identical to the h of every other pass
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
      if (!valid(q)) continue;
      const bf16_t* src = hl + row_of(q) * ldl;
      bf16_t* dst = a.h_out + (int64_t)(row0 + row_of(q)) * H;
#pragma unroll
      for (int j = 0; j < MAXC; ++j) {
        const int c = lane + 64 * j;
        if (c < nch) *(uint4*)(dst + 8 * c) = *(const uint4*)(src + 8 * c);
      }
    }

  // (a1, a2): m_t and the relative-L1 sums
  float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    if (spec && sums) load_r(a.r, q);
    if (!valid(q) || !mpass) continue;
    const int row = row0 + row_of(q);
    const bf16_t* src = hl + row_of(q) * ldl;
    float v[MAXC][8];
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = lane + 64 * j;
      unpack8(*(const uint4*)(src + 8 * min(c, nch - 1)), v[j]);
      if (c >= nch)
#pragma unroll
        for (int e = 0; e < 8; ++e) v[j][e] = 0.f;
    }
    float mean = 0.f, rstd = 1.f;
    if (mod) row_stats<MAXC>(v, nch, H, lane, mean, rstd);
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = lane + 64 * j;
      if (c >= nch) continue;
      float y[8];
      if (mod) {
        float k[8], d[8];
        load_f8(scl + 8 * c, k);
        load_f8(shl + 8 * c, d);
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = (v[j][e] - mean) * rstd * (1.f + k[e]) + d[e];
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = v[j][e];
      }
      const uint4 mt = pack8(y);
      st_stream(a.m_out + (int64_t)row * H + 8 * c, mt);
      if (sums) {
        float mv[8], p[8], l[8];
        unpack8(mt, mv);
        unpack8(pv[q][j], p);
        if (same) {
#pragma unroll
          for (int e = 0; e < 8; ++e) l[e] = p[e];
        } else {
          unpack8(lv[q][j], l);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          s0 += fabsf(mv[e] - p[e]);
          s1 += fabsf(p[e]);
          s2 += fabsf(mv[e] - l[e]);
          s3 += fabsf(l[e]);
        }
      }
    }
  }

  // (a4, a5) the reuse candidate
  if (spec) {
    float vres[4] = {0.f, 0.f, 0.f, 0.f};
    uint4 hk[NB > 1 ? RPW : 1][MAXC];  // h rows kept for the second branch
    for (int b = 0; b < NB; ++b) {
      const float* mf = b ? a.mf1 : a.mf0;
      lds_barrier();  // every wave is done with the vectors and the tile of the previous phase
      stage(mf + H, scl, H / 4);
      stage(mf, shl, H / 4);
      lds_barrier();
#pragma unroll
      for (int q = 0; q < RPW; ++q) {
        if (!valid(q)) continue;
        bf16_t* src = hl + row_of(q) * ldl;
        float v[MAXC][8];
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
          const int c = lane + 64 * j;
          uint4 hu;
          if (b == 0) {
            hu = *(const uint4*)(src + 8 * min(c, nch - 1));
            if (NB > 1) hk[NB > 1 ? q : 0][j] = hu;
          } else {
            hu = hk[NB > 1 ? q : 0][j];
          }
          float hv[8], rr[8];
          unpack8(hu, hv);
          unpack8(rv[q][j], rr);
#pragma unroll
          for (int e = 0; e < 8; ++e) v[j][e] = c < nch ? St<bf16_t>::rd(hv[e] + rr[e]) : 0.f;
        }
        float mean, rstd;
        row_stats<MAXC>(v, nch, H, lane, mean, rstd);
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
          const int c = lane + 64 * j;
          if (c >= nch) continue;
          float k[8], d[8], y[8];
          load_f8(scl + 8 * c, k);
          load_f8(shl + 8 * c, d);
#pragma unroll
          for (int e = 0; e < 8; ++e) y[e] = (v[j][e] - mean) * rstd * (1.f + k[e]) + d[e];
          *(uint4*)(src + 8 * c) = pack8(y);
        }
      }
      if (b + 1 < NB)  // the next branch's residual rows fly while this branch's projection runs
#pragma unroll
        for (int q = 0; q < RPW; ++q) load_r(a.r + (int64_t)(b + 1) * rows * H, q);
      lds_barrier();
      // v^T = W_out y^T: lane (lr, lq) of tile jt ends with v[row lr][16 jt + 4 lq + i];
      // KS waves share a tile, each a contiguous K range, partial sums added in wave order
      {
        const int jt = wave % NT, part = wave / NT;
        const int ks = H / 32, per = ks / KS;
        const int s0k = part * per;
        const int rot = (blockIdx.x * 8) % per;
        auto ks_of = [&](int u) { const int w = u + rot; return s0k + (w < per ? w : w - per); };
        const bf16_t* wp = a.W_out + (int64_t)(16 * jt + lr) * H + 8 * lq;
        const bf16_t* yp = hl + min(lr, TR - 1) * ldl + 8 * lq;
        f32x4_t acc[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) acc[u] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        constexpr int PB = 8;
        uint4 wb[PB], wn[PB];
#pragma unroll
        for (int u = 0; u < PB; ++u) wb[u] = *(const uint4*)(wp + 32 * ks_of(min(u, per - 1)));
        for (int s = 0; s < per; s += PB) {
          if (s + PB < per)
#pragma unroll
            for (int u = 0; u < PB; ++u) wn[u] = *(const uint4*)(wp + 32 * ks_of(min(s + PB + u, per - 1)));
#pragma unroll
          for (int u = 0; u < PB; ++u) {
            if (s + u >= per) break;
            acc[u & 3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8_t, wb[u]),
                __builtin_bit_cast(bf16x8_t, *(const uint4*)(yp + 32 * ks_of(s + u))), acc[u & 3], 0, 0, 0);
          }
#pragma unroll
          for (int u = 0; u < PB; ++u) wb[u] = wn[u];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) vpart[wave][lane][i] = (acc[0][i] + acc[1][i]) + (acc[2][i] + acc[3][i]);
      }
      lds_barrier();
      if (wave < NT) {
        const uint2 bb = *(const uint2*)(a.b_out + 16 * wave + 4 * lq);
        const float bias[4] = {__uint_as_float(bb.x << 16), __uint_as_float(bb.x & 0xffff0000u),
                               __uint_as_float(bb.y << 16), __uint_as_float(bb.y & 0xffff0000u)};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float vb = vpart[wave][lane][i];
#pragma unroll
          for (int p = 1; p < KS; ++p) vb += vpart[wave + NT * p][lane][i];
          vb += bias[i];
          // guidance: v = v_u + g (v_c - v_u), branch 0 conditional, branch 1 unconditional
          vres[i] = b == 0 ? vb : vb + a.guidance * (vres[i] - vb);
        }
      }
    }
    if (wave < NT && lr < TR && row0 + lr < rows) {
      const int64_t o = (int64_t)(row0 + lr) * C + 16 * wave + 4 * lq;
      if (a.v_spec) {
        *(float4*)(a.v_spec + o) = make_float4(vres[0], vres[1], vres[2], vres[3]);
      } else {
        const float4 xv = *(const float4*)(a.x + o);
        *(float4*)(a.x_spec + o) = make_float4(xv.x + a.dsig * vres[0], xv.y + a.dsig * vres[1],
                                               xv.z + a.dsig * vres[2], xv.w + a.dsig * vres[3]);
      }
    }
  }

  if (!sums) return;
  s0 = warp_sum(s0); s1 = warp_sum(s1); s2 = warp_sum(s2); s3 = warp_sum(s3);
  if (lane == 0) { red[wave][0] = s0; red[wave][1] = s1; red[wave][2] = s2; red[wave][3] = s3; }
  __syncthreads();
  if (threadIdx.x < 4) {
    double t = 0.0;
#pragma unroll
    for (int w = 0; w < RW; ++w) t += (double)red[w][threadIdx.x];
    a.partials[(int64_t)blockIdx.x * 4 + threadIdx.x] = t;
  }
}

template <typename F>
hipError_t dispatch_reuse(int C, int H, F f) {
  const int per_lane = (H / 8 + 63) / 64;
  auto with_c = [&](auto ck) -> hipError_t {
    if (per_lane <= 2) return f(ck, std::integral_constant<int, 2>());
    if (per_lane <= 4) return f(ck, std::integral_constant<int, 4>());
    if (per_lane <= 6) return f(ck, std::integral_constant<int, 6>());
    if (per_lane <= 10) return f(ck, std::integral_constant<int, 10>());
    return hipErrorInvalidValue;
  };
  if (C == 32) return with_c(std::integral_constant<int, 1>());
  if (C == 64) return with_c(std::integral_constant<int, 2>());
  if (C == 128) return with_c(std::integral_constant<int, 4>());
  return hipErrorInvalidValue;
}

// Dynamic LDS of both kernels: the row tile plus staged b_in, scale, shift.
size_t dyn_lds(int H) { return (size_t)RR * (H + LPAD) * 2 + (size_t)H * 2 + (size_t)H * 8; }

// Lets a kernel take `bytes` of dynamic LDS (beyond the 64 KB default).
hipError_t allow_lds(const void* kern, size_t bytes) {
  return hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

// Tile height of the fused step kernel: 16 rows (the MFMA's token lanes)
// when the tile, b_in and the two staged vectors fit the LDS next to the
// static reduction buffers and the row registers fit without spilling (at
// most 6 chunks per lane and row, one branch at 6); otherwise 8 rows (one
// per wave), which holds up to 10 chunks per lane for one branch or 6 for
// two; 0 when neither fits.
constexpr size_t kStepStaticLds = sizeof(float) * RW * 4 + sizeof(float) * RW * 64 * 4;
size_t step_lds(int TR, int H) { return (size_t)TR * (H + LPAD) * 2 + (size_t)H * 2 + (size_t)H * 8; }
int step_chunks(int H) {
  const int per_lane = (H / 8 + 63) / 64;
  return per_lane <= 2 ? 2 : per_lane <= 4 ? 4 : per_lane <= 6 ? 6 : per_lane <= 10 ? 10 : 0;
}
int step_rows(int H, int nb) {
  const int mc = step_chunks(H);
  const bool lds16 = step_lds(16, H) + kStepStaticLds <= 160 * 1024;
  const bool lds8 = step_lds(8, H) + kStepStaticLds <= 160 * 1024;
  if (mc == 0 || nb < 1 || nb > 2) return 0;
  if (lds16 && (mc <= 4 || (mc == 6 && nb == 1))) return 16;
  if (lds8 && (mc <= 6 || nb == 1)) return 8;
  return 0;
}

}  // namespace

bool reuse_fused_fits(int C, int H) {
  if (C != 32 && C != 64 && C != 128) return false;
  const int ks_waves = RW / (C / 16);  // waves sharing one projection tile
  return H >= 16 * RW && H % (32 * ks_waves) == 0 && (H / 8 + 63) / 64 <= 10 &&
         dyn_lds(H) + sizeof(float) * RW * 64 * 4 <= 160 * 1024;
}

int reuse_indicator_partials(int rows) { return (rows + RR - 1) / RR; }

hipError_t launch_reuse_indicator(const float* x, int C, const void* W_in, const void* b_in, void* m_out,
                                  const void* m_prev, const void* m_last, int rows, int H, const float* sh,
                                  const float* sc, double* partials, double* out, void* h_out, hipStream_t s) {
  if (!reuse_fused_fits(C, H) || rows < 1) return hipErrorInvalidValue;
  const int nblk = reuse_indicator_partials(rows);
  const size_t lds = dyn_lds(H);
  hipError_t e = dispatch_reuse(C, H, [&](auto ck, auto mc) {
    auto kern = reuse_indicator_kernel<decltype(ck)::value, decltype(mc)::value>;
    hipError_t a = allow_lds((const void*)kern, lds);
    if (a != hipSuccess) return a;
    hipLaunchKernelGGL(kern, dim3(nblk), dim3(64 * RW), lds, s, x, C, (const bf16_t*)W_in, (const bf16_t*)b_in,
                       (bf16_t*)m_out, (const bf16_t*)m_prev, (const bf16_t*)m_last, rows, H, sh, sc,
                       h_out ? nullptr : partials, (bf16_t*)h_out);
    return hipGetLastError();
  });
  if (e != hipSuccess || !partials || h_out) return e;
  return launch_reduce_partials(partials, nblk, out, s);
}

bool step_fused_fits(int C, int H, int nb) {
  // C = 64: four projection tiles of 16 columns, two waves each
  return C == 64 && H >= 16 * RW && H % 64 == 0 && step_rows(H, nb) > 0;
}

int step_fused_partials(int rows, int H, int nb) {
  const int TR = step_rows(H, nb);
  return TR ? (rows + TR - 1) / TR : 0;
}

hipError_t launch_step_fused(const float* x, int C, const void* W_in, const void* b_in, void* m_out,
                             const void* m_prev, const void* m_last, int rows, int H, const float* sh0,
                             const float* sc0, double* partials, double* out, const void* r, int nb,
                             const void* W_out, const void* b_out, const float* mf0, const float* mf1, float dsig,
                             float guidance, float* x_spec, float* v_spec, void* h_out, hipStream_t s) {
  if (!step_fused_fits(C, H, nb) || rows < 1 || (r && !x_spec && !v_spec)) return hipErrorInvalidValue;
  if ((partials != nullptr) != (m_prev != nullptr) || (partials && !m_out)) return hipErrorInvalidValue;
  const int TR = step_rows(H, nb), MC = step_chunks(H);
  const int nblk = (rows + TR - 1) / TR;
  const size_t lds = step_lds(TR, H);
  StepFusedArgs a{x, C, (const bf16_t*)W_in, (const bf16_t*)b_in, (bf16_t*)m_out, (const bf16_t*)m_prev,
                  (const bf16_t*)m_last, rows, H, sh0, sc0, partials, (const bf16_t*)r, nb,
                  (const bf16_t*)W_out, (const bf16_t*)b_out, mf0, mf1, dsig, guidance, x_spec, v_spec,
                  (bf16_t*)h_out};
  auto go = [&](auto kern) {
    hipError_t q = allow_lds((const void*)kern, lds);
    if (q != hipSuccess) return q;
    hipLaunchKernelGGL(kern, dim3(nblk), dim3(64 * RW), lds, s, a);
    return hipGetLastError();
  };
  // (chunks per lane, tile rows, branches) as step_rows admits them; C = 64
  hipError_t e = hipErrorInvalidValue;
  if (MC == 2) e = TR == 16 ? (nb == 1 ? go(step_fused_kernel<2, 2, 16, 4, 1>) : go(step_fused_kernel<2, 2, 16, 4, 2>))
                            : (nb == 1 ? go(step_fused_kernel<2, 2, 8, 4, 1>) : go(step_fused_kernel<2, 2, 8, 4, 2>));
  if (MC == 4) e = TR == 16 ? (nb == 1 ? go(step_fused_kernel<2, 4, 16, 4, 1>) : go(step_fused_kernel<2, 4, 16, 4, 2>))
                            : (nb == 1 ? go(step_fused_kernel<2, 4, 8, 4, 1>) : go(step_fused_kernel<2, 4, 8, 4, 2>));
  if (MC == 6) e = TR == 16 ? go(step_fused_kernel<2, 6, 16, 4, 1>)
                            : (nb == 1 ? go(step_fused_kernel<2, 6, 8, 4, 1>) : go(step_fused_kernel<2, 6, 8, 4, 2>));
  if (MC == 10) e = go(step_fused_kernel<2, 10, 8, 4, 1>);
  if (e != hipSuccess || !partials) return e;
  return launch_reduce_partials(partials, nblk, out, s);
}

hipError_t launch_reuse_final(float* x, int C, const void* W_in, const void* b_in, const void* r, int nb,
                              const void* W_out, const void* b_out, const float* mod0, const float* mod1,
                              float dsig, float guidance, int rows, int H, float* vout, hipStream_t s) {
  if (!reuse_fused_fits(C, H) || rows < 1 || nb < 1 || nb > 2) return hipErrorInvalidValue;
  const int nblk = (rows + RR - 1) / RR;
  const size_t lds = dyn_lds(H);
  return dispatch_reuse(C, H, [&](auto ck, auto mc) {
    constexpr int CK = decltype(ck)::value;
    auto kern = reuse_final_kernel<CK, decltype(mc)::value, 2 * CK>;
    hipError_t a = allow_lds((const void*)kern, lds);
    if (a != hipSuccess) return a;
    hipLaunchKernelGGL(kern, dim3(nblk), dim3(64 * RW), lds, s, x, C, (const bf16_t*)W_in, (const bf16_t*)b_in,
                       (const bf16_t*)r, nb, (const bf16_t*)W_out, (const bf16_t*)b_out, mod0, mod1, dsig,
                       guidance, rows, H, vout);
    return hipGetLastError();
  });
}

}  // namespace dit
