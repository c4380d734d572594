// Attention kernels of the DiT blocks.
//
// bf16 flash attention (head_dim 128) on gfx950 MFMA 32x32x16.  The score
// tile is computed transposed, S^T = K Q^T, so each lane owns one query
// column and its softmax statistics: the row max needs one exchange with the
// partner lane (lane ^ 32) and the running rescale of the output is a
// per-lane scalar.  The output is accumulated transposed as well,
// O^T = V^T P^T, which lets the probabilities feed the second MFMA straight
// from the score accumulators (same lane, same registers); V is therefore
// read from a per-head transposed copy [128][keys].  K and V^T tiles of 64
// keys are staged in padded LDS, double-buffered through registers.
// Exact-softmax semantics (non-causal), f32 statistics, P rounded to bf16
// for the second product, output normalised once at the end.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace dit {
namespace {

constexpr int D = 128;
constexpr int KT = 64;        // keys per tile
constexpr int KLD = D + 8;    // padded K row, elements
constexpr int VLD = KT + 8;   // padded V^T row, elements (144 bytes)
constexpr int QW = 32;        // queries per wave
constexpr int QB = 4 * QW;    // queries per workgroup

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void flash_attn_bf16_kernel(
    const bf16_t* __restrict__ q, int64_t ldq, const bf16_t* __restrict__ k, int64_t ldk,
    const bf16_t* __restrict__ vt, int ldvt, bf16_t* __restrict__ o, int64_t ldo, int Lq, int Lk,
    float scale_log2) {
  __shared__ __attribute__((aligned(16))) bf16_t sK[2][KT * KLD];
  __shared__ __attribute__((aligned(16))) bf16_t sV[2][D * VLD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lrow = lane & 31, lhalf = lane >> 5;
  const int h = blockIdx.y;
  const int qi = blockIdx.x * QB + wave * QW + lrow;
  const int qrow = min(qi, Lq - 1);

  // Q^T fragments: lane holds d = 16 s + 8 lhalf + [0, 8) of its query.
  bf16x8_t qf[8];
  {
    const bf16_t* qp = q + (int64_t)qrow * ldq + h * D + 8 * lhalf;
#pragma unroll
    for (int s = 0; s < 8; ++s) qf[s] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(qp + 16 * s));
  }

  const bf16_t* kh = k + h * D;
  const bf16_t* vh = vt + (int64_t)h * D * ldvt;
  uint4 rk[4], rv[4];
  auto gload = [&](int kb0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + 256 * i;
      const int key = min(kb0 + (c >> 4), Lk - 1);
      rk[i] = *(const uint4*)(kh + (int64_t)key * ldk + (c & 15) * 8);
      const int d = c >> 3;
      rv[i] = *(const uint4*)(vh + (int64_t)d * ldvt + kb0 + (c & 7) * 8);
    }
  };
  auto sstore = [&](int st) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + 256 * i;
      *(uint4*)(&sK[st][(c >> 4) * KLD + (c & 15) * 8]) = rk[i];
      *(uint4*)(&sV[st][(c >> 3) * VLD + (c & 7) * 8]) = rv[i];
    }
  };

  f32x16_t oacc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  const int ntiles = (Lk + KT - 1) / KT;
  gload(0);
  sstore(0);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int st = t & 1;
    if (t + 1 < ntiles) gload((t + 1) * KT);

    // S^T = K Q^T for 64 keys: two 32-key tiles.
    f32x16_t sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.f;
      const bf16_t* kp = &sK[st][(kb * 32 + lrow) * KLD + 8 * lhalf];
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        bf16x8_t kf = __builtin_bit_cast(bf16x8_t, *(const uint4*)(kp + 16 * s));
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sacc[kb], 0, 0, 0);
      }
    }
    // scale, mask, running max
    const int kbase = t * KT;
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kbase + kb * 32 + 8 * (r >> 2) + 4 * lhalf + (r & 3);
        float v = sacc[kb][r] * scale_log2;
        v = key < Lk ? v : -INFINITY;
        sacc[kb][r] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    float ls = 0.f;
    bf16x8_t pf[4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      uint32_t w[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float p0 = __builtin_amdgcn_exp2f(sacc[kb][2 * j] - m_new);
        const float p1 = __builtin_amdgcn_exp2f(sacc[kb][2 * j + 1] - m_new);
        ls += p0 + p1;
        w[j] = (uint32_t)f32_to_bf16(p0) | ((uint32_t)f32_to_bf16(p1) << 16);
      }
      pf[2 * kb] = __builtin_bit_cast(bf16x8_t, make_uint4(w[0], w[1], w[2], w[3]));
      pf[2 * kb + 1] = __builtin_bit_cast(bf16x8_t, make_uint4(w[4], w[5], w[6], w[7]));
    }
    l_run = l_run * alpha + ls;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;

    // O^T += V^T P^T
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const bf16_t* vp = &sV[st][(dt * 32 + lrow) * VLD + 4 * lhalf];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const uint2 lo = *(const uint2*)(vp + 16 * ks);
        const uint2 hi = *(const uint2*)(vp + 16 * ks + 8);
        const uint4 v4 = make_uint4(lo.x, lo.y, hi.x, hi.y);
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, v4), pf[ks],
                                                          oacc[dt], 0, 0, 0);
      }
    }
    if (t + 1 < ntiles) sstore(st ^ 1);
    __syncthreads();
  }

  const float l = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.f / l;
  if (qi < Lq) {
    bf16_t* op = o + (int64_t)qi * ldo + h * D;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d0 = dt * 32 + 8 * g + 4 * lhalf;
        uint32_t w0 = (uint32_t)f32_to_bf16(oacc[dt][4 * g] * inv) |
                      ((uint32_t)f32_to_bf16(oacc[dt][4 * g + 1] * inv) << 16);
        uint32_t w1 = (uint32_t)f32_to_bf16(oacc[dt][4 * g + 2] * inv) |
                      ((uint32_t)f32_to_bf16(oacc[dt][4 * g + 3] * inv) << 16);
        *(uint2*)(op + d0) = make_uint2(w0, w1);
      }
  }
}

// vt[h][d][l] = v[l][h*128 + d] for l < Lk, 0 for Lk <= l < ldvt.
__global__ __launch_bounds__(256) void transpose_v_kernel(const bf16_t* __restrict__ v, int64_t ldv,
                                                          bf16_t* __restrict__ vt, int Lk, int ldvt) {
  __shared__ bf16_t tile[64][D + 2];
  const int l0 = blockIdx.x * 64, h = blockIdx.y, tid = threadIdx.x;
  for (int i = tid; i < 64 * (D / 2); i += 256) {
    const int r = i / (D / 2), c2 = i % (D / 2);
    const int l = l0 + r;
    uint32_t w = 0;
    if (l < Lk) w = *(const uint32_t*)(v + (int64_t)l * ldv + h * D + 2 * c2);
    tile[r][2 * c2] = (bf16_t)(w & 0xffff);
    tile[r][2 * c2 + 1] = (bf16_t)(w >> 16);
  }
  __syncthreads();
  bf16_t* out = vt + (int64_t)h * D * ldvt + l0;
  for (int i = tid; i < D * 32; i += 256) {
    const int d = i / 32, c2 = i % 32;
    const uint32_t w = (uint32_t)tile[2 * c2][d] | ((uint32_t)tile[2 * c2 + 1][d] << 16);
    *(uint32_t*)(out + (int64_t)d * ldvt + 2 * c2) = w;
  }
}

// ------------------------------------------------------------------ f32 path
// One thread per query, keys streamed through LDS in tiles of 32.
template <int HD>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ q, int64_t ldq,
                                                      const float* __restrict__ k, int64_t ldk,
                                                      const float* __restrict__ v, int64_t ldv,
                                                      float* __restrict__ o, int64_t ldo, int Lq,
                                                      int Lk, float scale) {
  __shared__ float sk[32][HD], sv[32][HD];
  const int h = blockIdx.y, tid = threadIdx.x;
  const int qi = blockIdx.x * 64 + tid;
  const int qr = min(qi, Lq - 1);
  float qv[HD], acc[HD];
#pragma unroll
  for (int d = 0; d < HD; ++d) {
    qv[d] = q[(int64_t)qr * ldq + h * HD + d] * scale;
    acc[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int k0 = 0; k0 < Lk; k0 += 32) {
    __syncthreads();
    for (int i = tid; i < 32 * HD; i += 64) {
      const int r = i / HD, d = i % HD;
      const int key = min(k0 + r, Lk - 1);
      sk[r][d] = k[(int64_t)key * ldk + h * HD + d];
      sv[r][d] = v[(int64_t)key * ldv + h * HD + d];
    }
    __syncthreads();
    const int nk = min(32, Lk - k0);
    for (int j = 0; j < nk; ++j) {
      float s = 0.f;
#pragma unroll
      for (int d = 0; d < HD; ++d) s += qv[d] * sk[j][d];
      const float mn = fmaxf(m, s);
      const float a = expf(m - mn), p = expf(s - mn);
      l = l * a + p;
#pragma unroll
      for (int d = 0; d < HD; ++d) acc[d] = acc[d] * a + p * sv[j][d];
      m = mn;
    }
  }
  if (qi < Lq) {
#pragma unroll
    for (int d = 0; d < HD; ++d) o[(int64_t)qi * ldo + h * HD + d] = acc[d] / l;
  }
}

}  // namespace

hipError_t launch_transpose_v_bf16(const void* v, int64_t ldv, void* vt, int Lk, int heads,
                                   hipStream_t s) {
  const int ldvt = (Lk + 63) / 64 * 64;
  hipLaunchKernelGGL(transpose_v_kernel, dim3(ldvt / 64, heads), dim3(256), 0, s,
                     (const bf16_t*)v, ldv, (bf16_t*)vt, Lk, ldvt);
  return hipGetLastError();
}

hipError_t launch_flash_attn_bf16(const void* q, int64_t ldq, const void* k, int64_t ldk,
                                  const void* vt, int ldvt, void* o, int64_t ldo, int Lq, int Lk,
                                  int heads, hipStream_t s) {
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)D);
  hipLaunchKernelGGL(flash_attn_bf16_kernel, dim3((Lq + QB - 1) / QB, heads), dim3(256), 0, s,
                     (const bf16_t*)q, ldq, (const bf16_t*)k, ldk, (const bf16_t*)vt, ldvt,
                     (bf16_t*)o, ldo, Lq, Lk, scale_log2);
  return hipGetLastError();
}

hipError_t launch_attn_f32(const float* q, int64_t ldq, const float* k, int64_t ldk,
                           const float* v, int64_t ldv, float* o, int64_t ldo, int Lq, int Lk,
                           int heads, int head_dim, hipStream_t s) {
  const float scale = 1.f / sqrtf((float)head_dim);
  dim3 grid((Lq + 63) / 64, heads);
#define DIT_ATTN_F32(HD_)                                                                  \
  case HD_:                                                                                \
    hipLaunchKernelGGL(attn_f32_kernel<HD_>, grid, dim3(64), 0, s, q, ldq, k, ldk, v, ldv, \
                       o, ldo, Lq, Lk, scale);                                             \
    break;
  switch (head_dim) {
    DIT_ATTN_F32(16)
    DIT_ATTN_F32(32)
    DIT_ATTN_F32(64)
    DIT_ATTN_F32(128)
    default:
      return hipErrorInvalidValue;
  }
#undef DIT_ATTN_F32
  return hipGetLastError();
}

}  // namespace dit
