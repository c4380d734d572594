// Row-streaming and elementwise kernels of the sampler (HBM-bound):
// LN + adaLN modulation, the trajectory indicator with its relative-L1
// partial sums, the deterministic final reduction, residual refresh /
// reuse, the Euler update, and the once-per-sample embedding helpers.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace dit {
namespace {

constexpr int RT = 256;       // threads per row kernel
constexpr int MAXJ = 32;      // max elements per thread: H <= 8192

// Load one row (H elements) into registers, f32.
template <typename T>
__device__ __forceinline__ void load_row(const T* x, int H, float (&v)[MAXJ], int& nj) {
  nj = (H + RT - 1) / RT;
#pragma unroll
  for (int j = 0; j < MAXJ; ++j) {
    const int c = threadIdx.x + RT * j;
    v[j] = (j < nj && c < H) ? St<T>::ld(x + c) : 0.f;
  }
}

// mean and 1/sqrt(var + eps) of a row held in registers (two passes).
__device__ __forceinline__ void row_stats(const float (&v)[MAXJ], int nj, int H, float* red,
                                          float& mean, float& rstd) {
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < MAXJ; ++j) s += v[j];
  mean = block_sum<RT / 64>(s, red) / (float)H;
  float q = 0.f;
#pragma unroll
  for (int j = 0; j < MAXJ; ++j) {
    const int c = threadIdx.x + RT * j;
    const float d = (j < nj && c < H) ? v[j] - mean : 0.f;
    q += d * d;
  }
  const float var = block_sum<RT / 64>(q, red + 8) / (float)H;
  rstd = rsqrtf(var + DIT_LN_EPS);
}

template <typename T>
__global__ __launch_bounds__(RT) void ln_mod_kernel(const T* __restrict__ x, int64_t ldx,
                                                    T* __restrict__ out, int64_t ldo, int H,
                                                    int split, const float* sh0, const float* sc0,
                                                    const float* sh1, const float* sc1) {
  __shared__ float red[16];
  const int row = blockIdx.x;
  float v[MAXJ];
  int nj;
  load_row(x + (int64_t)row * ldx, H, v, nj);
  float mean, rstd;
  row_stats(v, nj, H, red, mean, rstd);
  const float* sh = row < split ? sh0 : sh1;
  const float* sc = row < split ? sc0 : sc1;
  T* o = out + (int64_t)row * ldo;
#pragma unroll
  for (int j = 0; j < MAXJ; ++j) {
    const int c = threadIdx.x + RT * j;
    if (j < nj && c < H) {
      float y = (v[j] - mean) * rstd;
      if (sc) y = y * (1.f + sc[c]) + sh[c];
      St<T>::st(o + c, y);
    }
  }
}

// One workgroup per group of IR rows: m = S(LN(h)(1+sc)+sh) (or S(h)),
// accumulate |m - mp|, |mp|, |m - ml|, |ml|.
constexpr int IR = 4;

template <typename T>
__global__ __launch_bounds__(RT) void indicator_kernel(const T* __restrict__ h, T* __restrict__ m,
                                                       const T* __restrict__ mp,
                                                       const T* __restrict__ ml, int rows, int H,
                                                       const float* sh, const float* sc,
                                                       double* __restrict__ partials) {
  __shared__ float red[16];
  __shared__ float red4[4][RT / 64];
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
  for (int rr = 0; rr < IR; ++rr) {
    const int row = blockIdx.x * IR + rr;
    if (row >= rows) break;
    const int64_t base = (int64_t)row * H;
    float v[MAXJ];
    int nj;
    load_row(h + base, H, v, nj);
    float mean = 0.f, rstd = 1.f;
    if (sc) row_stats(v, nj, H, red, mean, rstd);
#pragma unroll
    for (int j = 0; j < MAXJ; ++j) {
      const int c = threadIdx.x + RT * j;
      if (j < nj && c < H) {
        float y = sc ? ((v[j] - mean) * rstd) * (1.f + sc[c]) + sh[c] : v[j];
        y = St<T>::rd(y);
        St<T>::st(m + base + c, y);
        if (mp) {
          const float p = St<T>::ld(mp + base + c);
          const float l = St<T>::ld(ml + base + c);
          a0 += fabsf(y - p);
          a1 += fabsf(p);
          a2 += fabsf(y - l);
          a3 += fabsf(l);
        }
      }
    }
  }
  if (!partials) return;
  a0 = warp_sum(a0); a1 = warp_sum(a1); a2 = warp_sum(a2); a3 = warp_sum(a3);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { red4[0][w] = a0; red4[1][w] = a1; red4[2][w] = a2; red4[3][w] = a3; }
  __syncthreads();
  if (threadIdx.x < 4) {
    double s = 0.0;
    for (int i = 0; i < RT / 64; ++i) s += (double)red4[threadIdx.x][i];
    partials[(int64_t)blockIdx.x * 4 + threadIdx.x] = s;
  }
}

// Fixed-order f64 sum of n partial 4-vectors: thread t sums t, t+256, ...,
// then a fixed binary tree.  Deterministic for a given n.
__global__ __launch_bounds__(256) void reduce_partials_kernel(const double* __restrict__ p, int n,
                                                              double* out) {
  __shared__ double s[4][256];
  double a[4] = {0, 0, 0, 0};
  for (int i = threadIdx.x; i < n; i += 256)
#pragma unroll
    for (int c = 0; c < 4; ++c) a[c] += p[(int64_t)i * 4 + c];
#pragma unroll
  for (int c = 0; c < 4; ++c) s[c][threadIdx.x] = a[c];
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w)
#pragma unroll
      for (int c = 0; c < 4; ++c) s[c][threadIdx.x] += s[c][threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x < 4) out[threadIdx.x] = s[threadIdx.x][0];
  __threadfence_system();
}

template <typename T>
__global__ void add_kernel(const T* __restrict__ a, const T* __restrict__ b, T* __restrict__ out,
                           int64_t n, float sign) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    St<T>::st(out + i, St<T>::ld(a + i) + sign * St<T>::ld(b + i));
}

__global__ void euler_kernel(float* __restrict__ x, const float* __restrict__ vc,
                             const float* __restrict__ vu, float g, float dsig, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    float v = vc[i];
    if (vu) v = vu[i] + g * (v - vu[i]);
    x[i] = fmaf(dsig, v, x[i]);
  }
}

template <typename T>
__global__ void cast_kernel(const float* __restrict__ x, T* __restrict__ out, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    St<T>::st(out + i, x[i]);
}

// One wave per (row, head); head_dim <= 128.
__global__ void rms_heads_f32_kernel(float* x, int64_t ld, int rows, int heads, int hd) {
  const int wid = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (wid >= rows * heads) return;
  const int row = wid / heads, hh = wid % heads;
  float* p = x + (int64_t)row * ld + hh * hd;
  const float a = lane < hd ? p[lane] : 0.f;
  const float b = lane + 64 < hd ? p[lane + 64] : 0.f;
  const float ss = warp_sum(a * a + b * b);
  const float sc = rsqrtf(ss / (float)hd + DIT_RMS_EPS);
  if (lane < hd) p[lane] = a * sc;
  if (lane + 64 < hd) p[lane + 64] = b * sc;
}

template <typename T>
__global__ void time_embed_kernel(const double* __restrict__ sig, T* __restrict__ out, int Tn,
                                  int dim) {
  const int half = dim / 2;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= Tn * half) return;
  const int t = i / half, kk = i % half;
  const double f = exp(-log(10000.0) * (double)kk / (double)half);
  const double a = 1000.0 * sig[t] * f;
  St<T>::st(out + (int64_t)t * dim + kk, (float)cos(a));
  St<T>::st(out + (int64_t)t * dim + half + kk, (float)sin(a));
}

template <typename T>
__global__ void mean_rows_kernel(const T* __restrict__ x, int rows, int cols, T* __restrict__ out) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= cols) return;
  double s = 0.0;
  for (int r = 0; r < rows; ++r) s += (double)St<T>::ld(x + (int64_t)r * cols + c);
  St<T>::st(out + c, (float)(s / rows));
}

template <typename T>
__global__ void vec_silu_kernel(const float* __restrict__ a, const float* __restrict__ b,
                                T* __restrict__ out, int rows, int cols) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * cols) return;
  const int c = i % cols;
  const float v = St<T>::rd(a[i] + (b ? b[c] : 0.f));
  St<T>::st(out + i, silu_f(v));
}

template <typename T>
__global__ void add_offset_kernel(const float* __restrict__ mod, int64_t ld, int base,
                                  const T* __restrict__ off, float* __restrict__ out, int rows,
                                  int cols) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * cols) return;
  const int r = i / cols, c = i % cols;
  out[i] = mod[(int64_t)r * ld + base + c] + St<T>::ld(off + c);
}

inline int grid_for(int64_t n, int bs) {
  int64_t g = (n + bs - 1) / bs;
  return (int)(g < 65536 ? (g > 0 ? g : 1) : 65536);
}

}  // namespace

template <typename T>
hipError_t launch_ln_mod(const T* x, int64_t ldx, T* out, int64_t ldo, int rows, int H, int split,
                         const float* sh0, const float* sc0, const float* sh1, const float* sc1,
                         hipStream_t s) {
  if (H > RT * MAXJ) return hipErrorInvalidValue;
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(ln_mod_kernel<T>, dim3(rows), dim3(RT), 0, s, x, ldx, out, ldo, H, split, sh0,
                     sc0, sh1, sc1);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_indicator(const T* h, T* m_out, const T* m_prev, const T* m_last, int rows, int H,
                            const float* sh, const float* sc, double* partials, int* n_partials,
                            hipStream_t s) {
  if (H > RT * MAXJ) return hipErrorInvalidValue;
  const int nb = (rows + IR - 1) / IR;
  if (n_partials) *n_partials = nb;
  hipLaunchKernelGGL(indicator_kernel<T>, dim3(nb), dim3(RT), 0, s, h, m_out, m_prev, m_last, rows,
                     H, sh, sc, partials);
  return hipGetLastError();
}

hipError_t launch_reduce_partials(const double* partials, int n, double* out, hipStream_t s) {
  hipLaunchKernelGGL(reduce_partials_kernel, dim3(1), dim3(256), 0, s, partials, n, out);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_add(const T* a, const T* b, T* out, int64_t n, float sign, hipStream_t s) {
  hipLaunchKernelGGL(add_kernel<T>, dim3(grid_for(n, 256)), dim3(256), 0, s, a, b, out, n, sign);
  return hipGetLastError();
}

hipError_t launch_euler(float* x, const float* v_c, const float* v_u, float g, float dsigma,
                        int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(euler_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, x, v_c, v_u, g, dsigma, n);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_cast_from_f32(const float* x, T* out, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(cast_kernel<T>, dim3(grid_for(n, 256)), dim3(256), 0, s, x, out, n);
  return hipGetLastError();
}

hipError_t launch_rms_heads_f32(float* x, int64_t ld, int rows, int cols, int head_dim,
                                hipStream_t s) {
  if (head_dim > 128) return hipErrorInvalidValue;
  const int heads = cols / head_dim;
  const int waves = rows * heads;
  hipLaunchKernelGGL(rms_heads_f32_kernel, dim3((waves + 3) / 4), dim3(256), 0, s, x, ld, rows,
                     heads, head_dim);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_time_embed(const double* sigmas, T* out, int T_, int dim, hipStream_t s) {
  const int n = T_ * (dim / 2);
  hipLaunchKernelGGL(time_embed_kernel<T>, dim3(grid_for(n, 256)), dim3(256), 0, s, sigmas, out, T_, dim);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_mean_rows(const T* x, int rows, int cols, T* out, hipStream_t s) {
  hipLaunchKernelGGL(mean_rows_kernel<T>, dim3(grid_for(cols, 256)), dim3(256), 0, s, x, rows, cols, out);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_vec_silu(const float* a, const float* b, T* out, int rows, int cols, hipStream_t s) {
  hipLaunchKernelGGL(vec_silu_kernel<T>, dim3(grid_for((int64_t)rows * cols, 256)), dim3(256), 0, s,
                     a, b, out, rows, cols);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_add_offset(const float* mod, int64_t ld, int base, const T* offset, float* out,
                             int rows, int cols, hipStream_t s) {
  hipLaunchKernelGGL(add_offset_kernel<T>, dim3(grid_for((int64_t)rows * cols, 256)), dim3(256), 0,
                     s, mod, ld, base, offset, out, rows, cols);
  return hipGetLastError();
}

#define DIT_INST(T)                                                                              \
  template hipError_t launch_ln_mod<T>(const T*, int64_t, T*, int64_t, int, int, int, const float*, \
                                       const float*, const float*, const float*, hipStream_t);     \
  template hipError_t launch_indicator<T>(const T*, T*, const T*, const T*, int, int, const float*, \
                                          const float*, double*, int*, hipStream_t);               \
  template hipError_t launch_add<T>(const T*, const T*, T*, int64_t, float, hipStream_t);         \
  template hipError_t launch_cast_from_f32<T>(const float*, T*, int64_t, hipStream_t);            \
  template hipError_t launch_time_embed<T>(const double*, T*, int, int, hipStream_t);             \
  template hipError_t launch_mean_rows<T>(const T*, int, int, T*, hipStream_t);                   \
  template hipError_t launch_vec_silu<T>(const float*, const float*, T*, int, int, hipStream_t);  \
  template hipError_t launch_add_offset<T>(const float*, int64_t, int, const T*, float*, int, int,  \
                                           hipStream_t);
DIT_INST(float)
DIT_INST(bf16_t)
#undef DIT_INST

}  // namespace dit
