// Row-streaming and elementwise kernels of the sampler (HBM-bound):
// LN + adaLN modulation, the trajectory indicator with its relative-L1
// partial sums, the deterministic final reduction, residual refresh /
// reuse, the Euler update, and the once-per-sample embedding helpers.
#include <math.h>

#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace dit {
namespace {

// 16-byte chunks of a row: 8 bf16 or 4 f32 values.
template <typename T> struct Chunk;
template <> struct Chunk<bf16_t> {
  static constexpr int E = 8;
  static __device__ __forceinline__ void load(const bf16_t* p, float (&v)[8]) {
    const uint4 u = *(const uint4*)p;
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  static __device__ __forceinline__ void unpack(const uint4& u, float (&v)[8]) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  static __device__ __forceinline__ void store(bf16_t* p, const float (&v)[8]) {
    *(uint4*)p = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                            pack_bf16x2(v[6], v[7]));
  }
};
template <> struct Chunk<float> {
  static constexpr int E = 4;
  static __device__ __forceinline__ void load(const float* p, float (&v)[4]) {
    const float4 u = *(const float4*)p;
    v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
  }
  static __device__ __forceinline__ void unpack(const uint4& u, float (&v)[4]) {
    v[0] = __uint_as_float(u.x); v[1] = __uint_as_float(u.y);
    v[2] = __uint_as_float(u.z); v[3] = __uint_as_float(u.w);
  }
  static __device__ __forceinline__ void store(float* p, const float (&v)[4]) {
    *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
  }
};

// One wave per row: the row lives in registers as MAXC chunks per lane.
// FULL: the row is exactly 64 MAXC chunks, so no lane needs a range test
// (tests become branches, and a load behind a branch waits for the previous
// one).
template <typename T, int MAXC, bool FULL = false>
struct RowRegs {
  static constexpr int E = Chunk<T>::E;
  float v[MAXC][E];
  int nch;
  // Every chunk load is issued unconditionally (chunk index clamped into the
  // row) so they all stay in flight together; chunks past the row end are
  // then zeroed.  A tested load would become a branch with a wait behind it.
  __device__ __forceinline__ void load(const T* x, int H, int lane) {
    nch = H / E;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) Chunk<T>::load(x + cl(lane + 64 * j) * E, v[j]);
#pragma unroll
    for (int j = 0; j < MAXC; ++j)
      if (!ok(lane + 64 * j))
#pragma unroll
        for (int e = 0; e < E; ++e) v[j][e] = 0.f;
  }
  __device__ __forceinline__ int cl(int c) const { return FULL || c < nch ? c : nch - 1; }
  __device__ __forceinline__ bool ok(int c) const { return FULL || c < nch; }
  // LN statistics over H values (two passes over registers)
  __device__ __forceinline__ void stats(int H, int lane, float& mean, float& rstd) const {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < MAXC; ++j)
#pragma unroll
      for (int e = 0; e < E; ++e) s += v[j][e];
    mean = warp_sum(s) / (float)H;
    float q = 0.f;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      if (ok(lane + 64 * j))
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float d = v[j][e] - mean;
          q += d * d;
        }
    }
    rstd = rsqrtf(warp_sum(q) / (float)H + DIT_LN_EPS);
  }
};

__device__ __forceinline__ void load_mod(const float* p, float (&m)[8]) {
  const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
  m[0] = a.x; m[1] = a.y; m[2] = a.z; m[3] = a.w; m[4] = b.x; m[5] = b.y; m[6] = b.z; m[7] = b.w;
}
__device__ __forceinline__ void load_mod(const float* p, float (&m)[4]) {
  const float4 a = *(const float4*)p;
  m[0] = a.x; m[1] = a.y; m[2] = a.z; m[3] = a.w;
}

template <typename T, int MAXC, bool FULL>
__global__ __launch_bounds__(256) void ln_mod_kernel(const T* __restrict__ x, int64_t ldx,
                                                    T* __restrict__ out, int64_t ldo, int rows, int H,
                                                    int split, const float* sh0, const float* sc0,
                                                    const float* sh1, const float* sc1, int seg0, int seg1,
                                                    int64_t mstride) {
  constexpr int E = Chunk<T>::E;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  RowRegs<T, MAXC, FULL> r;
  r.load(x + (int64_t)row * ldx, H, lane);
  float mean, rstd;
  r.stats(H, lane, mean, rstd);
  const bool lo = row < split;
  const int64_t mo = (int64_t)(lo ? row / seg0 : (row - split) / seg1) * mstride;
  const float* sh = (lo ? sh0 : sh1) + mo;
  const float* sc = lo ? sc0 : sc1;
  if (sc) sc += mo;
  T* o = out + (int64_t)row * ldo;
  if (sc) {
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = lane + 64 * j, cc = r.cl(c);  // clamped: loads without branches
      float y[E], a[E], b[E];
      load_mod(sc + cc * E, a);
      load_mod(sh + cc * E, b);
#pragma unroll
      for (int e = 0; e < E; ++e) y[e] = (r.v[j][e] - mean) * rstd * (1.f + a[e]) + b[e];
      if (r.ok(c)) Chunk<T>::store(o + c * E, y);
    }
  } else {
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = lane + 64 * j;
      float y[E];
#pragma unroll
      for (int e = 0; e < E; ++e) y[e] = (r.v[j][e] - mean) * rstd;
      if (r.ok(c)) Chunk<T>::store(o + c * E, y);
    }
  }
}

// Indicator: each wave handles IRW consecutive rows; m = S(LN(h)(1+sc)+sh)
// (or m = h when sc == nullptr) is written, and |m - mp|, |mp|, |m - ml|,
// |ml| are summed per lane, then per workgroup (f64 partial 4-vector).  The
// rows of m_prev / m_last are loaded together with h, before the
// statistics, so the three streams are in flight at once.
constexpr int IRW = 1;
constexpr int IROWS = 4 * IRW;  // rows per workgroup

template <typename T, int MAXC, bool FULL>
__global__ __launch_bounds__(256) void indicator_kernel(const T* __restrict__ h, T* __restrict__ m,
                                                       const T* __restrict__ mp,
                                                       const T* __restrict__ ml, int rows, int H,
                                                       const float* sh, const float* sc,
                                                       double* __restrict__ partials) {
  constexpr int E = Chunk<T>::E;
  __shared__ float red[4][4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const bool same = mp == ml;
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
  for (int i = 0; i < IRW; ++i) {
    const int row = (blockIdx.x * 4 + wave) * IRW + i;
    if (row >= rows) break;
    const int64_t base = (int64_t)row * H;
    RowRegs<T, MAXC, FULL> r;
    r.load(h + base, H, lane);
    uint4 pv[MAXC], lv[MAXC];
    if (mp) {
#pragma unroll
      for (int j = 0; j < MAXC; ++j) {
        const int cc = r.cl(lane + 64 * j);  // clamped: loads without branches
        pv[j] = *(const uint4*)(mp + base + cc * E);
        if (!same) lv[j] = *(const uint4*)(ml + base + cc * E);
      }
    }
    float mean = 0.f, rstd = 1.f;
    if (sc) r.stats(H, lane, mean, rstd);
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = lane + 64 * j, cc = r.cl(c);
      float y[E];
      if (sc) {
        float a[E], b[E];
        load_mod(sc + cc * E, a);
        load_mod(sh + cc * E, b);
#pragma unroll
        for (int e = 0; e < E; ++e) y[e] = St<T>::rd((r.v[j][e] - mean) * rstd * (1.f + a[e]) + b[e]);
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) y[e] = r.v[j][e];
      }
      if (!r.ok(c)) continue;
      Chunk<T>::store(m + base + c * E, y);
      if (mp) {
        float p[E], l[E];
        Chunk<T>::unpack(pv[j], p);
        if (same) {
#pragma unroll
          for (int e = 0; e < E; ++e) l[e] = p[e];
        } else {
          Chunk<T>::unpack(lv[j], l);
        }
#pragma unroll
        for (int e = 0; e < E; ++e) {
          a0 += fabsf(y[e] - p[e]);
          a1 += fabsf(p[e]);
          a2 += fabsf(y[e] - l[e]);
          a3 += fabsf(l[e]);
        }
      }
    }
  }
  if (!partials) return;
  a0 = warp_sum(a0); a1 = warp_sum(a1); a2 = warp_sum(a2); a3 = warp_sum(a3);
  if (lane == 0) { red[wave][0] = a0; red[wave][1] = a1; red[wave][2] = a2; red[wave][3] = a3; }
  __syncthreads();
  if (threadIdx.x < 4) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < 4; ++w) s += (double)red[w][threadIdx.x];
    partials[(int64_t)blockIdx.x * 4 + threadIdx.x] = s;
  }
}

// Fixed-order f64 sum of n partial 4-vectors: thread t sums t, t+256, ...,
// then a fixed binary tree.  Deterministic for a given n.  `out` is
// host-mapped pinned memory.
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

// Reuse-step final-layer input: y = S(LN(S(a + b)) (1 + sc) + sh), one wave
// per row (a = h, b = cached residual r).
template <typename T, int MAXC, bool FULL>
__global__ __launch_bounds__(256) void add_ln_mod_kernel(const T* __restrict__ a, const T* __restrict__ b,
                                                        T* __restrict__ out, int rows, int H,
                                                        const float* sh, const float* sc) {
  constexpr int E = Chunk<T>::E;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int64_t base = (int64_t)row * H;
  RowRegs<T, MAXC, FULL> r;
  r.load(a + base, H, lane);
  float q[MAXC][E];
#pragma unroll
  for (int j = 0; j < MAXC; ++j) Chunk<T>::load(b + base + r.cl(lane + 64 * j) * E, q[j]);
#pragma unroll
  for (int j = 0; j < MAXC; ++j)
    if (r.ok(lane + 64 * j))
#pragma unroll
      for (int e = 0; e < E; ++e) r.v[j][e] = St<T>::rd(r.v[j][e] + q[j][e]);
  float mean, rstd;
  r.stats(H, lane, mean, rstd);
#pragma unroll
  for (int j = 0; j < MAXC; ++j) {
    const int c = lane + 64 * j, cc = r.cl(c);
    float y[E], s1[E], s2[E];
    load_mod(sc + cc * E, s1);
    load_mod(sh + cc * E, s2);
#pragma unroll
    for (int e = 0; e < E; ++e) y[e] = (r.v[j][e] - mean) * rstd * (1.f + s1[e]) + s2[e];
    if (r.ok(c)) Chunk<T>::store(out + base + c * E, y);
  }
}

// out = S(a + sign b), 16-byte vectors (n is a multiple of the vector width).
template <typename T>
__global__ void add_kernel(const T* __restrict__ a, const T* __restrict__ b, T* __restrict__ out,
                           int64_t n, float sign) {
  constexpr int E = Chunk<T>::E;
  const int64_t nv = n / E;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nv;
       i += (int64_t)gridDim.x * blockDim.x) {
    float x[E], y[E];
    Chunk<T>::load(a + i * E, x);
    Chunk<T>::load(b + i * E, y);
#pragma unroll
    for (int e = 0; e < E; ++e) x[e] += sign * y[e];
    Chunk<T>::store(out + i * E, x);
  }
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

// One UniPC step per element (coefficients from the host, see UniCoef):
// v = v_c or v_u + g (v_c - v_u); m_t = x_t - sigma_t v (stored);
// corrector x_c = cx x_last + cs m_s + cp m_p + ct m_t (or x_t at step 0),
// stored as the new x_last; predictor x_{t+1} = px x_c + pt m_t + pp m_s.
// m_s = m_{t-1}, m_p = m_{t-2} (nullptr where the coefficient is 0).
__global__ void unipc_kernel(float* __restrict__ x, const float* __restrict__ vc, const float* __restrict__ vu,
                             float g, float sig_t, float* __restrict__ x_last, const float* __restrict__ m_s,
                             const float* __restrict__ m_p, float* __restrict__ m_t, UniCoef k, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    float v = vc[i];
    if (vu) v = vu[i] + g * (v - vu[i]);
    const float xv = x[i];
    const float m = xv - sig_t * v;
    m_t[i] = m;
    float xc = xv;
    if (k.corr) {
      xc = k.cx * x_last[i] + k.cs * m_s[i] + k.ct * m;
      if (m_p) xc += k.cp * m_p[i];
    }
    x_last[i] = xc;
    float xn = k.px * xc + k.pt * m;
    if (m_s) xn += k.pp * m_s[i];
    x[i] = xn;
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

// Calls f(MAXC, FULL) for the smallest MAXC in the set with 64 MAXC >= H / E
// chunks; FULL when the row is exactly 64 MAXC chunks.
template <typename T, typename F>
hipError_t dispatch_maxc(int H, F f) {
  constexpr int E = Chunk<T>::E;
  const int nch = H / E;
  const int per_lane = (nch + 63) / 64;
  auto go = [&](auto mc) -> hipError_t {
    if (nch == 64 * decltype(mc)::value) return f(mc, std::true_type());
    return f(mc, std::false_type());
  };
  if (per_lane <= 2) return go(std::integral_constant<int, 2>());
  if (per_lane <= 4) return go(std::integral_constant<int, 4>());
  if (per_lane <= 6) return go(std::integral_constant<int, 6>());
  if (per_lane <= 8) return go(std::integral_constant<int, 8>());
  if (per_lane <= 10) return go(std::integral_constant<int, 10>());
  if (per_lane <= 12) return go(std::integral_constant<int, 12>());
  if (per_lane <= 16) return go(std::integral_constant<int, 16>());
  if (per_lane <= 32) return go(std::integral_constant<int, 32>());
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_ln_mod(const T* x, int64_t ldx, T* out, int64_t ldo, int rows, int H, int split,
                         const float* sh0, const float* sc0, const float* sh1, const float* sc1,
                         hipStream_t s, int seg0, int seg1, int64_t mstride) {
  if (H % Chunk<T>::E || seg0 < 1 || seg1 < 1) return hipErrorInvalidValue;
  if (rows <= 0) return hipSuccess;
  return dispatch_maxc<T>(H, [&](auto mc, auto fl) {
    hipLaunchKernelGGL((ln_mod_kernel<T, decltype(mc)::value, decltype(fl)::value>), dim3((rows + 3) / 4), dim3(256), 0, s, x,
                       ldx, out, ldo, rows, H, split, sh0, sc0, sh1, sc1, seg0, seg1, mstride);
    return hipGetLastError();
  });
}

template <typename T>
hipError_t launch_indicator(const T* h, T* m_out, const T* m_prev, const T* m_last, int rows, int H,
                            const float* sh, const float* sc, double* partials, double* out, hipStream_t s) {
  if (H % Chunk<T>::E) return hipErrorInvalidValue;
  const int nb = (rows + IROWS - 1) / IROWS;
  hipError_t e = dispatch_maxc<T>(H, [&](auto mc, auto fl) {
    hipLaunchKernelGGL((indicator_kernel<T, decltype(mc)::value, decltype(fl)::value>), dim3(nb), dim3(256), 0, s, h, m_out,
                       m_prev, m_last, rows, H, sh, sc, partials);
    return hipGetLastError();
  });
  if (e != hipSuccess || !partials) return e;
  return launch_reduce_partials(partials, nb, out, s);
}

hipError_t launch_reduce_partials(const double* partials, int n, double* out, hipStream_t s) {
  hipLaunchKernelGGL(reduce_partials_kernel, dim3(1), dim3(256), 0, s, partials, n, out);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_add_ln_mod(const T* a, const T* b, T* out, int rows, int H, const float* sh,
                             const float* sc, hipStream_t s) {
  if (H % Chunk<T>::E) return hipErrorInvalidValue;
  if (rows <= 0) return hipSuccess;
  return dispatch_maxc<T>(H, [&](auto mc, auto fl) {
    hipLaunchKernelGGL((add_ln_mod_kernel<T, decltype(mc)::value, decltype(fl)::value>), dim3((rows + 3) / 4),
                       dim3(256), 0, s,
                       a, b, out, rows, H, sh, sc);
    return hipGetLastError();
  });
}

int indicator_partials(int rows) { return (rows + IROWS - 1) / IROWS; }

template <typename T>
hipError_t launch_add(const T* a, const T* b, T* out, int64_t n, float sign, hipStream_t s) {
  if (n % Chunk<T>::E) return hipErrorInvalidValue;
  hipLaunchKernelGGL(add_kernel<T>, dim3(grid_for(n / Chunk<T>::E, 256)), dim3(256), 0, s, a, b, out, n, sign);
  return hipGetLastError();
}

hipError_t launch_unipc(float* x, const float* v_c, const float* v_u, float g, float sig_t, float* x_last,
                        const float* m_s, const float* m_p, float* m_t, const UniCoef& k, int64_t n,
                        hipStream_t s) {
  hipLaunchKernelGGL(unipc_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, x, v_c, v_u, g, sig_t, x_last, m_s,
                     m_p, m_t, k, n);
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
                                       const float*, const float*, const float*, hipStream_t, int, \
                                       int, int64_t);                                              \
  template hipError_t launch_indicator<T>(const T*, T*, const T*, const T*, int, int, const float*, \
                                          const float*, double*, double*, hipStream_t);            \
  template hipError_t launch_add_ln_mod<T>(const T*, const T*, T*, int, int, const float*, const float*, \
                                           hipStream_t);                                           \
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
