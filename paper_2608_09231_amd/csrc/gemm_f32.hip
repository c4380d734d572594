// f32 GEMM for the f32 (small) workloads: C = epi(A . W^T + bias), 64x64
// tiles, 16-deep K slices in LDS, 4x4 outputs per thread.  Same epilogue
// flags as the bf16 kernel except the per-head RMS norm, which the f32 path
// applies with a separate kernel.
#include "common.h"
#include "kernels.h"

namespace dit {
namespace {

constexpr int TB = 64, TK = 16;

struct ProbF {
  const float* A; int64_t lda;
  const float* W; int64_t ldw;
  const float* bias;
  float* C; int64_t ldc;
  const float* gate;
  int M, N, K, flags, gelu_from, gap_at, gap, tiles_n;
};

__global__ __launch_bounds__(256) void gemm_f32_kernel(ProbF p) {
  __shared__ float sA[TK][TB + 1], sW[TK][TB + 1];
  const int tm = blockIdx.x / p.tiles_n, tn = blockIdx.x % p.tiles_n;
  const int m0 = tm * TB, n0 = tn * TB;
  const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < p.K; k0 += TK) {
    for (int i = tid; i < TB * TK; i += 256) {
      const int r = i / TK, kk = i % TK;
      const int gk = k0 + kk;
      const int gm = m0 + r, gn = n0 + r;
      sA[kk][r] = (gm < p.M && gk < p.K) ? p.A[(int64_t)gm * p.lda + gk] : 0.f;
      sW[kk][r] = (gn < p.N && gk < p.K) ? p.W[(int64_t)gn * p.ldw + gk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) { a[i] = sA[kk][ty * 4 + i]; w[i] = sW[kk][tx * 4 + i]; }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], w[j], acc[i][j]);
    }
    __syncthreads();
  }
  const bool gated = p.flags & DIT_EPI_GATED_RES, silu = p.flags & DIT_EPI_SILU;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= p.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n >= p.N) continue;
      float v = acc[i][j] + (p.bias ? p.bias[n] : 0.f);
      if (n >= p.gelu_from) v = gelu_tanh_f(v);
      if (silu) v = silu_f(v);
      const int nc = n + (n >= p.gap_at ? p.gap : 0);
      float* c = p.C + (int64_t)m * p.ldc + nc;
      if (gated) v = *c + p.gate[n] * v;
      *c = v;
    }
  }
}

}  // namespace

hipError_t launch_gemm_f32(const GemmArgs* g, int n, hipStream_t s) {
  for (int i = 0; i < n; ++i) {
    ProbF p;
    p.A = (const float*)g[i].A; p.lda = g[i].lda;
    p.W = (const float*)g[i].W; p.ldw = g[i].ldw;
    p.bias = (const float*)g[i].bias;
    p.C = (float*)g[i].C; p.ldc = g[i].ldc;
    p.gate = g[i].gate;
    p.M = g[i].M; p.N = g[i].N; p.K = g[i].K;
    p.flags = g[i].flags; p.gelu_from = g[i].gelu_from; p.gap_at = g[i].gap_at; p.gap = g[i].gap;
    p.tiles_n = (p.N + TB - 1) / TB;
    const int tiles = ((p.M + TB - 1) / TB) * p.tiles_n;
    if (tiles == 0) continue;
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(tiles), dim3(256), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace dit
