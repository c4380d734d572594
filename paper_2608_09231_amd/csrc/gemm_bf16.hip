// bf16 GEMM on gfx950 MFMA (v_mfma_f32_32x32x16_bf16) with the fused
// epilogues of the DiT blocks:  C = epi(A . W^T + bias).
//
// A [M,K] and W [N,K] are both K-contiguous (W in nn.Linear [out,in]
// layout), so every MFMA operand is a 16-byte run of K.  Tiles of BM x BN
// are staged through LDS in BK = 64 slices, double-buffered, with the
// 16-byte chunks of each 128-byte row XOR-swizzled by (row & 7) so that
// the fragment reads of 32 consecutive rows hit distinct banks.  Four waves
// per workgroup, each owning a WM x WN sub-tile of 32x32 MFMA tiles.
// Workgroups are remapped so that each of the 8 XCDs walks a contiguous,
// M-grouped range of tiles (its own L2 sees the shared A rows / W columns).
#include <stdlib.h>

#include "common.h"
#include "kernels.h"

namespace dit {

namespace {

constexpr int BK = 64;

struct Prob {
  const bf16_t* A; int64_t lda;
  const bf16_t* W; int64_t ldw;
  const bf16_t* bias;
  void* C; int64_t ldc;
  const float* gate;
  int M, N, K;
  int flags, rms_cols, gelu_from, gap_at, gap;
  int tiles_m, tiles_n;
};

struct Batch {
  Prob p0, p1;
  int tiles0, total;
};

__device__ __forceinline__ int xcd_remap(int bid, int n) {
  const int x = bid & 7, idx = bid >> 3;
  const int q = n >> 3, r = n & 7;
  return x * q + (x < r ? x : r) + idx;
}

// Epilogue over groups of G = min(TN, 4) adjacent 32x32 tiles (one 128-wide
// head when G = 4): bias, optional per-head RMS norm, GELU / SiLU, then
// store (bf16 round, f32, or gated residual).  acc[i][j][r] holds C[m][n]
// with m = m0 + wm*WM + i*32 + 8*(r/4) + 4*lhalf + (r%4) and
// n = n0 + wn*WN + j*32 + lrow.
template <int TM, int TN, int WM, int WN>
__device__ __forceinline__ void epilogue(const Prob& P, f32x16_t (&acc)[TM][TN], int m0, int n0, int wm,
                                         int wn, int lrow, int lhalf) {
  constexpr int G = TN < 4 ? TN : 4;
  const int ncol0 = n0 + wn * WN;
  const bool f32out = P.flags & DIT_EPI_F32;
  const bool gated = P.flags & DIT_EPI_GATED_RES;
  const bool silu = P.flags & DIT_EPI_SILU;
#pragma unroll
  for (int hb = 0; hb < TN / G; ++hb) {
    const int nh = ncol0 + hb * G * 32;   // first column of this group
    const bool rms = G == 4 && nh < P.rms_cols;
    float bv[G], gv[G];
    int col[G];
    bool gl[G], ok[G];
#pragma unroll
    for (int jj = 0; jj < G; ++jj) {
      const int n = nh + jj * 32 + lrow;
      ok[jj] = n < P.N;
      bv[jj] = (P.bias && ok[jj]) ? bf16_to_f32(P.bias[n]) : 0.f;
      gv[jj] = (gated && ok[jj]) ? P.gate[n] : 0.f;
      gl[jj] = n >= P.gelu_from;
      col[jj] = n + (n >= P.gap_at ? P.gap : 0);
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v[G];
#pragma unroll
        for (int jj = 0; jj < G; ++jj) v[jj] = acc[i][hb * G + jj][r] + bv[jj];
        if (rms) {
          float ss = 0.f;
#pragma unroll
          for (int jj = 0; jj < G; ++jj) ss += v[jj] * v[jj];
#pragma unroll
          for (int o = 1; o < 32; o <<= 1) ss += __shfl_xor(ss, o, 64);
          const float sc = rsqrtf(ss * (1.f / 128.f) + DIT_RMS_EPS);
#pragma unroll
          for (int jj = 0; jj < G; ++jj) v[jj] *= sc;
        }
        const int m = m0 + wm * WM + i * 32 + 8 * (r >> 2) + 4 * lhalf + (r & 3);
        if (m >= P.M) continue;
#pragma unroll
        for (int jj = 0; jj < G; ++jj) {
          if (!ok[jj]) continue;
          float y = v[jj];
          if (gl[jj]) y = gelu_tanh_f(y);
          if (silu) y = silu_f(y);
          if (f32out) {
            ((float*)P.C)[(int64_t)m * P.ldc + col[jj]] = y;
          } else {
            bf16_t* c = (bf16_t*)P.C + (int64_t)m * P.ldc + col[jj];
            if (gated) y = bf16_to_f32(*c) + gv[jj] * y;
            *c = f32_to_bf16(y);
          }
        }
      }
    }
  }
}

template <int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(Batch b) {
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int A_LD = BM * BK / (8 * 256);  // 16-byte chunks per thread
  constexpr int B_LD = BN * BK / (8 * 256);
  static_assert(WGM * WGN == 4, "4 waves");
  static_assert(A_LD >= 1 && B_LD >= 1, "tile too small");

  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * (BM + BN) * BK];

  if ((int)blockIdx.x >= b.total) return;
  int lt = xcd_remap(blockIdx.x, b.total);
  const bool second = lt >= b.tiles0;
  const Prob P = second ? b.p1 : b.p0;
  if (second) lt -= b.tiles0;

  // M-grouped tile order (8 tile-rows per group).
  constexpr int GROUP = 8;
  const int in_group = GROUP * P.tiles_n;
  const int gid = lt / in_group;
  const int first_m = gid * GROUP;
  const int gsz = min(P.tiles_m - first_m, GROUP);
  const int tm = first_m + (lt % in_group) % gsz;
  const int tn = (lt % in_group) / gsz;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;

  // global -> register staging of one BK slice
  uint4 ra[A_LD], rb[B_LD];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      const int q = tid + 256 * i, row = q >> 3, kc = q & 7;
      const int gm = min(m0 + row, P.M - 1);
      const int gk = k0 + kc * 8;
      ra[i] = (gk < P.K) ? *(const uint4*)(P.A + (int64_t)gm * P.lda + gk) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int q = tid + 256 * i, row = q >> 3, kc = q & 7;
      const int gn = min(n0 + row, P.N - 1);
      const int gk = k0 + kc * 8;
      rb[i] = (gk < P.K) ? *(const uint4*)(P.W + (int64_t)gn * P.ldw + gk) : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int stage) {
    bf16_t* sA = smem + stage * (BM + BN) * BK;
    bf16_t* sB = sA + BM * BK;
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      const int q = tid + 256 * i, row = q >> 3, kc = q & 7;
      *(uint4*)(sA + row * BK + ((kc ^ (row & 7)) << 3)) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int q = tid + 256 * i, row = q >> 3, kc = q & 7;
      *(uint4*)(sB + row * BK + ((kc ^ (row & 7)) << 3)) = rb[i];
    }
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = (P.K + BK - 1) / BK;
  gload(0);
  sstore(0);
  __syncthreads();

  const int lrow = lane & 31, lhalf = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) gload((kt + 1) * BK);
    const bf16_t* sA = smem + (kt & 1) * (BM + BN) * BK;
    const bf16_t* sB = sA + BM * BK;
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      const int kc = 2 * s + lhalf;
      bf16x8_t af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = wm * WM + i * 32 + lrow;
        uint4 v = *(const uint4*)(sA + row * BK + ((kc ^ (row & 7)) << 3));
        af[i] = __builtin_bit_cast(bf16x8_t, v);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = wn * WN + j * 32 + lrow;
        uint4 v = *(const uint4*)(sB + row * BK + ((kc ^ (row & 7)) << 3));
        bfr[j] = __builtin_bit_cast(bf16x8_t, v);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore((kt + 1) & 1);
    __syncthreads();
  }

  epilogue<TM, TN, WM, WN>(P, acc, m0, n0, wm, wn, lrow, lhalf);
}

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

// Direct-to-LDS variant (K % 64 == 0): tiles are copied by
// global_load_lds_dwordx4 (64 lanes x 16 bytes into a contiguous 1 KB per
// instruction), so no staging registers are needed and a wave can hold a
// 128 x 128 accumulator block.  The per-lane source chunk realises the same
// XOR swizzle as the register-staged kernel.
template <int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_bf16_dma_kernel(Batch b) {
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int NW = WGM * WGN;
  constexpr int A_INS = BM / (8 * NW), B_INS = BN / (8 * NW);  // 1 KB copies per wave per slice
  constexpr int STAGE = (BM + BN) * BK * 2;                   // bytes
  static_assert(A_INS >= 1 && B_INS >= 1 && A_INS * 8 * NW == BM && B_INS * 8 * NW == BN, "tile");

  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  if ((int)blockIdx.x >= b.total) return;
  int lt = xcd_remap(blockIdx.x, b.total);
  const bool second = lt >= b.tiles0;
  const Prob P = second ? b.p1 : b.p0;
  if (second) lt -= b.tiles0;
  constexpr int GROUP = 8;
  const int in_group = GROUP * P.tiles_n;
  const int gid = lt / in_group;
  const int first_m = gid * GROUP;
  const int gsz = min(P.tiles_m - first_m, GROUP);
  const int tm = first_m + (lt % in_group) % gsz;
  const int tn = (lt % in_group) / gsz;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int lrow = lane & 31, lhalf = lane >> 5;

  // per-lane source offsets in elements (fixed for the whole K loop; the
  // buffers of one problem stay below 2^31 elements)
  uint32_t aoff[A_INS], boff[B_INS];
#pragma unroll
  for (int j = 0; j < A_INS; ++j) {
    const int row = 8 * (wave * A_INS + j) + (lane >> 3);
    const int c = (lane & 7) ^ (row & 7);
    aoff[j] = (uint32_t)min(m0 + row, P.M - 1) * (uint32_t)P.lda + c * 8;
  }
#pragma unroll
  for (int j = 0; j < B_INS; ++j) {
    const int row = 8 * (wave * B_INS + j) + (lane >> 3);
    const int c = (lane & 7) ^ (row & 7);
    boff[j] = (uint32_t)min(n0 + row, P.N - 1) * (uint32_t)P.ldw + c * 8;
  }
  auto issue = [&](int k0, int st) {
    char* sA = smem + st * STAGE;
    char* sB = sA + BM * BK * 2;
    const bf16_t* Ab = P.A + k0;
    const bf16_t* Bb = P.W + k0;
#pragma unroll
    for (int j = 0; j < A_INS; ++j)
      __builtin_amdgcn_global_load_lds((glb_void_t*)(Ab + aoff[j]), (lds_void_t*)(sA + (wave * A_INS + j) * 1024), 16, 0, 0);
#pragma unroll
    for (int j = 0; j < B_INS; ++j)
      __builtin_amdgcn_global_load_lds((glb_void_t*)(Bb + boff[j]), (lds_void_t*)(sB + (wave * B_INS + j) * 1024), 16, 0, 0);
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = P.K / BK;
  issue(0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) issue((kt + 1) * BK, (kt + 1) & 1);
    const char* sA = smem + (kt & 1) * STAGE;
    const char* sB = sA + BM * BK * 2;
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      const int kc = 2 * s + lhalf;
      bf16x8_t af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = wm * WM + i * 32 + lrow;
        af[i] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(sA + row * 128 + ((kc ^ (row & 7)) << 4)));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = wn * WN + j * 32 + lrow;
        bfr[j] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(sB + row * 128 + ((kc ^ (row & 7)) << 4)));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  epilogue<TM, TN, WM, WN>(P, acc, m0, n0, wm, wn, lrow, lhalf);
}

struct Cfg {
  int bm, bn, wn, wg_per_cu, threads;
  float eff;
  bool dma;
  void (*fn)(Batch);
};

// eff: relative MFMA efficiency of a full tile (measured ordering); the
// chooser minimises rounds x per-round work / eff over the configs a
// problem admits.
const Cfg kCfgs[] = {
    {256, 256, 128, 1, 512, 1.00f, true, gemm_bf16_dma_kernel<256, 256, 4, 2>},
    {256, 128, 128, 1, 256, 0.72f, true, gemm_bf16_dma_kernel<256, 128, 4, 1>},
    {128, 128, 128, 2, 256, 0.85f, true, gemm_bf16_dma_kernel<128, 128, 4, 1>},
    {32, 256, 64, 2, 256, 0.45f, true, gemm_bf16_dma_kernel<32, 256, 1, 4>},
    {256, 128, 128, 1, 256, 0.60f, false, gemm_bf16_kernel<256, 128, 4, 1>},
    {128, 128, 128, 2, 256, 0.55f, false, gemm_bf16_kernel<128, 128, 4, 1>},
    {32, 256, 64, 2, 256, 0.30f, false, gemm_bf16_kernel<32, 256, 1, 4>},
};
constexpr int kNumCfgs = sizeof(kCfgs) / sizeof(kCfgs[0]);

Prob make_prob(const GemmArgs& g, int bm, int bn) {
  Prob p;
  p.A = (const bf16_t*)g.A; p.lda = g.lda;
  p.W = (const bf16_t*)g.W; p.ldw = g.ldw;
  p.bias = (const bf16_t*)g.bias;
  p.C = g.C; p.ldc = g.ldc;
  p.gate = g.gate;
  p.M = g.M; p.N = g.N; p.K = g.K;
  p.flags = g.flags; p.rms_cols = g.rms_cols;
  p.gelu_from = g.gelu_from; p.gap_at = g.gap_at; p.gap = g.gap;
  p.tiles_m = (g.M + bm - 1) / bm;
  p.tiles_n = (g.N + bn - 1) / bn;
  return p;
}

int forced_cfg() {
  static int v = [] {
    const char* e = getenv("DIT_GEMM_CONFIG");
    return e ? atoi(e) : -1;
  }();
  return v;
}

int pick_cfg(const GemmArgs* g, int n, int n_cu) {
  bool rms = false, k64 = true;
  for (int i = 0; i < n; ++i) {
    rms |= g[i].rms_cols > 0;
    k64 &= (g[i].K % BK) == 0 && (g[i].lda % 8) == 0 && (g[i].ldw % 8) == 0;
  }
  const int f = forced_cfg();
  if (f >= 0 && f < kNumCfgs && (k64 || !kCfgs[f].dma) && (!rms || kCfgs[f].wn % 128 == 0)) return f;
  int best = -1;
  double best_t = 1e300;
  for (int c = 0; c < kNumCfgs; ++c) {
    const Cfg& k = kCfgs[c];
    if (k.dma && !k64) continue;
    if (rms && k.wn % 128) continue;
    long tiles = 0;
    for (int i = 0; i < n; ++i)
      tiles += (long)((g[i].M + k.bm - 1) / k.bm) * ((g[i].N + k.bn - 1) / k.bn);
    const long slots = (long)n_cu * k.wg_per_cu;
    const long rounds = (tiles + slots - 1) / slots;
    const double t = (double)rounds * k.bm * k.bn * k.wg_per_cu / k.eff;
    if (t < best_t) { best_t = t; best = c; }
  }
  return best;
}

}  // namespace

hipError_t launch_gemm_bf16(const GemmArgs* g, int n, hipStream_t stream, int n_cu) {
  if (n < 1 || n > 2) return hipErrorInvalidValue;
  const int c = pick_cfg(g, n, n_cu);
  const Cfg& k = kCfgs[c];
  Batch b;
  b.p0 = make_prob(g[0], k.bm, k.bn);
  b.p1 = n > 1 ? make_prob(g[1], k.bm, k.bn) : b.p0;
  b.tiles0 = b.p0.tiles_m * b.p0.tiles_n;
  b.total = b.tiles0 + (n > 1 ? b.p1.tiles_m * b.p1.tiles_n : 0);
  if (b.total == 0) return hipSuccess;
  hipLaunchKernelGGL(k.fn, dim3(b.total), dim3(k.threads), 0, stream, b);
  return hipGetLastError();
}

}  // namespace dit
