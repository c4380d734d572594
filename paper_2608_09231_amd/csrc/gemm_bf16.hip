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

  // ---------------------------------------------------------------- epilogue
  // acc[i][j][r] holds C[m][n] with
  //   m = m0 + wm*WM + i*32 + 8*(r/4) + 4*lhalf + (r%4),  n = n0 + wn*WN + j*32 + lrow.
  const int ncol0 = n0 + wn * WN;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int n = ncol0 + j * 32 + lrow;
    const float bv = (P.bias && n < P.N) ? bf16_to_f32(P.bias[n]) : 0.f;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] += bv;
  }
  if (P.rms_cols > 0 && ncol0 < P.rms_cols) {
    // one 128-wide head = 4 consecutive 32-wide tiles of this wave
#pragma unroll
    for (int hb = 0; hb < TN / 4; ++hb) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float ss = 0.f;
#pragma unroll
          for (int j = 0; j < 4; ++j) ss += acc[i][hb * 4 + j][r] * acc[i][hb * 4 + j][r];
#pragma unroll
          for (int o = 1; o < 32; o <<= 1) ss += __shfl_xor(ss, o, 64);
          const float sc = rsqrtf(ss * (1.f / 128.f) + DIT_RMS_EPS);
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][hb * 4 + j][r] *= sc;
        }
    }
  }
  const bool f32out = P.flags & DIT_EPI_F32;
  const bool gated = P.flags & DIT_EPI_GATED_RES;
  const bool silu = P.flags & DIT_EPI_SILU;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int n = ncol0 + j * 32 + lrow;
    if (n >= P.N) continue;
    const bool gl = n >= P.gelu_from;
    const int nc = n + (n >= P.gap_at ? P.gap : 0);
    const float g = gated ? P.gate[n] : 0.f;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * WM + i * 32 + 8 * (r >> 2) + 4 * lhalf + (r & 3);
        if (m >= P.M) continue;
        float v = acc[i][j][r];
        if (gl) v = gelu_tanh_f(v);
        if (silu) v = silu_f(v);
        if (f32out) {
          ((float*)P.C)[(int64_t)m * P.ldc + nc] = v;
        } else {
          bf16_t* c = (bf16_t*)P.C + (int64_t)m * P.ldc + nc;
          if (gated) v = bf16_to_f32(*c) + g * v;
          *c = f32_to_bf16(v);
        }
      }
  }
}

struct Cfg {
  int bm, bn, wg_per_cu;
  float eff;
  void (*fn)(Batch);
};

const Cfg kCfgs[] = {
    {256, 128, 1, 0.92f, gemm_bf16_kernel<256, 128, 4, 1>},
    {128, 128, 2, 0.80f, gemm_bf16_kernel<128, 128, 4, 1>},
    {32, 256, 2, 0.45f, gemm_bf16_kernel<32, 256, 1, 4>},
};

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

int pick_cfg(const GemmArgs* g, int n, int n_cu) {
  bool rms = false;
  for (int i = 0; i < n; ++i) rms |= g[i].rms_cols > 0;
  int best = -1;
  double best_t = 1e300;
  for (int c = 0; c < (int)(sizeof(kCfgs) / sizeof(kCfgs[0])); ++c) {
    const Cfg& k = kCfgs[c];
    if (rms && k.bn < 128) continue;
    if (rms && k.bm == 32) continue;  // its waves are 64 columns wide: no whole head
    long tiles = 0;
    for (int i = 0; i < n; ++i)
      tiles += (long)((g[i].M + k.bm - 1) / k.bm) * ((g[i].N + k.bn - 1) / k.bn);
    const long slots = (long)n_cu * k.wg_per_cu;
    const long waves = (tiles + slots - 1) / slots;
    const double t = (double)waves * k.bm * k.bn / (k.wg_per_cu * k.eff);
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
  hipLaunchKernelGGL(k.fn, dim3(b.total), dim3(256), 0, stream, b);
  return hipGetLastError();
}

}  // namespace dit
