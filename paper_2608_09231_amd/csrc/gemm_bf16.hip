// bf16 GEMM on gfx950 MFMA (v_mfma_f32_32x32x16_bf16) with the fused
// epilogues of the DiT blocks:  C = epi(A . W^T + bias).
//
// A [M,K] and W [N,K] are both K-contiguous (W in nn.Linear [out,in]
// layout), so every MFMA operand is a 16-byte run of K.  Tiles are staged
// through LDS in BK = 64 slices (128-byte rows) by buffer loads with an LDS
// destination, the 16-byte chunks of each row XOR-swizzled by
// ((row >> 1) & 7): two consecutive 128-byte rows fill one 256-byte bank
// cycle, so the fragment reads of 16 consecutive rows hit 16 distinct 16-byte
// bank groups.  The main kernel (256 x 256 tiles, 8 waves of 64 x 128) keeps
// a ring of five operand slices in LDS: W slices (cold, from HBM) arrive two
// slices ahead of use, A slices one; smaller tiles use a two-stage pipeline.
// Workgroups are remapped so that each of the 8 XCDs walks a contiguous,
// M-grouped range of tiles (its own L2 sees the shared A rows / W columns).
#include <type_traits>
#include <utility>

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
  int64_t gstride;  // gate vector of row m: gate + (m / gseg) * gstride (gseg > 0)
  int M, N, K;
  int flags, rms_cols, gelu_from, gap_at, gap, gseg;
  int tiles_m, tiles_n;
  bf16_t* vt;  // transposed values (see GemmArgs)
  int vt_col0, vt_heads, vt_ld, vt_split, vt_rows0, vt_key0, vt_rows1, vt_key1;
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
  Prob P = second ? b.p1 : b.p0;
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
  // per-segment gate vectors: the host admits only BM | gseg, so a tile's
  // rows share one vector
  if (P.gseg > 0) P.gate += (int64_t)(m0 / P.gseg) * P.gstride;

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
      *(uint4*)(sA + row * BK + ((kc ^ ((row >> 1) & 7)) << 3)) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int q = tid + 256 * i, row = q >> 3, kc = q & 7;
      *(uint4*)(sB + row * BK + ((kc ^ ((row >> 1) & 7)) << 3)) = rb[i];
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
        uint4 v = *(const uint4*)(sA + row * BK + ((kc ^ ((row >> 1) & 7)) << 3));
        af[i] = __builtin_bit_cast(bf16x8_t, v);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = wn * WN + j * 32 + lrow;
        uint4 v = *(const uint4*)(sB + row * BK + ((kc ^ ((row >> 1) & 7)) << 3));
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

// LDS-staged epilogue for waves that own 128 output columns (WN == 128).
// Per 32-row slab: the raw f32 accumulators go to this wave's 16 KB of LDS
// (columns XOR 32 on rows with bit 2 set, so the two lane halves of a write
// hit different banks); then lane l handles rows l/16 + 4p (p = 0..7) and
// columns 4(l%16) + [0,4) and 64 + 4(l%16) + [0,4): bias, per-head RMS (a
// head is the 16 lanes of one row: 4 shuffles), GELU / SiLU, gated
// residual, and 8-byte stores that coalesce to 128 bytes per row.
// Requires N % 8 == 0, gelu_from and gap_at multiples of 4.
// KIND selects a specialised body: EPI_K_STORE (bf16 store; the per-head RMS
// norm, GELU and column gap each apply to whole 128-column groups, so they
// are wave-uniform), EPI_K_GATED (gated residual only), EPI_K_ANY (every
// flag, per column).
enum { EPI_K_STORE = 0, EPI_K_GATED = 1, EPI_K_ANY = 2 };
template <int KIND = EPI_K_ANY>
struct EpiLds {
  const Prob& P;
  int m_base, ncol0, cq, rq, lrow, lhalf;
  bool f32out, gated, silu, rms, gelu_u;
  float bv[2][4], gv[2][4];
  int col[2];
  bool ok[2], gl[2];
  float* slab;

  __device__ __forceinline__ EpiLds(const Prob& P_, int m_base_, int ncol0_, int lrow_, int lhalf_, float* slab_)
      : P(P_), m_base(m_base_), ncol0(ncol0_), lrow(lrow_), lhalf(lhalf_), slab(slab_) {}

  // Flags, column map, bias and gate values of this lane's 8 columns.
  __device__ __forceinline__ void prep() {
    const int lane = lhalf * 32 + lrow;
    cq = lane & 15;
    rq = lane >> 4;
    f32out = KIND == EPI_K_ANY && (P.flags & DIT_EPI_F32);
    gated = KIND == EPI_K_GATED || (KIND == EPI_K_ANY && (P.flags & DIT_EPI_GATED_RES));
    silu = KIND == EPI_K_ANY && (P.flags & DIT_EPI_SILU);
    rms = KIND != EPI_K_GATED && ncol0 < P.rms_cols;
    gelu_u = KIND == EPI_K_STORE && ncol0 >= P.gelu_from;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int n = ncol0 + 64 * hh + 4 * cq;
      ok[hh] = n < P.N;
      gl[hh] = n >= P.gelu_from;
      col[hh] = n + (n >= P.gap_at ? P.gap : 0);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        bv[hh][e] = (P.bias && ok[hh]) ? bf16_to_f32(P.bias[n + e]) : 0.f;
        gv[hh][e] = (gated && ok[hh]) ? P.gate[n + e] : 0.f;
      }
    }
  }

  // Residual values C[m][col .. col+3] of slab i (gated epilogue), loaded
  // before any slab is staged so their latency overlaps the staging.
  __device__ __forceinline__ void load_old(int i, uint2 (&old)[8][2]) const {
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      const int m = min(m_base + i * 32 + rq + 4 * p, P.M - 1);
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
        old[p][hh] = ok[hh] ? *(const uint2*)((const bf16_t*)P.C + (int64_t)m * P.ldc + col[hh]) : make_uint2(0, 0);
    }
  }

  // One 32-row slab: accumulators -> LDS -> 8-column row segments -> global.
  // Nothing waits on global memory here: a wave's LDS operations complete in
  // order, so neither the read-back nor the next slab's writes need more
  // than the wait for this wave's own slab writes.
  __device__ __forceinline__ void slab_pass(const f32x16_t (&a)[4], int i, const uint2 (&old)[8][2]) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 8 * (r >> 2) + 4 * lhalf + (r & 3);
        const int c = (j * 32 + lrow) ^ (((row >> 2) & 1) << 5);
        slab[row * 128 + c] = a[j][r];
      }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0) only
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      const int row = rq + 4 * p;
      const int sw = ((row >> 2) & 1) << 5;
      float v[2][4];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const float4 t = *(const float4*)(slab + row * 128 + ((64 * hh + 4 * cq) ^ sw));
        v[hh][0] = t.x + bv[hh][0]; v[hh][1] = t.y + bv[hh][1];
        v[hh][2] = t.z + bv[hh][2]; v[hh][3] = t.w + bv[hh][3];
      }
      if (KIND != EPI_K_GATED && rms) {
        float ss = 0.f;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int e = 0; e < 4; ++e) ss += v[hh][e] * v[hh][e];
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) ss += __shfl_xor(ss, o, 64);
        const float sc = rsqrtf(ss * (1.f / 128.f) + DIT_RMS_EPS);
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int e = 0; e < 4; ++e) v[hh][e] *= sc;
      }
      const int m = m_base + i * 32 + row;
      if constexpr (KIND == EPI_K_STORE) {
        if (gelu_u)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh)
#pragma unroll
            for (int e = 0; e < 4; ++e) v[hh][e] = gelu_tanh_f(v[hh][e]);
        if (m < P.M)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh)
            if (ok[hh])
              *(uint2*)((bf16_t*)P.C + (int64_t)m * P.ldc + col[hh]) =
                  make_uint2(pack_bf16x2(v[hh][0], v[hh][1]), pack_bf16x2(v[hh][2], v[hh][3]));
        continue;
      } else if constexpr (KIND == EPI_K_GATED) {
        if (m < P.M)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh)
            if (ok[hh]) {
              const uint2 o = old[p][hh];
              const float y0 = __uint_as_float(o.x << 16) + gv[hh][0] * v[hh][0];
              const float y1 = __uint_as_float(o.x & 0xffff0000u) + gv[hh][1] * v[hh][1];
              const float y2 = __uint_as_float(o.y << 16) + gv[hh][2] * v[hh][2];
              const float y3 = __uint_as_float(o.y & 0xffff0000u) + gv[hh][3] * v[hh][3];
              *(uint2*)((bf16_t*)P.C + (int64_t)m * P.ldc + col[hh]) =
                  make_uint2(pack_bf16x2(y0, y1), pack_bf16x2(y2, y3));
            }
        continue;
      }
      if (m < P.M) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          if (!ok[hh]) continue;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (gl[hh]) v[hh][e] = gelu_tanh_f(v[hh][e]);
            if (silu) v[hh][e] = silu_f(v[hh][e]);
          }
          if (f32out) {
            *(float4*)((float*)P.C + (int64_t)m * P.ldc + col[hh]) =
                make_float4(v[hh][0], v[hh][1], v[hh][2], v[hh][3]);
          } else {
            bf16_t* c = (bf16_t*)P.C + (int64_t)m * P.ldc + col[hh];
            if (gated) {
              const uint2 o = old[p][hh];
              v[hh][0] = __uint_as_float(o.x << 16) + gv[hh][0] * v[hh][0];
              v[hh][1] = __uint_as_float(o.x & 0xffff0000u) + gv[hh][1] * v[hh][1];
              v[hh][2] = __uint_as_float(o.y << 16) + gv[hh][2] * v[hh][2];
              v[hh][3] = __uint_as_float(o.y & 0xffff0000u) + gv[hh][3] * v[hh][3];
            }
            *(uint2*)c = make_uint2(pack_bf16x2(v[hh][0], v[hh][1]), pack_bf16x2(v[hh][2], v[hh][3]));
          }
        }
      }
    }
  }
};

// Runs the slab passes of a wave that owns TM x 32 rows and 128 columns;
// with the gated residual, the old values of every slab (of one slab at a
// time when TM > 2) are requested first.
// Each slab index is a compile-time constant so the accumulators stay in
// registers.
template <int TM, int KIND, size_t... Is>
__device__ __forceinline__ void epilogue_lds_impl(EpiLds<KIND>& e, f32x16_t (&acc)[TM][4], std::index_sequence<Is...>) {
  if constexpr (TM <= 2) {
    uint2 old[TM][8][2];
    if (e.gated) (e.load_old((int)Is, old[Is]), ...);
    (e.slab_pass(acc[Is], (int)Is, old[Is]), ...);
  } else {  // bounded registers: one slab's old values at a time
    auto one = [&](auto i) {
      constexpr int I = decltype(i)::value;
      uint2 old[8][2];
      if (e.gated) e.load_old(I, old);
      e.slab_pass(acc[I], I, old);
    };
    (one(std::integral_constant<int, (int)Is>{}), ...);
  }
}

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

// A DMA config uses the LDS-staged epilogue when its waves own 128 columns
// and its LDS holds one 32 x 128 f32 slab per wave; the host only picks such
// a config for problems that meet the epilogue's alignment conditions.
template <int WN, int NW, int LDS_BYTES>
constexpr bool kLdsEpilogue = WN == 128 && LDS_BYTES >= NW * 32 * 128 * 4;

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] | expcnt[6:4] = 7 | lgkmcnt[11:8] = 15 | vmcnt[5:4] at [15:14]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// 16 bytes per lane from base + voff + soff (bytes, 32-bit offsets) into LDS
// at dst + 16 lane: a raw buffer load with an LDS destination.  Offsets past
// 4 GiB - 1 read zeros; the host admits this path only when every row of
// the operand lies below that bound.
__device__ __forceinline__ void buf_lds16(const void* base, lds_void_t* dst, uint32_t voff, uint32_t soff) {
#if defined(__HIP_DEVICE_COMPILE__)
  const __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, (int)0xffffffffu, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, soff, 0, 0);
#endif
}

// Direct-to-LDS pipeline (K % BK == 0): BK-deep slices of A and W are copied
// by global_load_lds_dwordx4 (64 lanes x 16 bytes into a contiguous 1 KB per
// instruction: no staging registers), STAGES slices in flight.  A slice row
// has CPR = BK/8 chunks of 16 bytes; RPB = 256/(2 BK) rows share one 256-byte
// bank cycle, and chunk c of row r is stored at c ^ ((r / RPB) % CPR), so the
// fragment reads of 16 consecutive rows hit 16 distinct bank groups.  The
// per-lane source chunk of each copy realises the same swizzle.
template <int BM, int BN, int WGM, int WGN, int BK_, int STAGES>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_bf16_dma_kernel(Batch b) {
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int NW = WGM * WGN;
  constexpr int CPR = BK_ / 8, RPB = 256 / (2 * BK_);
  constexpr int ROWS_PER_INS = 64 / CPR;
  constexpr int A_INS = BM / (ROWS_PER_INS * NW), B_INS = BN / (ROWS_PER_INS * NW);
  constexpr int INS = A_INS + B_INS;                 // copies per wave per slice
  constexpr int STAGE = (BM + BN) * BK_ * 2;         // bytes
  static_assert(A_INS >= 1 && B_INS >= 1 && A_INS * ROWS_PER_INS * NW == BM &&
                    B_INS * ROWS_PER_INS * NW == BN, "tile");
  static_assert(STAGES >= 2 && (STAGES - 2) * INS < 64, "stages");

  __shared__ __attribute__((aligned(1024))) char smem[STAGES * STAGE];

  if ((int)blockIdx.x >= b.total) return;
  int lt = xcd_remap(blockIdx.x, b.total);
  const bool second = lt >= b.tiles0;
  Prob P = second ? b.p1 : b.p0;
  if (second) lt -= b.tiles0;
  constexpr int GROUP = 8;
  const int in_group = GROUP * P.tiles_n;
  const int gid = lt / in_group;
  const int first_m = gid * GROUP;
  const int gsz = min(P.tiles_m - first_m, GROUP);
  const int tm = first_m + (lt % in_group) % gsz;
  const int tn = (lt % in_group) / gsz;
  const int m0 = tm * BM, n0 = tn * BN;
  // per-segment gate vectors: the host admits only BM | gseg, so a tile's
  // rows share one vector
  if (P.gseg > 0) P.gate += (int64_t)(m0 / P.gseg) * P.gstride;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int lrow = lane & 31, lhalf = lane >> 5;

  // per-lane source offsets in bytes (fixed for the whole K loop; the host
  // admits this kernel only when they fit in 32 bits); the slice offset
  // kt * BK * 2 travels in the scalar offset of the buffer load
  uint32_t aoff[A_INS], boff[B_INS];
#pragma unroll
  for (int j = 0; j < A_INS; ++j) {
    const int row = ROWS_PER_INS * (wave * A_INS + j) + lane / CPR;
    const int c = (lane % CPR) ^ ((row / RPB) % CPR);
    aoff[j] = ((uint32_t)min(m0 + row, P.M - 1) * (uint32_t)P.lda + c * 8) * 2u;
  }
#pragma unroll
  for (int j = 0; j < B_INS; ++j) {
    const int row = ROWS_PER_INS * (wave * B_INS + j) + lane / CPR;
    const int c = (lane % CPR) ^ ((row / RPB) % CPR);
    boff[j] = ((uint32_t)min(n0 + row, P.N - 1) * (uint32_t)P.ldw + c * 8) * 2u;
  }
  auto issue = [&](int kt) {
    char* sA = smem + (kt % STAGES) * STAGE;
    char* sB = sA + BM * BK_ * 2;
    const uint32_t so = (uint32_t)kt * BK_ * 2;
#pragma unroll
    for (int j = 0; j < A_INS; ++j) buf_lds16(P.A, (lds_void_t*)(sA + (wave * A_INS + j) * 1024), aoff[j], so);
#pragma unroll
    for (int j = 0; j < B_INS; ++j) buf_lds16(P.W, (lds_void_t*)(sB + (wave * B_INS + j) * 1024), boff[j], so);
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  // The epilogue state (bias, gate, column map) is loaded before the K loop
  // when registers allow (TM <= 2), so those loads are done when the tile is.
  [[maybe_unused]] EpiLds<> epi(P, m0 + wm * TM * 32, n0 + wn * 128, lrow, lhalf, (float*)smem + wave * (32 * 128));
  if constexpr (kLdsEpilogue<WN, NW, STAGES * STAGE> && TM <= 2) epi.prep();

  const int nk = P.K / BK_;
  if constexpr (STAGES == 2 && BK_ == 64) {
    // Two 64-deep slices in LDS, fragments double-buffered in registers: the
    // LDS reads of substep s+1 (and, in substep 0, the copies of the next
    // slice) are interleaved with the 8 MFMAs of substep s; one barrier per
    // slice, the last iteration peeled so the loop body has no branch.
    auto rd = [&](int kt, int s, bf16x8_t(&af)[TM], bf16x8_t(&bfr)[TN]) {
      const char* sA = smem + (kt & 1) * STAGE;
      const char* sB = sA + BM * BK_ * 2;
      const int kc = 2 * s + lhalf;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = wm * WM + i * 32 + lrow;
        af[i] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(sA + row * (2 * BK_) + ((kc ^ ((row / RPB) % CPR)) << 4)));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = wn * WN + j * 32 + lrow;
        bfr[j] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(sB + row * (2 * BK_) + ((kc ^ ((row / RPB) % CPR)) << 4)));
      }
    };
    auto mm = [&](const bf16x8_t(&af)[TM], const bf16x8_t(&bfr)[TN]) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    };
    // Instruction order of one substep, fixed by scheduling groups: one MFMA,
    // then two LDS reads of the next substep (and, with WithCopy, two buffer
    // copies of the next slice), repeated; then the remaining MFMAs.  A
    // scheduling fence closes every substep, so the reads stay one substep
    // ahead of the MFMAs that consume them (two fragment sets live).
    auto sched = [&](auto with_copy) {
      constexpr bool WithCopy = decltype(with_copy)::value;
      constexpr int NM = TM * TN, ND = TM + TN, NG = (ND + 1) / 2;
      static_assert(NM >= NG, "substep shape");
#pragma unroll
      for (int q = 0; q < NG; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        if constexpr (WithCopy) __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);  // VMEM read
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // DS read
      }
      if constexpr (NM > NG) __builtin_amdgcn_sched_group_barrier(0x008, NM - NG, 0);
      __builtin_amdgcn_sched_barrier(0);
    };
    using copy_t = std::integral_constant<bool, true>;
    using nocopy_t = std::integral_constant<bool, false>;
    bf16x8_t a0[TM], b0[TN], a1[TM], b1[TN];
    issue(0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    rd(0, 0, a0, b0);
    for (int kt = 0; kt < nk - 1; ++kt) {
      issue(kt + 1);  // into the buffer of slice kt-1, which every wave has finished
      rd(kt, 1, a1, b1); mm(a0, b0); sched(copy_t{});
      rd(kt, 2, a0, b0); mm(a1, b1); sched(nocopy_t{});
      rd(kt, 3, a1, b1); mm(a0, b0); sched(nocopy_t{});
      mm(a1, b1);
      wait_vmcnt<0>();  // this wave's copies of slice kt+1 have landed
      __syncthreads();  // everyone's have, and every read of slice kt is done
      rd(kt + 1, 0, a0, b0);
    }
    rd(nk - 1, 1, a1, b1); mm(a0, b0); sched(nocopy_t{});
    rd(nk - 1, 2, a0, b0); mm(a1, b1); sched(nocopy_t{});
    rd(nk - 1, 3, a1, b1); mm(a0, b0); sched(nocopy_t{});
    mm(a1, b1);
  } else {
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nk) issue(s);

  for (int kt = 0; kt < nk; ++kt) {
    // slice kt must have landed: later slices may stay in flight
    if (nk - 1 - kt >= STAGES - 2) wait_vmcnt<(STAGES - 2) * INS>();
    else __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();  // every wave's copies of slice kt are in; slice kt-1 is no longer read
    if (kt + STAGES - 1 < nk) issue(kt + STAGES - 1);
    const char* sA = smem + (kt % STAGES) * STAGE;
    const char* sB = sA + BM * BK_ * 2;
#pragma unroll
    for (int s = 0; s < BK_ / 16; ++s) {
      const int kc = 2 * s + lhalf;
      bf16x8_t af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = wm * WM + i * 32 + lrow;
        af[i] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(sA + row * (2 * BK_) + ((kc ^ ((row / RPB) % CPR)) << 4)));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = wn * WN + j * 32 + lrow;
        bfr[j] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(sB + row * (2 * BK_) + ((kc ^ ((row / RPB) % CPR)) << 4)));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
  }
  }
  __syncthreads();  // all waves are done with the slices before the epilogue reuses LDS
  if constexpr (kLdsEpilogue<WN, NW, STAGES * STAGE>) {
    if constexpr (TM > 2) epi.prep();
    epilogue_lds_impl<TM>(epi, acc, std::make_index_sequence<TM>{});
  } else {
    epilogue<TM, TN, WM, WN>(P, acc, m0, n0, wm, wn, lrow, lhalf);
  }
}

// Transposed values straight from the accumulators of a wave that owns 64
// rows x one 128-column head group (TM = 2, TN = 4).  In a 32 x 32 block,
// lane (lrow, lhalf) holds column lrow and rows 8 (r / 4) + 4 lhalf + r % 4;
// with the key order of the transposed layout (slot 8 ((k >> 2) & 1) +
// 4 (k >> 3) + (k & 3) inside each 16-key group) its registers r = 0..7 are
// slots 8 lhalf .. 8 lhalf + 7 of the first group and r = 8..15 the same
// slots of the second, so each lane stores two 16-byte runs per block.  The
// host admits this only for 32-row aligned segments (a block is one
// sequence's keys kb .. kb + 31, kb a multiple of 32), or for one sequence in
// one piece, whose last block may end past its last key inside the padded
// key range).
__device__ __forceinline__ void store_vt(const Prob& P, const f32x16_t (&acc)[2][4], int m_base, int ncol0,
                                         int lrow, int lhalf) {
  const int h = (ncol0 - P.vt_col0) >> 7;
  float bias[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) bias[j] = P.bias ? bf16_to_f32(P.bias[ncol0 + 32 * j + lrow]) : 0.f;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int m = m_base + 32 * i;
    if (m >= P.M) continue;
    int z, key;
    if (m < P.vt_split) {
      z = m / P.vt_rows0;
      key = P.vt_key0 + m % P.vt_rows0;
    } else {
      const int mm = m - P.vt_split;
      z = mm / P.vt_rows1;
      key = P.vt_key1 + mm % P.vt_rows1;
    }
    bf16_t* base = P.vt + ((int64_t)(z * P.vt_heads + h) * 128 + lrow) * P.vt_ld + key + 8 * lhalf;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x16_t& a = acc[i][j];
      const float b = bias[j];
      bf16_t* row = base + (int64_t)(32 * j) * P.vt_ld;
      *(uint4*)row = make_uint4(pack_bf16x2(a[0] + b, a[1] + b), pack_bf16x2(a[2] + b, a[3] + b),
                                pack_bf16x2(a[4] + b, a[5] + b), pack_bf16x2(a[6] + b, a[7] + b));
      *(uint4*)(row + 16) = make_uint4(pack_bf16x2(a[8] + b, a[9] + b), pack_bf16x2(a[10] + b, a[11] + b),
                                       pack_bf16x2(a[12] + b, a[13] + b), pack_bf16x2(a[14] + b, a[15] + b));
    }
  }
}

// vmcnt(N) and lgkmcnt(0) in one wait (same encoding as wait_vmcnt).
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | ((N >> 4) << 14));
}

// Workgroup barrier without the workgroup-scope fence of __syncthreads: that
// fence waits for every outstanding global load of the wave, copies to LDS
// included, which would drain the copies a deeper pipeline keeps in flight.
// The memory clobber keeps the compiler from moving memory operations across
// it; callers wait for their own LDS reads and copies first.
__device__ __forceinline__ void barrier_no_fence() { asm volatile("s_barrier" ::: "memory"); }

// 256 x 256 tiles, 8 waves of 64 x 128, BK = 64, with the whole 160 KB of
// LDS as a ring of five 32 KB operand slices: operand i (W slice s = 2s,
// A slice s = 2s + 1) lives in unit i % 5.  When slice kt starts, the units
// of slice kt-1 are free and receive A slice kt+1 and W slice kt+2, so W
// slices are copied two slices ahead of use and A slices one ahead, and the
// end-of-slice wait leaves the W copies in flight.  The weights lead: they
// come cold from HBM, while A was mostly written just before (about 3%
// faster over the block-stack shapes than A leading; same result bits).
// The substep schedule is the one of the two-stage kernel above (fragments
// double-buffered in registers, LDS reads of the next substep between the
// MFMAs).
// Requires K % 64 == 0, K >= 128 and the LDS-staged epilogue's conditions.
template <int KIND>
__global__ __launch_bounds__(512) void gemm_bf16_ring_kernel(Batch b) {
  constexpr int BM = 256, BN = 256, BK_ = 64, WGN = 2;
  constexpr int WM = 64, WN = 128, TM = 2, TN = 4;
  constexpr int UNIT = 256 * BK_ * 2;  // one operand slice
  constexpr int INS = 4;                // 1 KB copies per wave per operand slice
  __shared__ __attribute__((aligned(1024))) char smem[5 * UNIT];

  if ((int)blockIdx.x >= b.total) return;
  int lt = xcd_remap(blockIdx.x, b.total);
  const bool second = lt >= b.tiles0;
  Prob P = second ? b.p1 : b.p0;
  if (second) lt -= b.tiles0;
  constexpr int GROUP = 8;
  const int in_group = GROUP * P.tiles_n;
  const int gid = lt / in_group;
  const int first_m = gid * GROUP;
  const int gsz = min(P.tiles_m - first_m, GROUP);
  const int tm = first_m + (lt % in_group) % gsz;
  const int tn = (lt % in_group) / gsz;
  const int m0 = tm * BM, n0 = tn * BN;
  // per-segment gate vectors: the host admits only BM | gseg
  if (P.gseg > 0) P.gate += (int64_t)(m0 / P.gseg) * P.gstride;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const int lrow = lane & 31, lhalf = lane >> 5;

  // per-lane source byte offsets: copy j of this wave moves rows
  // 8 (4 wave + j) .. + 7 of the slice, 16-byte chunks XOR-swizzled by
  // ((row >> 1) & 7) as in the two-stage kernel
  uint32_t aoff[INS], boff[INS];
#pragma unroll
  for (int j = 0; j < INS; ++j) {
    const int row = 8 * (wave * INS + j) + (lane >> 3);
    const int c = (lane & 7) ^ ((row >> 1) & 7);
    aoff[j] = ((uint32_t)min(m0 + row, P.M - 1) * (uint32_t)P.lda + c * 8) * 2u;
    boff[j] = ((uint32_t)min(n0 + row, P.N - 1) * (uint32_t)P.ldw + c * 8) * 2u;
  }
  auto unit = [&](int op) { return smem + (op % 5) * UNIT; };
  auto issue_a = [&](int s) {
    char* d = unit(2 * s + 1);
    const uint32_t so = (uint32_t)s * BK_ * 2;
#pragma unroll
    for (int j = 0; j < INS; ++j) buf_lds16(P.A, (lds_void_t*)(d + (wave * INS + j) * 1024), aoff[j], so);
  };
  auto issue_w = [&](int s) {
    char* d = unit(2 * s);
    const uint32_t so = (uint32_t)s * BK_ * 2;
#pragma unroll
    for (int j = 0; j < INS; ++j) buf_lds16(P.W, (lds_void_t*)(d + (wave * INS + j) * 1024), boff[j], so);
  };
  auto rd = [&](int kt, int s, bf16x8_t(&af)[TM], bf16x8_t(&bfr)[TN]) {
    const char* sA = unit(2 * kt + 1);
    const char* sB = unit(2 * kt);
    const int kc = 2 * s + lhalf;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int row = wm * WM + i * 32 + lrow;
      af[i] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(sA + row * 128 + ((kc ^ ((row >> 1) & 7)) << 4)));
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int row = wn * WN + j * 32 + lrow;
      bfr[j] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(sB + row * 128 + ((kc ^ ((row >> 1) & 7)) << 4)));
    }
  };
  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  EpiLds<KIND> epi(P, m0 + wm * WM, n0 + wn * WN, lrow, lhalf, (float*)smem + wave * (32 * 128));
  epi.prep();
  auto mm = [&](const bf16x8_t(&af)[TM], const bf16x8_t(&bfr)[TN]) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
  };
  // one MFMA, then the copies of this substep (if any) and two LDS reads,
  // three times; then the other five MFMAs; a fence closes the substep
  auto sched = [&](auto with_copy) {
    constexpr bool WithCopy = decltype(with_copy)::value;
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      if constexpr (WithCopy) __builtin_amdgcn_sched_group_barrier(0x010, 2, 0);  // VMEM
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // DS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, TM * TN - 3, 0);
    __builtin_amdgcn_sched_barrier(0);
  };
  using copy_t = std::integral_constant<bool, true>;
  using nocopy_t = std::integral_constant<bool, false>;

  const int nk = P.K / BK_;  // >= 2
  bf16x8_t a0[TM], b0[TN], a1[TM], b1[TN];
  issue_w(0);
  issue_a(0);
  issue_w(1);
  wait_vmcnt_lgkm0<INS>();  // slice 0 has landed; W slice 1 may be in flight
  barrier_no_fence();
  rd(0, 0, a0, b0);
  // slice kt with A slice kt+1 (H1) and W slice kt+2 (H2) copied meanwhile
  auto slice = [&](int kt, auto h1, auto h2) {
    constexpr bool H1 = decltype(h1)::value, H2 = decltype(h2)::value;
    if constexpr (H1) issue_a(kt + 1);
    rd(kt, 1, a1, b1); mm(a0, b0);
    if constexpr (H1) sched(copy_t{}); else sched(nocopy_t{});
    if constexpr (H2) issue_w(kt + 2);
    rd(kt, 2, a0, b0); mm(a1, b1);
    if constexpr (H2) sched(copy_t{}); else sched(nocopy_t{});
    rd(kt, 3, a1, b1); mm(a0, b0); sched(nocopy_t{});
    mm(a1, b1);
    // slice kt+1 has landed (W slice kt+2 may still be in flight) and every
    // LDS read of slice kt has returned, so after the barrier its units are free
    if constexpr (H2) wait_vmcnt_lgkm0<INS>();
    else __builtin_amdgcn_s_waitcnt(0);
    barrier_no_fence();
  };
  using yes = std::integral_constant<bool, true>;
  using no = std::integral_constant<bool, false>;
  for (int kt = 0; kt < nk - 2; ++kt) {
    slice(kt, yes{}, yes{});
    rd(kt + 1, 0, a0, b0);
  }
  slice(nk - 2, yes{}, no{});
  rd(nk - 1, 0, a0, b0);
  rd(nk - 1, 1, a1, b1); mm(a0, b0); sched(nocopy_t{});
  rd(nk - 1, 2, a0, b0); mm(a1, b1); sched(nocopy_t{});
  rd(nk - 1, 3, a1, b1); mm(a0, b0); sched(nocopy_t{});
  mm(a1, b1);
  __syncthreads();  // every wave is done with the ring before the epilogue reuses LDS
  if constexpr (KIND == EPI_K_STORE) {
    const int ncol0 = n0 + wn * WN;  // wave-uniform: whole head groups are values or not
    if (P.vt && ncol0 >= P.vt_col0 && ncol0 < P.vt_col0 + 128 * P.vt_heads) {
      store_vt(P, acc, m0 + wm * WM, ncol0, lrow, lhalf);
      return;
    }
  }
  epilogue_lds_impl<TM>(epi, acc, std::make_index_sequence<TM>{});
}

typedef __bf16 bf16x8v_t __attribute__((ext_vector_type(8)));

// Small-N projection (the final layer, N = C <= 128): v[m][c] = sum_k A[m][k] W[c][k]
// + bias[c], or with x != nullptr the Euler update x[m][c] += alpha * v[m][c]
// fused in.  16 rows per workgroup, the K range split over 4 waves, MFMA
// 16x16x32 bf16; A rows stream from HBM once, W (N x K, a few hundred KB)
// stays in L2.  The 4 partial tiles are summed through LDS in wave order.
template <int NT>  // N / 16 output tiles
__global__ __launch_bounds__(256) void proj_small_n_kernel(const bf16_t* __restrict__ A, int64_t lda,
                                                           const bf16_t* __restrict__ W, int64_t ldw,
                                                           const bf16_t* __restrict__ bias, float* out,
                                                           int64_t ldo, float* x, int64_t ldx, float alpha,
                                                           int M, int K) {
  __shared__ float part[4][16][NT * 16 + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m0 = blockIdx.x * 16;
  const int lr = lane & 15, lq = lane >> 4;  // row / column within 16, k-quarter of the 32-deep step
  const int row = min(m0 + lr, M - 1);
  const int ksteps = K / 32, per = (ksteps + 3) / 4;
  const int s0 = wave * per, s1 = min(ksteps, s0 + per);
  f32x4_t acc[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const bf16_t* ap = A + (int64_t)row * lda + 8 * lq;
  const bf16_t* wp = W + (int64_t)lr * ldw + 8 * lq;
  for (int st = s0; st < s1; ++st) {
    const bf16x8_t a = __builtin_bit_cast(bf16x8_t, *(const uint4*)(ap + 32 * st));
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const bf16x8_t w = __builtin_bit_cast(bf16x8_t, *(const uint4*)(wp + (int64_t)16 * j * ldw + 32 * st));
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, w, acc[j], 0, 0, 0);
    }
  }
  // acc[j][i] = C[row 4 lq + i][col 16 j + lr]
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) part[wave][4 * lq + i][16 * j + lr] = acc[j][i];
  __syncthreads();
  for (int e = threadIdx.x; e < 16 * NT * 16; e += 256) {
    const int r = e / (NT * 16), c = e % (NT * 16);
    const int m = m0 + r;
    if (m >= M) continue;
    float v = part[0][r][c] + part[1][r][c] + part[2][r][c] + part[3][r][c];
    if (bias) v += bf16_to_f32(bias[c]);
    if (x) x[(int64_t)m * ldx + c] += alpha * v;
    else out[(int64_t)m * ldo + c] = v;
  }
}

struct Cfg {
  int bm, bn, wn, wg_per_cu, threads, bk;
  bool lds_epi;
  float eff;
  bool dma;
  void (*fn)(Batch);
  int min_k;  // smallest K the kernel's pipeline admits
};

// eff: relative MFMA efficiency of a full tile (measured ordering); the
// chooser minimises rounds x per-round work / eff over the configs a
// problem admits.
#define DIT_DMA_CFG(BM, BN, WGM, WGN, BK_, ST, WPC, EFF)                                      \
  {BM, BN, BN / WGN, WPC, 64 * WGM * WGN, BK_,                                                 \
   kLdsEpilogue<BN / WGN, WGM * WGN, ST * (BM + BN) * BK_ * 2>, EFF, true,                     \
   gemm_bf16_dma_kernel<BM, BN, WGM, WGN, BK_, ST>, 0}
const Cfg kCfgs[] = {
    {256, 256, 128, 1, 512, 64, true, 1.02f, true, gemm_bf16_ring_kernel<EPI_K_ANY>, 128},
    DIT_DMA_CFG(256, 256, 4, 2, 64, 2, 1, 1.00f),
    DIT_DMA_CFG(256, 128, 4, 1, 64, 2, 1, 0.72f),
    DIT_DMA_CFG(128, 128, 4, 1, 64, 2, 2, 0.85f),
    DIT_DMA_CFG(32, 256, 1, 4, 64, 2, 2, 0.45f),
    {256, 128, 128, 1, 256, 64, false, 0.60f, false, gemm_bf16_kernel<256, 128, 4, 1>, 0},
    {128, 128, 128, 2, 256, 64, false, 0.55f, false, gemm_bf16_kernel<128, 128, 4, 1>, 0},
    {32, 256, 64, 2, 256, 64, false, 0.30f, false, gemm_bf16_kernel<32, 256, 1, 4>, 0},
};
#undef DIT_DMA_CFG
constexpr int kNumCfgs = sizeof(kCfgs) / sizeof(kCfgs[0]);

Prob make_prob(const GemmArgs& g, int bm, int bn) {
  Prob p;
  p.A = (const bf16_t*)g.A; p.lda = g.lda;
  p.W = (const bf16_t*)g.W; p.ldw = g.ldw;
  p.bias = (const bf16_t*)g.bias;
  p.C = g.C; p.ldc = g.ldc;
  p.gate = g.gate;
  p.gseg = g.gseg; p.gstride = g.gstride;
  p.M = g.M; p.N = g.N; p.K = g.K;
  p.flags = g.flags; p.rms_cols = g.rms_cols;
  p.gelu_from = g.gelu_from; p.gap_at = g.gap_at; p.gap = g.gap;
  p.tiles_m = (g.M + bm - 1) / bm;
  p.tiles_n = (g.N + bn - 1) / bn;
  p.vt = (bf16_t*)g.vt;
  p.vt_col0 = g.vt_col0; p.vt_heads = g.vt_heads; p.vt_ld = g.vt_ld; p.vt_split = g.vt_split;
  p.vt_rows0 = g.vt_rows0; p.vt_key0 = g.vt_key0; p.vt_rows1 = g.vt_rows1; p.vt_key1 = g.vt_key1;
  return p;
}

int pick_cfg(const GemmArgs* g, int n, int n_cu) {
  bool rms = false, aligned = true;
  for (int i = 0; i < n; ++i) {
    rms |= g[i].rms_cols > 0;
    aligned &= (g[i].lda % 8) == 0 && (g[i].ldw % 8) == 0;
  }
  bool epi_ok = true;  // conditions of the LDS-staged epilogue
  for (int i = 0; i < n; ++i) {
    epi_ok &= (g[i].N % 8) == 0 && (g[i].ldc % 4) == 0;
    epi_ok &= g[i].gelu_from >= g[i].N || (g[i].gelu_from % 4) == 0;
    epi_ok &= g[i].gap == 0 || ((g[i].gap_at | g[i].gap) % 4) == 0;
  }
  bool off32 = true;  // byte offsets of every A / W row fit the buffer loads' 32 bits
  for (int i = 0; i < n; ++i) {
    off32 &= ((uint64_t)(g[i].M - 1) * g[i].lda + g[i].K) * 2 <= 0xffffffffull;
    off32 &= ((uint64_t)(g[i].N - 1) * g[i].ldw + g[i].K) * 2 <= 0xffffffffull;
  }
  auto admits = [&](const Cfg& k) {
    if (rms && k.wn % 128) return false;
    for (int i = 0; i < n; ++i)
      if (g[i].gseg > 0 && g[i].gseg % k.bm) return false;
    if (!k.dma) return true;
    if (!aligned || !off32 || (k.lds_epi && !epi_ok)) return false;
    for (int i = 0; i < n; ++i)
      if (g[i].K % k.bk || g[i].K < k.min_k) return false;
    return true;
  };
  bool shallow = true;  // K <= 256: the tile writes dominate, more workgroups stream better
  for (int i = 0; i < n; ++i) shallow &= g[i].K <= 256 && g[i].M >= 512;
  if (shallow)
    for (int c = 0; c < kNumCfgs; ++c)
      if (kCfgs[c].bm == 128 && kCfgs[c].bn == 128 && admits(kCfgs[c])) return c;
  int best = -1;
  double best_t = 1e300;
  for (int c = 0; c < kNumCfgs; ++c) {
    const Cfg& k = kCfgs[c];
    if (!admits(k)) continue;
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

hipError_t launch_proj_small_n(const void* A, int64_t lda, const void* W, int64_t ldw, const void* bias,
                               float* out, int64_t ldo, float* x, int64_t ldx, float alpha, int M, int N,
                               int K, hipStream_t s) {
  if (K % 32 || N % 16 || N > 128 || M < 1) return hipErrorInvalidValue;
  const dim3 grid((M + 15) / 16);
#define DIT_PROJ(NT_)                                                                             \
  case NT_:                                                                                       \
    hipLaunchKernelGGL(proj_small_n_kernel<NT_>, grid, dim3(256), 0, s, (const bf16_t*)A, lda,     \
                       (const bf16_t*)W, ldw, (const bf16_t*)bias, out, ldo, x, ldx, alpha, M, K); \
    break;
  switch (N / 16) {
    DIT_PROJ(1) DIT_PROJ(2) DIT_PROJ(3) DIT_PROJ(4) DIT_PROJ(5) DIT_PROJ(6) DIT_PROJ(7) DIT_PROJ(8)
    default:
      return hipErrorInvalidValue;
  }
#undef DIT_PROJ
  return hipGetLastError();
}

// The kernel for these problems (config c): the 256 x 256 ring kernel takes
// a specialised epilogue when every problem admits it.
static void (*kernel_for(const GemmArgs* g, int n, int c))(Batch) {
  void (*fn)(Batch) = kCfgs[c].fn;
  if (fn == gemm_bf16_ring_kernel<EPI_K_ANY>) {
    bool store = true, gated = true;
    for (int i = 0; i < n; ++i) {
      const GemmArgs& a = g[i];
      const bool plain = !(a.flags & (DIT_EPI_F32 | DIT_EPI_SILU));
      store &= plain && !(a.flags & DIT_EPI_GATED_RES) && (a.gelu_from >= a.N || a.gelu_from % 128 == 0) &&
               (a.gap == 0 || a.gap_at % 128 == 0);
      gated &= plain && (a.flags & DIT_EPI_GATED_RES) && a.rms_cols == 0 && a.gelu_from >= a.N && a.gap == 0;
    }
    if (store) fn = gemm_bf16_ring_kernel<EPI_K_STORE>;
    else if (gated) fn = gemm_bf16_ring_kernel<EPI_K_GATED>;
  }
  return fn;
}

// The transposed-value output: the store kernel, head groups inside the
// output, no column gap or GELU or RMS over them, 32-row aligned segments
// and key offsets, and 16-byte aligned rows of vt.
static bool vt_ok(const GemmArgs* g, int n, int c) {
  if (c < 0 || kernel_for(g, n, c) != gemm_bf16_ring_kernel<EPI_K_STORE>) return false;
  for (int i = 0; i < n; ++i) {
    const GemmArgs& a = g[i];
    if (!a.vt) continue;
    const int end = a.vt_col0 + 128 * a.vt_heads;
    if (a.vt_heads < 1 || a.vt_col0 % 128 || end > a.N || a.vt_ld % 8 || ((uintptr_t)a.vt & 15)) return false;
    if (a.vt_col0 < a.rms_cols || end > a.gelu_from || (a.gap && end > a.gap_at)) return false;
    // one sequence in one piece may end inside a 32-row block: that block's
    // rows past M repeat row M - 1 (clamped loads), so the keys it writes past
    // the sequence hold finite values that attention masks out
    const bool single = a.vt_split >= a.M && a.vt_rows0 >= a.M;
    if (single) {
      if (a.vt_key0 % 32 || a.vt_key0 + (a.M + 31) / 32 * 32 > a.vt_ld) return false;
    } else if (a.M % 32 || a.vt_rows0 % 32 || a.vt_key0 % 32 || a.vt_rows0 < 1) {
      return false;
    }
    if (a.vt_split < a.M && (a.vt_split % 32 || a.vt_rows1 % 32 || a.vt_key1 % 32 || a.vt_rows1 < 1)) return false;
  }
  return true;
}

bool gemm_bf16_fuses_vt(const GemmArgs* g, int n, int n_cu) {
  if (n < 1 || n > 2) return false;
  return vt_ok(g, n, pick_cfg(g, n, n_cu));
}

hipError_t launch_gemm_bf16(const GemmArgs* g, int n, hipStream_t stream, int n_cu) {
  if (n < 1 || n > 2) return hipErrorInvalidValue;
  for (int i = 0; i < n; ++i)
    if (g[i].gseg < 0 || (g[i].gseg > 0 && (g[i].gseg % 32 || !(g[i].flags & DIT_EPI_GATED_RES))))
      return hipErrorInvalidValue;
  const int c = pick_cfg(g, n, n_cu);
  if (c < 0) return hipErrorInvalidValue;
  bool want_vt = false;
  for (int i = 0; i < n; ++i) want_vt |= g[i].vt != nullptr;
  if (want_vt && !vt_ok(g, n, c)) return hipErrorInvalidValue;
  const Cfg& k = kCfgs[c];
  void (*fn)(Batch) = kernel_for(g, n, c);
  Batch b;
  b.p0 = make_prob(g[0], k.bm, k.bn);
  b.p1 = n > 1 ? make_prob(g[1], k.bm, k.bn) : b.p0;
  b.tiles0 = b.p0.tiles_m * b.p0.tiles_n;
  b.total = b.tiles0 + (n > 1 ? b.p1.tiles_m * b.p1.tiles_n : 0);
  if (b.total == 0) return hipSuccess;
  hipLaunchKernelGGL(fn, dim3(b.total), dim3(k.threads), 0, stream, b);
  return hipGetLastError();
}

}  // namespace dit
