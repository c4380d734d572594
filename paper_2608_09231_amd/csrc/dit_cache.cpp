// Host driver and C ABI of the budget-aware cached DiT sampler.
//
// Per sample: text projection, timestep/pooled embeddings and the whole
// modulation table (all steps) run once.  Per step t: patch embed + the
// indicator kernel (modulated first-block input and its relative-L1
// partial sums) + a fixed-order reduction written straight into pinned
// host memory; the host waits for that one event, evaluates the gate
// (Eq. 1) on the 8-feature state and applies Alg. 2's budget rules in
// double precision; then it enqueues either the full block stack (with
// the residual refresh) or the residual reuse, and the final layer with
// the Euler update.  Every tensor operation is a HIP kernel.
#include <hip/hip_runtime.h>

#include <chrono>
#include <cmath>
#include <mutex>
#include <cstdio>
#include <cstring>
#include <string>
#include <type_traits>
#include <vector>

#include "../../include/dit_cache.h"
#include "../../include/dit_kernels.h"
#include "common.h"
#include "kernels.h"

namespace {

thread_local std::string g_create_error;

struct Lin {
  const void* w = nullptr;
  const void* b = nullptr;
  int out = 0, in = 0;
};
struct DoubleW { Lin qkv[2], o[2], mlp0[2], mlp1[2]; };  // [0] image, [1] text stream
struct SingleW { Lin l1, l2; };
struct CrossW { const void* mod_off = nullptr; Lin qkv, o, xq, xkv, xo, ffn0, ffn1; };

struct Model {
  Lin img_in, txt_in, time0, time2, pool0, pool2, mod, fin;
  std::vector<DoubleW> dbl;
  std::vector<SingleW> sgl;
  std::vector<CrossW> crs;
};

// One dense ReLU network: widths d_0..d_{k-1}, layers W_l [d_l, d_{l-1}].
struct DenseNet {
  std::vector<int> widths;
  std::vector<std::vector<double>> W, b;
};

// The gate: optional branches (each reads the next d_0 features, ReLU after
// every layer) feeding a trunk (ReLU after every hidden layer, none on the
// logit); without branches the trunk reads the features directly.
struct GateMLP {
  int d_in = 0;
  bool z = false;
  std::vector<double> mu, sd;
  std::vector<DenseNet> branches;
  DenseNet trunk;
};

struct Pending {
  int cls;
  double work;
  hipEvent_t a, b;
};

}  // namespace

// One sample's device state and its pacing-rule state (Alg. 2).
struct Lane {
  void* h = nullptr;        // [N, H] patch embedding of this step (the block stack's input)
  void* mbuf[3] = {};       // [N, H] indicator tensors (rotating)
  void* r = nullptr;        // [nb, N, H] cached residual per branch
  void* txt = nullptr;      // [nb, Nt, H] projected text tokens
  float* x_last = nullptr;  // f32 [N, C]: UniPC's corrected sample of the previous step
  float* mh[3] = {};        // f32 [N, C]: UniPC data predictions (rotating)
  float* xalt = nullptr;    // f32 [N, C]: second latent buffer (the reuse candidate's Euler result)
  float* vspec = nullptr;   // f32 [N, C]: the reuse candidate's velocity (UniPC)
  double* mag = nullptr;    // f64 [3]: sum |m| of each indicator buffer (column-sliced step kernel)
  // video blocks: the cross-attention keys | values of the text tokens [nb, n_cross, Nt, 2H] and (bf16)
  // the values transposed [nb, n_cross, heads, 128, round_up(Nt, 64)]; the same at every step, so
  // formed once per sample
  void* xkv = nullptr;
  void* xvt = nullptr;
  int cnt = 0, t_last = 0, i_prev = -1, i_last = -1, i_new = 0;
  double acc = 0.0;
  bool dec = true;
  bool spec = false;  // this step's fused launch formed a reuse candidate
};

struct dit_cache {
  dit_model_config cfg{};
  hipStream_t stream = nullptr;
  int n_cu = 256;
  bool bf16 = true;
  size_t esz = 2;
  int H = 0, F = 0, N = 0, Nt = 0, L = 0, C = 0, nb = 1, n_mod = 0, ldY = 0;
  // bf16 MMDiT: every sequence computed at a step (each branch of each
  // sample that computes) runs the block stack together, stream-major rows
  // [txt_0; ...; txt_{Q-1}; img_0; ...; img_{Q-1}] (see full_stack_multi)
  bool stacked = false;

  void* wdev = nullptr;
  size_t wbytes = 0;
  Model M;

  std::vector<Lane> lanes;  // per-sample state, grown on demand
  int cap_seq = 0;          // sequences the block-stack workspace holds

  // workspace (storage dtype unless noted)
  void* xs = nullptr;      // [N, C]
  void* X = nullptr;       // [cap_seq L, H] joint hidden state
  void* A = nullptr;       // [cap_seq L, H] modulated block input
  void* Y = nullptr;       // [cap_seq L, 4H+F]: q | k | v | attn out | mlp hidden
  void* vt = nullptr;      // bf16 [cap_seq, heads, 128, round_up(L, 64)]
  float* modq = nullptr;   // f32 [cap_seq, n_mod]: gathered modulation vectors of one step
  void* yf = nullptr;      // [N, H] final-layer input
  float* vel = nullptr;    // f32 [nb, N, C]
  float* ones = nullptr;   // f32 [H] (ungated residual)
  double* partials = nullptr;
  int max_partials = 0;
  // column-sliced step kernel (bf16, C = 64): LN statistics matrix of the
  // patch embedding (bf16 hi / lo [80][64]) and the candidate partials
  void* st_hi = nullptr;
  void* st_lo = nullptr;
  float st_bbar = 0.f, st_b2 = 0.f;
  float* cand = nullptr;
  double* sums_host = nullptr;  // pinned, mapped [lanes, 4]
  double* sums_dev = nullptr;
  int cap_sums = 0;
  hipEvent_t ev_sums = nullptr;

  // per-call tables, grown on demand (sized by T and the modulation slots:
  // one per branch of each sample with pooled text, else one)
  int cap_T = 0, cap_slots = 0;
  float* mod = nullptr;    // f32 [slots, T, n_mod]
  float* fconst = nullptr; // f32 [slots, T, 128]: final-layer constants A | B of each table row
  float* modx = nullptr;   // f32 [slots, n_cross, T, 6H]
  void* temb = nullptr;    // [T, time_dim]
  void* th = nullptr;      // [T, H]
  float* tv = nullptr;     // f32 [T, H]
  void* pooled = nullptr;  // [1, ctx]
  void* ph = nullptr;      // [1, H]
  float* pv = nullptr;     // f32 [1, H]
  void* svec = nullptr;    // [T, H]
  double* sig_dev = nullptr;

  std::string err;

  bool prof = false;
  dit_stats stats{};
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;
  std::vector<Pending> pending;
  // end event of the last timed scope: the next scope starts from it unless
  // the host has waited in between (then the GPU may have idled)
  hipEvent_t ev_chain = nullptr;
};

namespace {

using dit::GemmArgs;

dit_status fail(dit_cache* c, dit_status s, const std::string& msg) {
  if (c) c->err = msg; else g_create_error = msg;
  return s;
}

#define HIPCK(expr)                                                                    \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(c, DIT_EHIP, std::string(#expr) + ": " + hipGetErrorString(e_));     \
  } while (0)

#define TRY(expr)                          \
  do {                                     \
    dit_status s_ = (expr);                \
    if (s_ != DIT_OK) return s_;           \
  } while (0)

inline size_t rup(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ---------------------------------------------------------------- profiling
hipEvent_t next_event(dit_cache* c) {
  if (c->ev_used == c->ev_pool.size()) {
    hipEvent_t e;
    // timing only: no system-scope release / acquire around the timestamps
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    c->ev_pool.push_back(e);
  }
  return c->ev_pool[c->ev_used++];
}

struct Scope {
  dit_cache* c;
  int cls;
  double work;
  hipEvent_t a = nullptr;
  // Back-to-back scopes share their boundary event (one timestamp per kernel
  // class launch instead of two); a scope's span then also holds the launch
  // gap before its first kernel.
  Scope(dit_cache* c_, int cls_, double work_) : c(c_), cls(cls_), work(work_) {
    if (c->prof) {
      a = c->ev_chain;
      if (!a) {
        a = next_event(c);
        if (a) hipEventRecord(a, c->stream);
      }
    }
  }
  ~Scope() {
    if (c->prof && a) {
      hipEvent_t b = next_event(c);
      if (b) {
        hipEventRecord(b, c->stream);
        c->pending.push_back({cls, work, a, b});
      }
      c->ev_chain = b;
    }
  }
};

// The host is about to wait for the GPU: the next timed scope starts afresh.
void break_chain(dit_cache* c) { c->ev_chain = nullptr; }

void collect_events(dit_cache* c) {
  if (!c->prof) return;
  hipStreamSynchronize(c->stream);
  for (const Pending& p : c->pending) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      c->stats.ms[p.cls] += ms;
      c->stats.work[p.cls] += p.work;
      c->stats.launches[p.cls] += 1;
    }
  }
  c->pending.clear();
  c->ev_used = 0;
  c->ev_chain = nullptr;
}

// ---------------------------------------------------------------- helpers
const char* sp(const dit_cache* c, const void* base, size_t elem_off) {
  return (const char*)base + elem_off * c->esz;
}
char* sp(const dit_cache* c, void* base, size_t elem_off) { return (char*)base + elem_off * c->esz; }

GemmArgs lin_args(const dit_cache* c, const void* A, int64_t lda, const Lin& l, void* C, int64_t ldc,
                  int M, int flags = DIT_EPI_STORE) {
  GemmArgs g{};
  g.A = A; g.lda = lda; g.W = l.w; g.ldw = l.in; g.bias = l.b;
  g.C = C; g.ldc = ldc; g.gate = nullptr;
  g.M = M; g.N = l.out; g.K = l.in; g.flags = flags;
  return g;
}

dit_status gemm(dit_cache* c, GemmArgs* g, int n, int cls) {
  double flops = 0;
  for (int i = 0; i < n; ++i) flops += 2.0 * g[i].M * (double)g[i].N * g[i].K;
  Scope sc(c, cls, flops);
  if (c->bf16) {
    HIPCK(dit::launch_gemm_bf16(g, n, c->stream, c->n_cu));
  } else {
    HIPCK(dit::launch_gemm_f32(g, n, c->stream));
    for (int i = 0; i < n; ++i)
      if (g[i].rms_cols > 0)
        HIPCK(dit::launch_rms_heads_f32((float*)g[i].C, g[i].ldc, g[i].M, g[i].rms_cols,
                                        c->cfg.head_dim, c->stream));
  }
  return DIT_OK;
}

template <typename Fn>
dit_status typed(dit_cache* c, Fn fn) {
  hipError_t e = c->bf16 ? fn((bf16_t*)nullptr) : fn((float*)nullptr);
  if (e != hipSuccess) return fail(c, DIT_EHIP, std::string("kernel launch: ") + hipGetErrorString(e));
  return DIT_OK;
}

dit_status ln_mod(dit_cache* c, const void* x, int64_t ldx, void* out, int64_t ldo, int rows, int split,
                  const float* sh0, const float* sc0, const float* sh1, const float* sc1, int cls,
                  int seg0 = 0x7fffffff, int seg1 = 0x7fffffff, int64_t mstride = 0) {
  Scope s(c, cls, 2.0 * rows * c->H * c->esz);
  return typed(c, [&](auto* tp) {
    using T = std::remove_pointer_t<decltype(tp)>;
    return dit::launch_ln_mod<T>((const T*)x, ldx, (T*)out, ldo, rows, c->H, split, sh0, sc0, sh1, sc1,
                                 c->stream, seg0, seg1, mstride);
  });
}

// attention over joint rows: q,k,v inside Y (or separate), output into o;
// nseq stacked sequences in one launch (bf16; see launch_flash_attn_bf16)
// vt_ready: the projection has already written the transposed values into vt_ws
dit_status attention(dit_cache* c, const void* q, int64_t ldq, const void* k, int64_t ldk, const void* v,
                     int64_t ldv, void* o, int64_t ldo, int Lq, int Lk, void* vt_ws, int split = 0x7fffffff,
                     int64_t gap = 0, int nseq = 1, int64_t zs = 0, int64_t gz = 0, bool vt_ready = false) {
  const int heads = c->cfg.heads, hd = c->cfg.head_dim;
  const double flops = 4.0 * Lq * (double)Lk * heads * hd * nseq;
  if (c->bf16) {
    if (!vt_ready) {
      Scope s(c, DIT_K_FULL_OTHER, 2.0 * Lk * heads * hd * 2 * nseq);
      HIPCK(dit::launch_transpose_v_bf16(v, ldv, vt_ws, Lk, heads, c->stream, split, gap, nseq, zs, gz));
    }
    Scope s(c, DIT_K_ATTN, flops);
    // q and k leave the projection through a unit-gain RMS norm: bounded logits
    HIPCK(dit::launch_flash_attn_bf16(q, ldq, k, ldk, vt_ws, (int)rup(Lk, 64), o, ldo, Lq, Lk, heads,
                                      true, c->stream, split, gap, nseq, zs, gz));
  } else {
    if (nseq != 1) return fail(c, DIT_EINVAL, "f32 attention runs one sequence per launch");
    Scope s(c, DIT_K_ATTN, flops);
    HIPCK(dit::launch_attn_f32((const float*)q, ldq, (const float*)k, ldk, (const float*)v, ldv,
                               (float*)o, ldo, Lq, Lk, heads, hd, c->stream));
  }
  return DIT_OK;
}

// ---------------------------------------------------------------- weights
dit_status layout(dit_cache* c, size_t* total_elems) {
  const dit_model_config& g = c->cfg;
  const int H = g.hidden, F = g.mlp_hidden, C = g.in_channels, X = g.ctx_dim;
  size_t off = 0;
  auto take = [&](Lin& l, int out, int in) {
    l.out = out; l.in = in;
    l.w = (const void*)(uintptr_t)off; off += (size_t)out * in;
    l.b = (const void*)(uintptr_t)off; off += out;
  };
  Model& m = c->M;
  take(m.img_in, H, C);
  take(m.txt_in, H, X);
  take(m.time0, H, g.time_dim);
  take(m.time2, H, H);
  if (g.pooled_text) { take(m.pool0, H, X); take(m.pool2, H, H); }
  take(m.mod, c->n_mod, H);
  m.dbl.resize(g.n_double);
  for (auto& d : m.dbl)
    for (int s = 0; s < 2; ++s) {
      take(d.qkv[s], 3 * H, H); take(d.o[s], H, H); take(d.mlp0[s], F, H); take(d.mlp1[s], H, F);
    }
  m.sgl.resize(g.n_single);
  for (auto& s : m.sgl) { take(s.l1, 3 * H + F, H); take(s.l2, H, H + F); }
  m.crs.resize(g.n_cross);
  for (auto& x : m.crs) {
    x.mod_off = (const void*)(uintptr_t)off; off += 6 * (size_t)H;
    take(x.qkv, 3 * H, H); take(x.o, H, H); take(x.xq, H, H); take(x.xkv, 2 * H, H); take(x.xo, H, H);
    take(x.ffn0, F, H); take(x.ffn1, H, F);
  }
  take(m.fin, C, H);
  *total_elems = off;
  return DIT_OK;
}

void rebase(dit_cache* c) {
  auto fix = [&](const void*& p) { p = (const char*)c->wdev + (uintptr_t)p * c->esz; };
  auto fl = [&](Lin& l) { if (l.out) { fix(l.w); fix(l.b); } };
  Model& m = c->M;
  fl(m.img_in); fl(m.txt_in); fl(m.time0); fl(m.time2); fl(m.pool0); fl(m.pool2); fl(m.mod); fl(m.fin);
  for (auto& d : m.dbl)
    for (int s = 0; s < 2; ++s) { fl(d.qkv[s]); fl(d.o[s]); fl(d.mlp0[s]); fl(d.mlp1[s]); }
  for (auto& s : m.sgl) { fl(s.l1); fl(s.l2); }
  for (auto& x : m.crs) {
    fix(x.mod_off);
    fl(x.qkv); fl(x.o); fl(x.xq); fl(x.xkv); fl(x.xo); fl(x.ffn0); fl(x.ffn1);
  }
}

dit_status validate(const dit_model_config* g, std::string& why) {
  auto bad = [&](const char* m) { why = m; return DIT_ESHAPE; };
  if (g->abi_version != DIT_ABI_VERSION) { why = "abi_version mismatch"; return DIT_EINVAL; }
  if (g->dtype != DIT_DTYPE_F32 && g->dtype != DIT_DTYPE_BF16) { why = "bad dtype"; return DIT_EINVAL; }
  if (g->n_double < 0 || g->n_single < 0 || g->n_cross < 0) return bad("negative block count");
  if (g->n_double + g->n_single + g->n_cross < 1) return bad("no blocks");
  if (g->n_cross && (g->n_double || g->n_single)) return bad("video blocks cannot mix with MMDiT blocks");
  if (g->heads < 1 || g->head_dim < 1 || g->heads * g->head_dim != g->hidden) return bad("hidden != heads*head_dim");
  if (g->mlp_hidden < 1 || g->in_channels < 1 || g->ctx_dim < 1 || g->time_dim < 2 || (g->time_dim & 1))
    return bad("bad widths");
  if (g->n_img < 1 || g->n_txt < 1) return bad("token counts must be >= 1");
  if (g->batch != 1 && g->batch != 2) return bad("batch must be 1 or 2");
  if (g->hidden > 8192) return bad("hidden > 8192");
  if (g->dtype == DIT_DTYPE_BF16) {
    if (g->head_dim != 128) return bad("bf16 path needs head_dim == 128");
    if (g->hidden % 8 || g->mlp_hidden % 8 || g->ctx_dim % 8 || g->in_channels % 8 || g->time_dim % 8)
      return bad("bf16 widths must be multiples of 8");
  } else {
    if (g->hidden % 4) return bad("f32 hidden must be a multiple of 4");
    if (g->head_dim > 128 || (g->head_dim != 16 && g->head_dim != 32 && g->head_dim != 64 && g->head_dim != 128))
      return bad("f32 path needs head_dim in {16, 32, 64, 128}");
  }
  return DIT_OK;
}

template <typename P>
dit_status dalloc(dit_cache* c, P** p, size_t bytes) {
  void* q = nullptr;
  if (bytes == 0) bytes = 16;
  hipError_t e = hipMalloc(&q, bytes);
  if (e != hipSuccess) return fail(c, DIT_ENOMEM, "hipMalloc(" + std::to_string(bytes) + ") failed");
  *p = (P*)q;
  return DIT_OK;
}

// LN statistics matrix of the patch embedding for the column-sliced step
// kernel, from the host weight blob (W_in, b_in still blob offsets).
dit_status upload_stream_stats(dit_cache* c, const uint16_t* blob) {
  std::vector<uint16_t> hi((size_t)80 * 64), lo((size_t)80 * 64);
  dit::step_stream_stats(blob + (uintptr_t)c->M.img_in.w, blob + (uintptr_t)c->M.img_in.b, c->H, hi.data(),
                         lo.data(), &c->st_bbar, &c->st_b2);
  TRY(dalloc(c, &c->st_hi, hi.size() * 2));
  TRY(dalloc(c, &c->st_lo, lo.size() * 2));
  HIPCK(hipMemcpy(c->st_hi, hi.data(), hi.size() * 2, hipMemcpyHostToDevice));
  HIPCK(hipMemcpy(c->st_lo, lo.data(), lo.size() * 2, hipMemcpyHostToDevice));
  return DIT_OK;
}

// Per video block: the text tokens' keys | values, and the values transposed.
size_t xkv_elems(const dit_cache* c) { return (size_t)c->Nt * 2 * c->H; }
size_t xvt_elems(const dit_cache* c) { return (size_t)c->cfg.heads * 128 * rup(c->Nt, 64); }

void free_lane(Lane& l) {
  void* ps[] = {l.h, l.mbuf[0], l.mbuf[1], l.mbuf[2], l.r, l.txt, l.x_last, l.mh[0], l.mh[1], l.mh[2],
                l.xalt, l.vspec, l.mag, l.xkv, l.xvt};
  for (void* p : ps)
    if (p) hipFree(p);
  l = Lane{};
}

dit_status alloc_lane(dit_cache* c, Lane& l) {
  const size_t e = c->esz;
  const size_t NH = (size_t)c->N * c->H, NC = (size_t)c->N * c->C;
  TRY(dalloc(c, &l.h, NH * e));
  for (auto& m : l.mbuf) TRY(dalloc(c, &m, NH * e));
  TRY(dalloc(c, &l.r, c->nb * NH * e));
  TRY(dalloc(c, &l.txt, (size_t)c->nb * c->Nt * c->H * e));
  TRY(dalloc(c, &l.x_last, NC * 4));
  for (auto& m : l.mh) TRY(dalloc(c, &m, NC * 4));
  TRY(dalloc(c, &l.xalt, NC * 4));
  TRY(dalloc(c, &l.vspec, NC * 4));
  TRY(dalloc(c, &l.mag, 3 * sizeof(double)));
  if (c->cfg.n_cross) {
    const size_t nblk = (size_t)c->nb * c->cfg.n_cross;
    TRY(dalloc(c, &l.xkv, nblk * xkv_elems(c) * e));
    if (c->bf16) TRY(dalloc(c, &l.xvt, nblk * xvt_elems(c) * 2));
  }
  return DIT_OK;
}

// Block-stack workspace for Q sequences (stacked: Q L rows; else one).
dit_status ensure_seq(dit_cache* c, int Q) {
  if (!c->stacked) Q = 1;
  if (Q <= c->cap_seq) return DIT_OK;
  for (void* p : {c->X, c->A, c->Y, c->vt, (void*)c->modq})
    if (p) hipFree(p);
  c->X = c->A = c->Y = c->vt = nullptr;
  c->modq = nullptr;
  c->cap_seq = 0;
  const size_t e = c->esz, LB = (size_t)c->L * Q;
  TRY(dalloc(c, &c->X, LB * c->H * e));
  TRY(dalloc(c, &c->A, LB * c->H * e));
  TRY(dalloc(c, &c->Y, LB * c->ldY * e));
  if (c->bf16) {
    // keys past L stay zero for good: attention reads whole 64-key tiles, and
    // the projection that writes the transposed values never touches them
    const size_t vb = (size_t)Q * c->cfg.heads * 128 * rup(c->L, 64) * 2;
    TRY(dalloc(c, &c->vt, vb));
    HIPCK(hipMemsetAsync(c->vt, 0, vb, c->stream));
  }
  if (c->stacked && c->cfg.pooled_text) TRY(dalloc(c, &c->modq, (size_t)Q * c->n_mod * 4));
  c->cap_seq = Q;
  return DIT_OK;
}

// S sample lanes, the pinned indicator sums of each and the stack workspace
// for all their sequences.
dit_status ensure_lanes(dit_cache* c, int S) {
  while ((int)c->lanes.size() < S) {
    c->lanes.emplace_back();
    dit_status st = alloc_lane(c, c->lanes.back());
    if (st != DIT_OK) {
      free_lane(c->lanes.back());
      c->lanes.pop_back();
      return st;
    }
  }
  if (S > c->cap_sums) {
    if (c->sums_host) hipHostFree(c->sums_host);
    c->sums_host = c->sums_dev = nullptr;
    c->cap_sums = 0;
    if (hipHostMalloc((void**)&c->sums_host, (size_t)S * 4 * sizeof(double), hipHostMallocMapped) != hipSuccess)
      return fail(c, DIT_ENOMEM, "pinned host allocation failed");
    HIPCK(hipHostGetDevicePointer((void**)&c->sums_dev, c->sums_host, 0));
    c->cap_sums = S;
  }
  return ensure_seq(c, S * c->nb);
}

dit_status alloc_workspace(dit_cache* c) {
  const size_t e = c->esz;
  const int H = c->H, N = c->N;
  TRY(dalloc(c, &c->xs, (size_t)N * c->C * e));
  TRY(dalloc(c, &c->yf, (size_t)N * H * e));
  TRY(dalloc(c, &c->vel, (size_t)c->nb * N * c->C * 4));
  TRY(dalloc(c, &c->ones, (size_t)H * 4));
  {
    std::vector<float> one(H, 1.f);
    HIPCK(hipMemcpy(c->ones, one.data(), H * 4, hipMemcpyHostToDevice));
  }
  c->max_partials = std::max({dit::indicator_partials(N), dit::reuse_indicator_partials(N),
                              dit::step_fused_partials(N, H, c->nb), dit::step_stream_partials(N, H)});
  if (c->bf16 && dit::step_stream_fits(c->C, H, c->nb))
    TRY(dalloc(c, &c->cand, dit::step_stream_cand_floats(N, H, c->nb) * 4));
  TRY(dalloc(c, &c->partials, (size_t)c->max_partials * 4 * sizeof(double)));
  HIPCK(hipEventCreateWithFlags(&c->ev_sums, hipEventDisableTiming));
  return ensure_lanes(c, 1);
}

void free_per_call(dit_cache* c) {
  void* ps[] = {c->mod, c->modx, c->temb, c->th, c->tv, c->pooled, c->ph, c->pv, c->svec, c->sig_dev, c->fconst};
  for (void* p : ps)
    if (p) hipFree(p);
  c->mod = c->modx = c->tv = c->pv = c->fconst = nullptr;
  c->temb = c->th = c->pooled = c->ph = c->svec = nullptr;
  c->sig_dev = nullptr;
  c->cap_T = c->cap_slots = 0;
}

int mod_slots(const dit_cache* c, int S) { return c->cfg.pooled_text ? S * c->nb : 1; }

dit_status ensure_T(dit_cache* c, int T, int S) {
  const int slots = mod_slots(c, S);
  if (T <= c->cap_T && slots <= c->cap_slots) return DIT_OK;
  T = std::max(T, c->cap_T);
  free_per_call(c);
  const size_t e = c->esz;
  const int H = c->H;
  TRY(dalloc(c, &c->mod, (size_t)slots * T * c->n_mod * 4));
  if (c->cand) TRY(dalloc(c, &c->fconst, (size_t)slots * T * 128 * 4));
  if (c->cfg.n_cross) TRY(dalloc(c, &c->modx, (size_t)slots * c->cfg.n_cross * T * 6 * H * 4));
  TRY(dalloc(c, &c->temb, (size_t)T * c->cfg.time_dim * e));
  TRY(dalloc(c, &c->th, (size_t)T * H * e));
  TRY(dalloc(c, &c->tv, (size_t)T * H * 4));
  TRY(dalloc(c, &c->pooled, (size_t)c->cfg.ctx_dim * e));
  TRY(dalloc(c, &c->ph, (size_t)H * e));
  TRY(dalloc(c, &c->pv, (size_t)H * 4));
  TRY(dalloc(c, &c->svec, (size_t)T * H * e));
  TRY(dalloc(c, &c->sig_dev, (size_t)(T + 1) * sizeof(double)));
  c->cap_T = T;
  c->cap_slots = slots;
  return DIT_OK;
}

// ---------------------------------------------------------------- gate
// Reads "k, d_0..d_{k-1}" at blob[p]; false on a malformed header.
bool read_widths(const float* blob, size_t n, size_t& p, std::vector<int>& w) {
  if (p >= n) return false;
  const double k = blob[p];
  if (k < 2 || k > 16 || k != std::floor(k) || p + 1 + (size_t)k > n) return false;
  w.resize((int)k);
  for (int i = 0; i < (int)k; ++i) {
    const double v = blob[p + 1 + i];
    if (v < 1 || v > 4096 || v != std::floor(v)) return false;
    w[i] = (int)v;
  }
  p += 1 + (size_t)k;
  return true;
}

size_t net_params(const DenseNet& d) {
  size_t m = 0;
  for (size_t i = 1; i < d.widths.size(); ++i) m += (size_t)d.widths[i] * d.widths[i - 1] + d.widths[i];
  return m;
}

void read_params(const float* blob, size_t& p, DenseNet& d) {
  d.W.clear(); d.b.clear();
  for (size_t i = 1; i < d.widths.size(); ++i) {
    const size_t nw = (size_t)d.widths[i] * d.widths[i - 1];
    d.W.emplace_back(blob + p, blob + p + nw); p += nw;
    d.b.emplace_back(blob + p, blob + p + d.widths[i]); p += d.widths[i];
  }
}

// Eq. 1's gate from its self-describing blob: a plain MLP
// [k, widths, zflag, (mu, sd), params] or a branched network
// [-n, (k_j, widths_j) x n, k, trunk widths, zflag, (mu, sd), params of
// branch 1..n, params of the trunk] (App. A.2's two-group gate).
dit_status parse_gate(dit_cache* c, const float* blob, size_t n, GateMLP& g) {
  if (!blob || n < 4) return fail(c, DIT_EINVAL, "gate blob missing or too short");
  size_t p = 0;
  g.branches.clear();
  if (blob[0] < 0) {
    const double nb = -(double)blob[0];
    if (nb != std::floor(nb) || nb > DIT_N_FEATURES) return fail(c, DIT_EINVAL, "gate blob: bad branch count");
    p = 1;
    g.branches.resize((int)nb);
    for (auto& br : g.branches)
      if (!read_widths(blob, n, p, br.widths)) return fail(c, DIT_EINVAL, "gate blob: bad branch header");
  }
  if (!read_widths(blob, n, p, g.trunk.widths)) return fail(c, DIT_EINVAL, "gate blob: bad layer count");
  if (g.trunk.widths.back() != 1) return fail(c, DIT_EINVAL, "gate blob: output width must be 1");
  int d_in = g.trunk.widths[0];
  if (!g.branches.empty()) {
    int outs = 0;
    d_in = 0;
    for (auto& br : g.branches) { outs += br.widths.back(); d_in += br.widths[0]; }
    if (outs != g.trunk.widths[0])
      return fail(c, DIT_EINVAL, "gate blob: trunk input width != sum of branch outputs");
  }
  if (d_in > DIT_N_FEATURES) return fail(c, DIT_EINVAL, "gate blob: more than 8 inputs");
  g.d_in = d_in;
  if (p >= n) return fail(c, DIT_EINVAL, "gate blob: length mismatch");
  g.z = blob[p++] != 0.f;
  size_t need = p + (g.z ? 2 * (size_t)d_in : 0) + net_params(g.trunk);
  for (auto& br : g.branches) need += net_params(br);
  if (need != n) return fail(c, DIT_EINVAL, "gate blob: length mismatch");
  if (g.z) {
    g.mu.assign(blob + p, blob + p + d_in); p += d_in;
    g.sd.assign(blob + p, blob + p + d_in); p += d_in;
  }
  for (auto& br : g.branches) read_params(blob, p, br);
  read_params(blob, p, g.trunk);
  return DIT_OK;
}

// u <- net(u), in float64; ReLU after every layer but the last unless last_relu.
void dense_forward(const DenseNet& d, std::vector<double>& u, bool last_relu) {
  std::vector<double> nx;
  const int nl = (int)d.W.size();
  for (int l = 0; l < nl; ++l) {
    const int o = d.widths[l + 1], in = d.widths[l];
    nx.assign(o, 0.0);
    for (int j = 0; j < o; ++j) {
      double s = d.b[l][j];
      for (int i = 0; i < in; ++i) s += d.W[l][(size_t)j * in + i] * u[i];
      nx[j] = (l < nl - 1 || last_relu) ? (s > 0.0 ? s : 0.0) : s;
    }
    u.swap(nx);
  }
}

double gate_logit(const GateMLP& g, const double* f) {
  std::vector<double> u(f, f + g.d_in);
  if (g.z)
    for (int i = 0; i < g.d_in; ++i) u[i] = (u[i] - g.mu[i]) / g.sd[i];
  if (!g.branches.empty()) {
    std::vector<double> cat, part;
    int off = 0;
    for (const auto& br : g.branches) {
      part.assign(u.begin() + off, u.begin() + off + br.widths[0]);
      off += br.widths[0];
      dense_forward(br, part, true);
      cat.insert(cat.end(), part.begin(), part.end());
    }
    u.swap(cat);
  }
  dense_forward(g.trunk, u, false);
  return u[0];
}

// ---------------------------------------------------------------- steps
// One sequence through the block stack: one branch of one sample.
struct Seq {
  const void* txt;    // [Nt, H] projected text tokens
  const void* h;      // [N, H] image-token input
  void* r;            // [N, H] refreshed residual (out)
  const float* mod;   // this step's modulation vector [n_mod]
  const float* modx;  // video blocks: base of [n_cross][T][6H]
  const void* m0;     // [N, H] the first block's modulated image input (m_t), or nullptr
  const void* xkv;    // video blocks: this branch's [n_cross, Nt, 2H] text keys | values
  void* xvt;          // bf16 video blocks: [n_cross, ...] the values transposed
};

// One sequence at a time (f32 storage, video blocks).
dit_status full_stack(dit_cache* c, const Seq& q, int t, int T) {
  const int H = c->H, N = c->N, Nt = c->Nt, L = c->L, ldY = c->ldY;
  const float* md = q.mod;
  char* Xi = sp(c, c->X, (size_t)Nt * H);  // image rows of the joint state
  char* Ai = sp(c, c->A, (size_t)Nt * H);
  char* Yi = sp(c, c->Y, (size_t)Nt * ldY);
  const int cls = DIT_K_GEMM;

  if (c->cfg.n_cross) {
    HIPCK(hipMemcpyAsync(c->X, q.h, (size_t)N * H * c->esz, hipMemcpyDeviceToDevice, c->stream));
    for (int i = 0; i < c->cfg.n_cross; ++i) {
      const CrossW& w = c->M.crs[i];
      const float* e = q.modx + ((size_t)i * T + t) * 6 * H;
      // block 0's modulated input is this step's indicator tensor m_t
      const bool use_m0 = i == 0 && q.m0;
      if (!use_m0) TRY(ln_mod(c, c->X, H, c->A, H, N, N, e, e + H, e, e + H, DIT_K_FULL_OTHER));
      GemmArgs g = lin_args(c, use_m0 ? q.m0 : c->A, H, w.qkv, c->Y, ldY, N);
      g.rms_cols = 2 * H;
      // the projection writes the values transposed for attention when it can
      bool vt_fused = false;
      if (c->bf16) {
        g.vt = c->vt;
        g.vt_col0 = 2 * H;
        g.vt_heads = c->cfg.heads;
        g.vt_ld = (int)rup(N, 64);
        g.vt_rows0 = N;
        g.vt_key0 = 0;
        vt_fused = dit::gemm_bf16_fuses_vt(&g, 1, c->n_cu);
        if (!vt_fused) g.vt = nullptr;
      }
      TRY(gemm(c, &g, 1, cls));
      TRY(attention(c, c->Y, ldY, sp(c, c->Y, H), ldY, sp(c, c->Y, 2 * H), ldY, sp(c, c->Y, 3 * H), ldY, N,
                    N, c->vt, 0x7fffffff, 0, 1, 0, 0, vt_fused));
      g = lin_args(c, sp(c, c->Y, 3 * H), ldY, w.o, c->X, H, N, DIT_EPI_GATED_RES);
      g.gate = e + 2 * H;
      TRY(gemm(c, &g, 1, cls));
      // cross-attention: q from LN(x), k/v from the text tokens
      TRY(ln_mod(c, c->X, H, c->A, H, N, N, nullptr, nullptr, nullptr, nullptr, DIT_K_FULL_OTHER));
      GemmArgs gq = lin_args(c, c->A, H, w.xq, c->Y, ldY, N);
      gq.rms_cols = H;
      TRY(gemm(c, &gq, 1, cls));
      // the text tokens' keys and values (and the transposed values) were formed once for the sample
      const char* kv = sp(c, q.xkv, (size_t)i * xkv_elems(c));
      void* vt = c->bf16 ? (void*)((char*)q.xvt + (size_t)i * xvt_elems(c) * 2) : nullptr;
      TRY(attention(c, c->Y, ldY, kv, 2 * H, kv + (size_t)H * c->esz, 2 * H, sp(c, c->Y, 3 * H), ldY, N, Nt, vt,
                    0x7fffffff, 0, 1, 0, 0, c->bf16));
      g = lin_args(c, sp(c, c->Y, 3 * H), ldY, w.xo, c->X, H, N, DIT_EPI_GATED_RES);
      g.gate = c->ones;
      TRY(gemm(c, &g, 1, cls));
      TRY(ln_mod(c, c->X, H, c->A, H, N, N, e + 3 * H, e + 4 * H, e + 3 * H, e + 4 * H, DIT_K_FULL_OTHER));
      g = lin_args(c, c->A, H, w.ffn0, sp(c, c->Y, 4 * H), ldY, N);
      g.gelu_from = 0;
      TRY(gemm(c, &g, 1, cls));
      g = lin_args(c, sp(c, c->Y, 4 * H), ldY, w.ffn1, c->X, H, N, DIT_EPI_GATED_RES);
      g.gate = e + 5 * H;
      TRY(gemm(c, &g, 1, cls));
    }
    {
      Scope sc(c, DIT_K_FULL_OTHER, 3.0 * N * H * c->esz);
      TRY(typed(c, [&](auto* tp) {
        using T_ = std::remove_pointer_t<decltype(tp)>;
        return dit::launch_add<T_>((const T_*)c->X, (const T_*)q.h, (T_*)q.r, (int64_t)N * H, -1.f, c->stream);
      }));
    }
    return DIT_OK;
  }

  // MMDiT: X = [txt; img]
  HIPCK(hipMemcpyAsync(c->X, q.txt, (size_t)Nt * H * c->esz, hipMemcpyDeviceToDevice, c->stream));
  HIPCK(hipMemcpyAsync(Xi, q.h, (size_t)N * H * c->esz, hipMemcpyDeviceToDevice, c->stream));
  for (int i = 0; i < c->cfg.n_double; ++i) {
    const DoubleW& w = c->M.dbl[i];
    const float* mi = md + (size_t)12 * H * i;  // image stream chunk
    const float* mt = mi + 6 * H;               // text stream chunk
    // block 0's image-stream input is this step's indicator tensor m_t
    const bool use_m0 = i == 0 && q.m0;
    TRY(ln_mod(c, c->X, H, c->A, H, use_m0 ? Nt : L, Nt, mt, mt + H, mi, mi + H, DIT_K_FULL_OTHER));
    GemmArgs g[2];
    g[0] = lin_args(c, use_m0 ? q.m0 : (const void*)Ai, H, w.qkv[0], Yi, ldY, N);
    g[1] = lin_args(c, c->A, H, w.qkv[1], c->Y, ldY, Nt);
    g[0].rms_cols = g[1].rms_cols = 2 * H;
    TRY(gemm(c, g, 2, cls));
    TRY(attention(c, c->Y, ldY, sp(c, c->Y, H), ldY, sp(c, c->Y, 2 * H), ldY, sp(c, c->Y, 3 * H), ldY, L, L,
                  c->vt));
    g[0] = lin_args(c, Yi + 3 * H * c->esz, ldY, w.o[0], Xi, H, N, DIT_EPI_GATED_RES);
    g[1] = lin_args(c, sp(c, c->Y, 3 * H), ldY, w.o[1], c->X, H, Nt, DIT_EPI_GATED_RES);
    g[0].gate = mi + 2 * H;
    g[1].gate = mt + 2 * H;
    TRY(gemm(c, g, 2, cls));
    TRY(ln_mod(c, c->X, H, c->A, H, L, Nt, mt + 3 * H, mt + 4 * H, mi + 3 * H, mi + 4 * H, DIT_K_FULL_OTHER));
    g[0] = lin_args(c, Ai, H, w.mlp0[0], Yi + 4 * H * c->esz, ldY, N);
    g[1] = lin_args(c, c->A, H, w.mlp0[1], sp(c, c->Y, 4 * H), ldY, Nt);
    g[0].gelu_from = g[1].gelu_from = 0;
    TRY(gemm(c, g, 2, cls));
    g[0] = lin_args(c, Yi + 4 * H * c->esz, ldY, w.mlp1[0], Xi, H, N, DIT_EPI_GATED_RES);
    g[1] = lin_args(c, sp(c, c->Y, 4 * H), ldY, w.mlp1[1], c->X, H, Nt, DIT_EPI_GATED_RES);
    g[0].gate = mi + 5 * H;
    g[1].gate = mt + 5 * H;
    TRY(gemm(c, g, 2, cls));
  }
  for (int i = 0; i < c->cfg.n_single; ++i) {
    const SingleW& w = c->M.sgl[i];
    const float* ms = md + (size_t)12 * H * c->cfg.n_double + (size_t)3 * H * i;
    TRY(ln_mod(c, c->X, H, c->A, H, L, L, ms, ms + H, ms, ms + H, DIT_K_FULL_OTHER));
    GemmArgs g = lin_args(c, c->A, H, w.l1, c->Y, ldY, L);
    g.rms_cols = 2 * H;
    g.gelu_from = 3 * H;
    g.gap_at = 3 * H;
    g.gap = H;
    TRY(gemm(c, &g, 1, cls));
    TRY(attention(c, c->Y, ldY, sp(c, c->Y, H), ldY, sp(c, c->Y, 2 * H), ldY, sp(c, c->Y, 3 * H), ldY, L, L,
                  c->vt));
    g = lin_args(c, sp(c, c->Y, 3 * H), ldY, w.l2, c->X, H, L, DIT_EPI_GATED_RES);
    g.gate = ms + 2 * H;
    TRY(gemm(c, &g, 1, cls));
  }
  {
    Scope sc(c, DIT_K_FULL_OTHER, 3.0 * N * H * c->esz);
    TRY(typed(c, [&](auto* tp) {
      using T_ = std::remove_pointer_t<decltype(tp)>;
      return dit::launch_add<T_>((const T_*)Xi, (const T_*)q.h, (T_*)q.r, (int64_t)N * H, -1.f, c->stream);
    }));
  }
  return DIT_OK;
}

// Modulation vectors of the Q stacked sequences: sequence q's at base + q d
// (d = 0: one vector shared by all).
struct ModRef {
  const float* base;
  int64_t d;
};

// Q sequences through the MMDiT stack at once (bf16).  Rows are
// stream-major, [txt_0; ...; txt_{Q-1}; img_0; ...; img_{Q-1}], so each
// linear layer is one launch over every sequence's rows of a stream (Q
// times the rows per weight read); attention is one launch over the Q
// sequences, each read as its two row pieces.  Modulation vectors are per
// sequence (pooled text) or shared.
dit_status full_stack_multi(dit_cache* c, const Seq* seqs, int Q) {
  const int H = c->H, N = c->N, Nt = c->Nt, L = c->L, ldY = c->ldY;
  const int Lt = Q * Nt, Li = Q * N, LL = Q * L;
  const size_t es = c->esz;
  char* Xi = sp(c, c->X, (size_t)Lt * H);
  char* Ai = sp(c, c->A, (size_t)Lt * H);
  char* Yi = sp(c, c->Y, (size_t)Lt * ldY);
  const int cls = DIT_K_GEMM;
  for (int q = 0; q < Q; ++q) {
    HIPCK(hipMemcpyAsync(sp(c, c->X, (size_t)q * Nt * H), seqs[q].txt, (size_t)Nt * H * es,
                         hipMemcpyDeviceToDevice, c->stream));
    HIPCK(hipMemcpyAsync(sp(c, Xi, (size_t)q * N * H), seqs[q].h, (size_t)N * H * es, hipMemcpyDeviceToDevice,
                         c->stream));
  }
  // the sequences' modulation vectors as base + q d: shared, evenly spaced,
  // or gathered into modq
  ModRef mr{seqs[0].mod, 0};
  if (Q > 1) {
    mr.d = seqs[1].mod - seqs[0].mod;
    bool even = true;
    for (int q = 2; q < Q; ++q) even &= seqs[q].mod - seqs[0].mod == q * mr.d;
    if (!even) {
      for (int q = 0; q < Q; ++q)
        HIPCK(hipMemcpyAsync(c->modq + (size_t)q * c->n_mod, seqs[q].mod, (size_t)c->n_mod * 4,
                             hipMemcpyDeviceToDevice, c->stream));
      mr = ModRef{c->modq, c->n_mod};
    }
  }
  // per-segment gate vectors in the GEMM need 32 | segment rows; otherwise
  // the gated layers run per sequence
  const bool seg_gemm = mr.d == 0 || (N % 32 == 0 && Nt % 32 == 0);
  // gated residual over the image rows (gi, column offset oi of the
  // modulation vector) and the text rows (gt, offset ot) of every sequence
  auto gated = [&](GemmArgs gi, GemmArgs gt, size_t oi, size_t ot) -> dit_status {
    gi.gate = mr.base + oi;
    gt.gate = mr.base + ot;
    if (mr.d == 0 || seg_gemm) {
      if (mr.d) {
        gi.gseg = N; gt.gseg = Nt;
        gi.gstride = gt.gstride = mr.d;
      }
      GemmArgs g[2] = {gi, gt};
      return gemm(c, g, 2, cls);
    }
    for (int q = 0; q < Q; ++q) {
      GemmArgs g[2] = {gi, gt};
      g[0].A = sp(c, gi.A, (size_t)q * N * gi.lda);
      g[0].C = sp(c, gi.C, (size_t)q * N * gi.ldc);
      g[0].M = N;
      g[0].gate = mr.base + q * mr.d + oi;
      g[1].A = sp(c, gt.A, (size_t)q * Nt * gt.lda);
      g[1].C = sp(c, gt.C, (size_t)q * Nt * gt.ldc);
      g[1].M = Nt;
      g[1].gate = mr.base + q * mr.d + ot;
      TRY(gemm(c, g, 2, cls));
    }
    return DIT_OK;
  };
  // adaLN over all rows: text rows take offset ot, image rows oi
  auto lnm = [&](size_t ot, size_t oi) {
    const float* b = mr.base;
    return ln_mod(c, c->X, H, c->A, H, LL, Lt, b + ot, b + ot + H, b + oi, b + oi + H, DIT_K_FULL_OTHER, Nt, N,
                  mr.d);
  };
  auto attn = [&](bool vt_ready) {
    return attention(c, c->Y, ldY, sp(c, c->Y, H), ldY, sp(c, c->Y, 2 * H), ldY, sp(c, c->Y, 3 * H), ldY, L, L,
                     c->vt, Nt, (int64_t)(Q - 1) * Nt, Q, Nt, (int64_t)N - Nt, vt_ready);
  };
  // The QKV projection writes the values transposed for attention itself
  // (layout [sequence][head][128][rup(L, 64)], the keys of a sequence being
  // its text rows then its image rows) when the GEMM admits it; otherwise
  // they are stored in Y and transposed by a separate pass.
  const int ldvt = (int)rup(L, 64);
  auto with_vt = [&](GemmArgs& g, int rows0, int key0, int split = 0x7fffffff, int rows1 = 1, int key1 = 0) {
    g.vt = c->vt;
    g.vt_col0 = 2 * H;
    g.vt_heads = c->cfg.heads;
    g.vt_ld = ldvt;
    g.vt_split = split;
    g.vt_rows0 = rows0; g.vt_key0 = key0;
    g.vt_rows1 = rows1; g.vt_key1 = key1;
  };
  // one sequence: block 0's image-stream input is this step's indicator tensor m_t
  const void* m0 = Q == 1 ? seqs[0].m0 : nullptr;
  for (int i = 0; i < c->cfg.n_double; ++i) {
    const DoubleW& w = c->M.dbl[i];
    const size_t mi = (size_t)12 * H * i, mt = mi + 6 * H;  // image / text stream chunks
    const bool use_m0 = i == 0 && m0;
    if (use_m0) TRY(ln_mod(c, c->X, H, c->A, H, Lt, Lt, mr.base + mt, mr.base + mt + H, mr.base + mt,
                           mr.base + mt + H, DIT_K_FULL_OTHER));
    else TRY(lnm(mt, mi));
    GemmArgs g[2];
    g[0] = lin_args(c, use_m0 ? m0 : (const void*)Ai, H, w.qkv[0], Yi, ldY, Li);
    g[1] = lin_args(c, c->A, H, w.qkv[1], c->Y, ldY, Lt);
    g[0].rms_cols = g[1].rms_cols = 2 * H;
    with_vt(g[0], N, Nt);   // image rows: keys Nt .. Nt + N - 1 of sequence m / N
    with_vt(g[1], Nt, 0);   // text rows: keys 0 .. Nt - 1 of sequence m / Nt
    const bool vt_fused = dit::gemm_bf16_fuses_vt(g, 2, c->n_cu);
    if (!vt_fused) g[0].vt = g[1].vt = nullptr;
    TRY(gemm(c, g, 2, cls));
    TRY(attn(vt_fused));
    TRY(gated(lin_args(c, Yi + 3 * H * es, ldY, w.o[0], Xi, H, Li, DIT_EPI_GATED_RES),
              lin_args(c, sp(c, c->Y, 3 * H), ldY, w.o[1], c->X, H, Lt, DIT_EPI_GATED_RES), mi + 2 * H,
              mt + 2 * H));
    TRY(lnm(mt + 3 * H, mi + 3 * H));
    g[0] = lin_args(c, Ai, H, w.mlp0[0], Yi + 4 * H * es, ldY, Li);
    g[1] = lin_args(c, c->A, H, w.mlp0[1], sp(c, c->Y, 4 * H), ldY, Lt);
    g[0].gelu_from = g[1].gelu_from = 0;
    TRY(gemm(c, g, 2, cls));
    TRY(gated(lin_args(c, Yi + 4 * H * es, ldY, w.mlp1[0], Xi, H, Li, DIT_EPI_GATED_RES),
              lin_args(c, sp(c, c->Y, 4 * H), ldY, w.mlp1[1], c->X, H, Lt, DIT_EPI_GATED_RES), mi + 5 * H,
              mt + 5 * H));
  }
  for (int i = 0; i < c->cfg.n_single; ++i) {
    const SingleW& w = c->M.sgl[i];
    const size_t ms = (size_t)12 * H * c->cfg.n_double + (size_t)3 * H * i;
    TRY(lnm(ms, ms));
    GemmArgs g = lin_args(c, c->A, H, w.l1, c->Y, ldY, LL);
    g.rms_cols = 2 * H;
    g.gelu_from = 3 * H;
    g.gap_at = 3 * H;
    g.gap = H;
    with_vt(g, Nt, 0, Lt, N, Nt);  // the Q text row blocks, then the Q image row blocks
    const bool vt_fused = dit::gemm_bf16_fuses_vt(&g, 1, c->n_cu);
    if (!vt_fused) g.vt = nullptr;
    TRY(gemm(c, &g, 1, cls));
    TRY(attn(vt_fused));
    if (mr.d == 0) {
      g = lin_args(c, sp(c, c->Y, 3 * H), ldY, w.l2, c->X, H, LL, DIT_EPI_GATED_RES);
      g.gate = mr.base + ms + 2 * H;
      TRY(gemm(c, &g, 1, cls));
    } else {
      TRY(gated(lin_args(c, Yi + 3 * H * es, ldY, w.l2, Xi, H, Li, DIT_EPI_GATED_RES),
                lin_args(c, sp(c, c->Y, 3 * H), ldY, w.l2, c->X, H, Lt, DIT_EPI_GATED_RES), ms + 2 * H,
                ms + 2 * H));
    }
  }
  for (int q = 0; q < Q; ++q) {
    Scope sc(c, DIT_K_FULL_OTHER, 3.0 * N * H * es);
    HIPCK(dit::launch_add<bf16_t>((const bf16_t*)sp(c, Xi, (size_t)q * N * H), (const bf16_t*)seqs[q].h,
                                  (bf16_t*)seqs[q].r, (int64_t)N * H, -1.f, c->stream));
  }
  return DIT_OK;
}

// v_b = Final(h_out) from the already modulated final-layer input c->yf.
// Single-branch bf16 sampling folds the Euler update into the projection
// (x += dsigma v); returns whether it did.
bool proj_fits(const dit_cache* c) {
  return c->bf16 && c->C % 16 == 0 && c->C <= 128 && c->H % 32 == 0;
}

dit_status final_project(dit_cache* c, int b, int cls, float* latent = nullptr, float dsig = 0.f) {
  const int H = c->H, N = c->N;
  Scope sc(c, cls, 0);
  if (proj_fits(c)) {
    HIPCK(dit::launch_proj_small_n(c->yf, H, c->M.fin.w, H, c->M.fin.b, c->vel + (size_t)b * N * c->C, c->C,
                                   latent, c->C, dsig, N, c->C, H, c->stream));
    return DIT_OK;
  }
  GemmArgs g = lin_args(c, c->yf, H, c->M.fin, c->vel + (size_t)b * N * c->C, c->C, N, DIT_EPI_F32);
  if (c->bf16) {
    HIPCK(dit::launch_gemm_bf16(&g, 1, c->stream, c->n_cu));
  } else {
    HIPCK(dit::launch_gemm_f32(&g, 1, c->stream));
  }
  return DIT_OK;
}

// full step: y = S(LN(h_out)(1+scale_f)+shift_f), then the projection
dit_status final_layer(dit_cache* c, int b, const void* hout, const float* mod, int cls, float* latent = nullptr,
                       float dsig = 0.f) {
  const int H = c->H, N = c->N;
  const float* mf = mod + (c->n_mod - 2 * H);
  TRY(ln_mod(c, hout, H, c->yf, H, N, N, mf, mf + H, mf, mf + H, cls));
  return final_project(c, b, cls, latent, dsig);
}

// Modulation table slot of branch b of sample j.
int mod_slot(const dit_cache* c, int j, int b) { return c->cfg.pooled_text ? j * c->nb + b : 0; }

// once per call: text tokens of every sample, vec and the modulation table
// of every step (one per branch and sample with pooled text, else one)
dit_status prepare(dit_cache* c, int S, const void* text_emb, const std::vector<double>& sig, int T) {
  const int H = c->H, Nt = c->Nt, X = c->cfg.ctx_dim;
  const int cls = DIT_K_ONCE;
  HIPCK(hipMemcpyAsync(c->sig_dev, sig.data(), (T + 1) * sizeof(double), hipMemcpyHostToDevice, c->stream));
  {
    Scope s(c, cls, 0);
    TRY(typed(c, [&](auto* tp) {
      using Ty = std::remove_pointer_t<decltype(tp)>;
      return dit::launch_time_embed<Ty>(c->sig_dev, (Ty*)c->temb, T, c->cfg.time_dim, c->stream);
    }));
  }
  GemmArgs g = lin_args(c, c->temb, c->cfg.time_dim, c->M.time0, c->th, H, T, DIT_EPI_SILU);
  TRY(gemm(c, &g, 1, cls));
  g = lin_args(c, c->th, H, c->M.time2, c->tv, H, T, DIT_EPI_F32);
  TRY(gemm(c, &g, 1, cls));
  for (int j = 0; j < S; ++j)
    for (int b = 0; b < c->nb; ++b) {
      const void* te = (const char*)text_emb + ((size_t)j * c->nb + b) * Nt * X * c->esz;
      g = lin_args(c, te, X, c->M.txt_in, sp(c, c->lanes[j].txt, (size_t)b * Nt * H), H, Nt);
      TRY(gemm(c, &g, 1, cls));
      for (int i = 0; i < c->cfg.n_cross; ++i) {  // every video block's text keys | values (rms-normed k)
        const Lane& l = c->lanes[j];
        const size_t bi = (size_t)b * c->cfg.n_cross + i;
        char* kv = sp(c, l.xkv, bi * xkv_elems(c));
        GemmArgs gkv = lin_args(c, sp(c, l.txt, (size_t)b * Nt * H), H, c->M.crs[i].xkv, kv, 2 * H, Nt);
        gkv.rms_cols = H;
        TRY(gemm(c, &gkv, 1, cls));
        if (c->bf16) {
          Scope s(c, cls, 0);
          HIPCK(dit::launch_transpose_v_bf16(kv + (size_t)H * 2, 2 * H, (char*)l.xvt + bi * xvt_elems(c) * 2, Nt,
                                             c->cfg.heads, c->stream));
        }
      }
      if ((j > 0 || b > 0) && !c->cfg.pooled_text) continue;  // identical vec and mod table
      const int slot = mod_slot(c, j, b);
      const float* pvp = nullptr;
      if (c->cfg.pooled_text) {
        {
          Scope s(c, cls, 0);
          TRY(typed(c, [&](auto* tp) {
            using Ty = std::remove_pointer_t<decltype(tp)>;
            return dit::launch_mean_rows<Ty>((const Ty*)te, Nt, X, (Ty*)c->pooled, c->stream);
          }));
        }
        g = lin_args(c, c->pooled, X, c->M.pool0, c->ph, H, 1, DIT_EPI_SILU);
        TRY(gemm(c, &g, 1, cls));
        g = lin_args(c, c->ph, H, c->M.pool2, c->pv, H, 1, DIT_EPI_F32);
        TRY(gemm(c, &g, 1, cls));
        pvp = c->pv;
      }
      {
        Scope s(c, cls, 0);
        TRY(typed(c, [&](auto* tp) {
          using Ty = std::remove_pointer_t<decltype(tp)>;
          return dit::launch_vec_silu<Ty>(c->tv, pvp, (Ty*)c->svec, T, H, c->stream);
        }));
      }
      float* mod = c->mod + (size_t)slot * T * c->n_mod;
      g = lin_args(c, c->svec, H, c->M.mod, mod, c->n_mod, T, DIT_EPI_F32);
      TRY(gemm(c, &g, 1, cls));
      if (c->fconst) {  // the reuse candidate's final-layer constants of every step
        Scope s(c, cls, 0);
        HIPCK(dit::launch_final_consts(mod, c->n_mod, c->n_mod - 2 * H, T, c->M.fin.w, c->M.fin.b, H,
                                       c->fconst + (size_t)slot * T * 128, c->stream));
      }
      if (c->cfg.n_cross) {
        const int base = 12 * H * c->cfg.n_double + 3 * H * c->cfg.n_single;
        for (int i = 0; i < c->cfg.n_cross; ++i) {
          Scope s(c, cls, 0);
          float* dst = c->modx + ((size_t)slot * c->cfg.n_cross + i) * T * 6 * H;
          TRY(typed(c, [&](auto* tp) {
            using Ty = std::remove_pointer_t<decltype(tp)>;
            return dit::launch_add_offset<Ty>(mod, c->n_mod, base, (const Ty*)c->M.crs[i].mod_off, dst, T, 6 * H,
                                              c->stream);
          }));
        }
      }
    }
  return DIT_OK;
}

// ---------------------------------------------------------------- UniPC
// lambda = log(alpha / sigma) with alpha = 1 - sigma; +-inf at sigma = 0 / 1.
double unipc_lambda(double sg) {
  if (sg >= 1.0) return -INFINITY;
  if (sg <= 0.0) return INFINITY;
  return std::log(1.0 - sg) - std::log(sg);
}

// Step sigma_s -> sigma_t: B = e^{-h} - 1 and b_1 = phi_1 / B, b_2 = 2 phi_2 / B
// (phi_1 = B / (-h) - 1, phi_2 = phi_1 / (-h) - 1/2); h = +inf gives B = -1,
// b_1 = b_2 = 1, the exact limits.
struct UniStep { double h, B, b1, b2; };
UniStep unipc_step(double ss, double st) {
  const double h = unipc_lambda(st) - unipc_lambda(ss);
  if (std::isinf(h)) return {INFINITY, -1.0, 1.0, 1.0};
  const double hh = -h, B = std::expm1(hh);
  const double phi1 = B / hh - 1.0, phi2 = phi1 / hh - 0.5;
  return {h, B, phi1 / B, 2.0 * phi2 / B};
}

// r = (lambda_p - lambda_s) / h, -inf (its term vanishes) through sigma = 1.
double unipc_ratio(double sp, double ss, double h) {
  const double lp = unipc_lambda(sp);
  if (std::isinf(lp) || std::isinf(h)) return -INFINITY;
  return (lp - unipc_lambda(ss)) / h;
}

// Coefficients of step t: corrector of x_t (t >= 1, order of step t-1's
// predictor) and predictor of x_{t+1} (order min(2, t + 1, T - t)).
dit::UniCoef unipc_coef(const std::vector<double>& sig, int t, int T) {
  auto ord = [&](int i) { return std::min(2, std::min(i + 1, T - i)); };
  dit::UniCoef k{};
  if (t > 0) {
    const double ss = sig[t - 1], st = sig[t], sp = t > 1 ? sig[t - 2] : 1.0;
    const UniStep u = unipc_step(ss, st);
    const double a = 1.0 - st;
    double cx = st / ss, cs = -a * u.B, cp = 0.0, ct;
    if (ord(t - 1) == 1) {
      ct = -a * u.B * 0.5;
    } else {
      const double r = unipc_ratio(sp, ss, u.h);
      if (std::isinf(r)) {
        ct = -a * u.B * u.b1;
      } else {
        const double rho1 = (u.b1 - u.b2) / (1.0 - r), rhot = u.b1 - rho1;
        cp = -a * u.B * rho1 / r;
        cs -= cp;
        ct = -a * u.B * rhot;
      }
    }
    cs -= ct;  // the corrector's terms are differences against m_{t-1}
    k.corr = 1;
    k.cx = (float)cx; k.cs = (float)cs; k.cp = (float)cp; k.ct = (float)ct;
  }
  const double ss = sig[t], st = sig[t + 1];
  const UniStep u = unipc_step(ss, st);
  const double a = 1.0 - st;
  double pt = -a * u.B, pp = 0.0;
  if (ord(t) == 2) {
    const double r = unipc_ratio(sig[t - 1], ss, u.h);
    if (!std::isinf(r)) {
      pp = -a * u.B * 0.5 / r;
      pt -= pp;
    }
  }
  k.px = (float)(st / ss); k.pt = (float)pt; k.pp = (float)pp;
  return k;
}

// S samples in lockstep: each step runs (a1, a2) for every sample, one host
// wait for all their sums, each sample's own decision (a3), then the reuse
// samples (a4, a5) one by one and the computing ones' block stacks together.
dit_status run_batch(dit_cache* c, int S, float* latents, const void* text_emb, const GateMLP& gate,
                     const dit_sample_params& p, dit_schedule* out) {
  const int T = p.T, B = p.B;
  const int H = c->H, N = c->N, C = c->C, nb = c->nb;
  const size_t NC = (size_t)N * C, NH = (size_t)N * H;
  std::vector<double> sig(T + 1);
  if (p.sigmas) {
    for (int i = 0; i <= T; ++i) sig[i] = p.sigmas[i];
  } else {
    for (int i = 0; i <= T; ++i) {
      const double u = 1.0 - (double)i / T;
      sig[i] = p.shift * u / (1.0 + (p.shift - 1.0) * u);
    }
  }
  TRY(ensure_lanes(c, S));
  TRY(ensure_T(c, T, S));
  TRY(prepare(c, S, text_emb, sig, T));

  const bool pair = nb == 2;
  const bool unipc = p.solver == DIT_SOLVER_UNIPC;
  // sstream / step: the indicator and the reuse candidate of a sample and
  // step come from one pass over its rows, before the decision (bf16, C = 64;
  // sstream: the column-sliced kernels, step: the row-tiled fused kernel for
  // widths they do not take); fused: the older pair of fused kernels
  const bool sstream = c->cand != nullptr;
  const bool step = !sstream && c->bf16 && dit::step_fused_fits(C, H, nb);
  const bool spec_path = sstream || step;
  const bool fused = !spec_path && c->bf16 && dit::reuse_fused_fits(C, H);
  const bool fused_euler = !pair && proj_fits(c) && !unipc;  // Euler folded into the projection
  const double thr = std::log(p.tau / (1.0 - p.tau));
  // mu(B, T) of the static policy: computed steps at floor(i T / B)
  std::vector<uint8_t> mu(T, 0);
  for (int i = 0; i < B; ++i) mu[(size_t)((int64_t)i * T / B)] = 1;
  for (int j = 0; j < S; ++j) {
    Lane& l = c->lanes[j];
    l.cnt = 0; l.t_last = 0; l.acc = 0.0; l.i_prev = -1; l.i_last = -1; l.dec = true;
    out[j].nfe = 0;
    out[j].steps_done = 0;
  }
  auto modp = [&](int j, int b, int t) { return c->mod + ((size_t)mod_slot(c, j, b) * T + t) * c->n_mod; };
  auto modxp = [&](int j, int b) {
    return c->modx ? c->modx + (size_t)mod_slot(c, j, b) * c->cfg.n_cross * T * 6 * H : nullptr;
  };
  // Each lane's current latent: the caller's buffer or the lane's second
  // buffer, which trade places when a reused step takes the candidate's
  // Euler result; the caller's buffer receives x_T at the end.
  std::vector<float*> cur(S), alt(S);
  for (int j = 0; j < S; ++j) {
    cur[j] = latents + j * NC;
    alt[j] = c->lanes[j].xalt;
  }
  auto lat = [&](int j) { return cur[j]; };
  auto fail_all = [&](int t, dit_status st, const std::string& m) {
    for (int j = 0; j < S; ++j) out[j].steps_done = t;
    return fail(c, st, m);
  };
  std::vector<Seq> seqs;
  std::vector<int> comp;

  for (int t = 0; t < T; ++t) {
    const float dsig = (float)(sig[t + 1] - sig[t]);
    // (a1) patch embed and modulated indicator tensor, (a2) its sums
    for (int j = 0; j < S; ++j) {
      Lane& l = c->lanes[j];
      l.i_new = 0;
      while (l.i_new == l.i_prev || l.i_new == l.i_last) ++l.i_new;
      const float *sh0 = nullptr, *sc0 = nullptr;
      if (p.indicator == DIT_INDICATOR_MODULATED) {
        sh0 = c->cfg.n_cross ? modxp(j, 0) + (size_t)t * 6 * H  // block 0
                             : modp(j, 0, t);                  // first block's image-stream (or single) shift
        sc0 = sh0 + H;
      }
      double* sums = c->sums_dev + 4 * j;
      const void* mp = t ? l.mbuf[l.i_prev] : nullptr;
      const void* ml = t ? l.mbuf[l.i_last] : nullptr;
      if (spec_path) {
        // a step known to compute (t = 0, replay mask, spend-the-remainder,
        // static mask) writes h for the block stack instead of a reuse candidate
        bool known_full = t == 0;
        if (p.forced_mask) known_full = known_full || p.forced_mask[(size_t)j * T + t];
        else if (p.policy == DIT_POLICY_GATE) known_full = known_full || B - l.cnt >= T - t;
        else if (p.policy == DIT_POLICY_STATIC) known_full = known_full || mu[t];
        l.spec = !known_full;
        const int reads = t == 0 ? 0 : (l.i_prev == l.i_last ? 1 : 2);
        // algorithmic bytes: m_t written, m_{t-1} / m_last read, and either r read per branch
        // (reuse candidate) or h written (the block stack's input)
        Scope sc(c, DIT_K_INDICATOR, (double)NH * c->esz * (1 + reads + (l.spec ? nb : 1)));
        const float* mf0 = modp(j, 0, t) + (c->n_mod - 2 * H);
        const float* mf1 = pair ? modp(j, 1, t) + (c->n_mod - 2 * H) : nullptr;
        if (sstream) {
          dit::StepStreamDesc d;
          d.x = lat(j); d.rows = N; d.H = H;
          d.W_in = c->M.img_in.w; d.b_in = c->M.img_in.b;
          d.st_hi = c->st_hi; d.st_lo = c->st_lo; d.bbar = c->st_bbar; d.b2 = c->st_b2;
          d.m_out = l.mbuf[l.i_new]; d.m_prev = mp; d.m_last = ml;
          d.sh0 = sh0; d.sc0 = sc0;
          // every step records sum |m_t|; later steps read the older buffers' sums from it
          d.partials = c->partials; d.out = sums;
          d.mag = l.mag; d.i_new = l.i_new; d.i_prev = l.i_prev; d.i_last = l.i_last;
          if (l.spec) {
            d.r = l.r; d.nb = nb;
            d.W_out = c->M.fin.w; d.mf0 = mf0; d.mf1 = mf1;
            d.fc0 = c->fconst + ((size_t)mod_slot(c, j, 0) * T + t) * 128;
            d.fc1 = pair ? c->fconst + ((size_t)mod_slot(c, j, 1) * T + t) * 128 : nullptr;
            d.cand = c->cand; d.dsig = dsig; d.guidance = (float)p.guidance;
            d.x_spec = unipc ? nullptr : alt[j]; d.v_spec = unipc ? l.vspec : nullptr;
          } else {
            d.h_out = l.h;
          }
          HIPCK(dit::launch_step_stream(d, c->stream));
        } else {
          HIPCK(dit::launch_step_fused(lat(j), C, c->M.img_in.w, c->M.img_in.b, l.mbuf[l.i_new], mp, ml, N, H, sh0,
                                       sc0, t ? c->partials : nullptr, sums, l.spec ? l.r : nullptr, nb, c->M.fin.w,
                                       c->M.fin.b, mf0, mf1, dsig, (float)p.guidance, unipc ? nullptr : alt[j],
                                       unipc ? l.vspec : nullptr, l.spec ? nullptr : l.h, c->stream));
        }
      } else if (fused) {
        // embedding recomputed in LDS: reads m_{t-1} and m_{t_last} (once if equal), writes m_t
        Scope sc(c, DIT_K_INDICATOR, (double)NH * c->esz * (t == 0 ? 1 : (l.i_prev == l.i_last ? 2 : 3)));
        HIPCK(dit::launch_reuse_indicator(lat(j), C, c->M.img_in.w, c->M.img_in.b, l.mbuf[l.i_new], mp, ml, N, H,
                                          sh0, sc0, t ? c->partials : nullptr, sums, nullptr, c->stream));
      } else {
        Scope sc(c, DIT_K_INDICATOR, (double)NH * c->esz * (t == 0 ? 2 : (l.i_prev == l.i_last ? 3 : 4)));
        TRY(typed(c, [&](auto* tp) {
          using Ty = std::remove_pointer_t<decltype(tp)>;
          return dit::launch_cast_from_f32<Ty>(lat(j), (Ty*)c->xs, (int64_t)NC, c->stream);
        }));
        GemmArgs g = lin_args(c, c->xs, C, c->M.img_in, l.h, H, N);
        if (c->bf16) { HIPCK(dit::launch_gemm_bf16(&g, 1, c->stream, c->n_cu)); }
        else { HIPCK(dit::launch_gemm_f32(&g, 1, c->stream)); }
        TRY(typed(c, [&](auto* tp) {
          using Ty = std::remove_pointer_t<decltype(tp)>;
          return dit::launch_indicator<Ty>((const Ty*)l.h, (Ty*)l.mbuf[l.i_new], (const Ty*)mp, (const Ty*)ml, N,
                                           H, sh0, sc0, t ? c->partials : nullptr, sums, c->stream);
        }));
      }
    }

    // (a3) gate + pacing on the host, per sample, after one wait for all sums
    if (t > 0) {
      HIPCK(hipEventRecord(c->ev_sums, c->stream));
      HIPCK(hipEventSynchronize(c->ev_sums));
      break_chain(c);
    }
    const auto h0 = std::chrono::steady_clock::now();
    comp.clear();
    for (int j = 0; j < S; ++j) {
      Lane& l = c->lanes[j];
      int dec = 1, forced = 1;
      double z = NAN;
      double f[DIT_N_FEATURES];
      for (double& v : f) v = NAN;
      double sums[4] = {NAN, NAN, NAN, NAN};
      if (t > 0) {
        for (int k = 0; k < 4; ++k) sums[k] = ((volatile double*)c->sums_host)[4 * j + k];
        for (double v : sums)
          if (!std::isfinite(v))
            return fail_all(t, DIT_ENONFINITE, "indicator sum is not finite at step " + std::to_string(t) +
                                                   " of sample " + std::to_string(j));
        const double d_prev = sums[0] / std::max(sums[1], 1e-30);
        const double d_last = sums[2] / std::max(sums[3], 1e-30);
        l.acc += d_prev;
        f[0] = (double)B / T;
        f[1] = (double)(B - l.cnt) / B;
        f[2] = (double)(B - l.cnt) / (T - t);
        f[3] = (double)(t - l.t_last);
        f[4] = d_last;
        f[5] = d_prev;
        f[6] = (double)t / T;
        f[7] = l.acc;
        forced = 0;
        if (p.policy == DIT_POLICY_GATE) {
          z = gate_logit(gate, f);
          dec = (z > thr) ? 1 : 0;
          if (B - l.cnt >= T - t) { dec = 1; forced = 1; }
          if (B - l.cnt == 0) { dec = 0; forced = 1; }
        } else if (p.policy == DIT_POLICY_STATIC) {
          dec = mu[t];
        } else {
          z = l.acc;
          dec = (l.acc > p.delta) ? 1 : 0;
        }
        if (p.forced_mask) dec = p.forced_mask[(size_t)j * T + t] ? 1 : 0;
      }
      l.dec = dec != 0;
      if (l.dec) comp.push_back(j);
      dit_schedule& o = out[j];
      o.full[t] = (uint8_t)dec;
      if (o.logit) o.logit[t] = (float)z;
      if (o.forced) o.forced[t] = (uint8_t)forced;
      if (o.features)
        for (int k = 0; k < DIT_N_FEATURES; ++k) o.features[(size_t)t * DIT_N_FEATURES + k] = f[k];
      if (o.sums)
        for (int k = 0; k < 4; ++k) o.sums[(size_t)t * 4 + k] = sums[k];
    }
    if (t > 0)
      c->stats.host_gate_ms +=
          std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - h0).count();

    // the step rule of sample j once its velocity (or velocities) are in vel
    auto step_rule = [&](int j, bool vpair, bool folded, const float* vbuf = nullptr) -> dit_status {
      Lane& l = c->lanes[j];
      if (!unipc && folded) return DIT_OK;
      if (!vbuf) vbuf = c->vel;
      Scope sc(c, l.dec ? DIT_K_FULL_OTHER : DIT_K_REUSE, 0);
      if (unipc) {
        // the guidance pair's two velocities are combined here unless the
        // fused reuse kernel has already combined them
        const dit::UniCoef k = unipc_coef(sig, t, T);
        float* m_t = l.mh[t % 3];
        const float* m_s = t >= 1 ? l.mh[(t + 2) % 3] : nullptr;
        const float* m_p = (t >= 2 && k.cp != 0.f) ? l.mh[(t + 1) % 3] : nullptr;
        HIPCK(dit::launch_unipc(lat(j), vbuf, vpair ? vbuf + NC : nullptr, (float)p.guidance, (float)sig[t],
                                l.x_last, (k.pp != 0.f || k.corr) ? m_s : nullptr, m_p, m_t, k, (int64_t)NC,
                                c->stream));
      } else if (!folded) {
        HIPCK(dit::launch_euler(lat(j), vbuf, pair ? vbuf + NC : nullptr, (float)p.guidance, dsig,
                                (int64_t)NC, c->stream));
      }
      return DIT_OK;
    };

    // (a4) reuse, (a5) final layer + step rule, sample by sample
    for (int j = 0; j < S; ++j) {
      Lane& l = c->lanes[j];
      if (l.dec) continue;
      if (spec_path) {
        // the candidate formed with the indicator is this step's result
        if (!l.spec) return fail_all(t, DIT_EINVAL, "internal: reused step without a reuse candidate");
        if (unipc) {
          TRY(step_rule(j, false, false, l.vspec));
        } else {
          std::swap(cur[j], alt[j]);
        }
        continue;
      }
      if (fused) {
        // h + r, final adaLN, projection, guidance and Euler in one pass per row tile
        Scope sc(c, DIT_K_REUSE, (double)nb * NH * c->esz);
        const float* mf0 = modp(j, 0, t) + (c->n_mod - 2 * H);
        const float* mf1 = pair ? modp(j, 1, t) + (c->n_mod - 2 * H) : nullptr;
        HIPCK(dit::launch_reuse_final(lat(j), C, c->M.img_in.w, c->M.img_in.b, l.r, nb, c->M.fin.w, c->M.fin.b,
                                      mf0, mf1, dsig, (float)p.guidance, N, H, unipc ? c->vel : nullptr,
                                      c->stream));
        if (unipc) TRY(step_rule(j, false, true));
        continue;
      }
      for (int b = 0; b < nb; ++b) {
        {
          // h_out = S(h + r) and the final adaLN in one pass over the rows
          Scope sc(c, DIT_K_REUSE, 3.0 * NH * c->esz);
          const float* mf = modp(j, b, t) + (c->n_mod - 2 * H);
          TRY(typed(c, [&](auto* tp) {
            using Ty = std::remove_pointer_t<decltype(tp)>;
            return dit::launch_add_ln_mod<Ty>((const Ty*)l.h, (const Ty*)sp(c, l.r, b * NH), (Ty*)c->yf, N, H, mf,
                                              mf + H, c->stream);
          }));
        }
        TRY(final_project(c, b, DIT_K_REUSE, fused_euler ? lat(j) : nullptr, dsig));
      }
      TRY(step_rule(j, pair, fused_euler));
    }

    // (a4) full: the computing samples' block stacks, (a5) per sample
    if (!comp.empty()) {
      if (spec_path)  // the block stack's input h, unless the indicator launch already wrote it
        for (int j : comp) {
          Lane& l = c->lanes[j];
          if (!l.spec) continue;
          Scope sc(c, DIT_K_FULL_OTHER, (double)NH * c->esz);
          if (sstream) {
            dit::StepStreamDesc d;
            d.x = lat(j); d.rows = N; d.H = H;
            d.W_in = c->M.img_in.w; d.b_in = c->M.img_in.b;
            d.h_out = l.h;
            HIPCK(dit::launch_step_stream(d, c->stream));
          } else {
            HIPCK(dit::launch_step_fused(lat(j), C, c->M.img_in.w, c->M.img_in.b, nullptr, nullptr, nullptr, N, H,
                                         nullptr, nullptr, nullptr, nullptr, nullptr, nb, c->M.fin.w, c->M.fin.b,
                                         nullptr, nullptr, 0.f, 0.f, nullptr, nullptr, l.h, c->stream));
          }
        }
      if (fused)  // the block stack's input h, bit-identical to the one the indicator used
        for (int j : comp) {
          Scope sc(c, DIT_K_FULL_OTHER, (double)NH * c->esz);
          HIPCK(dit::launch_reuse_indicator(lat(j), C, c->M.img_in.w, c->M.img_in.b, nullptr, nullptr, nullptr, N,
                                            H, nullptr, nullptr, nullptr, nullptr, c->lanes[j].h, c->stream));
        }
      seqs.clear();
      for (int j : comp)
        for (int b = 0; b < nb; ++b) {
          Lane& l = c->lanes[j];
          // the indicator tensor is the first block's modulated image input of branch 0
          const void* m0 = (p.indicator == DIT_INDICATOR_MODULATED && b == 0) ? l.mbuf[l.i_new] : nullptr;
          const size_t nx = (size_t)b * c->cfg.n_cross;
          seqs.push_back(Seq{sp(c, l.txt, (size_t)b * c->Nt * H), l.h, sp(c, l.r, b * NH), modp(j, b, t),
                             modxp(j, b), m0, l.xkv ? sp(c, l.xkv, nx * xkv_elems(c)) : nullptr,
                             l.xvt ? (char*)l.xvt + nx * xvt_elems(c) * 2 : nullptr});
        }
      const int Q = (int)seqs.size();
      if (c->stacked) TRY(full_stack_multi(c, seqs.data(), Q));
      for (size_t k = 0; k < comp.size(); ++k) {
        const int j = comp[k];
        for (int b = 0; b < nb; ++b) {
          const int q = (int)k * nb + b;
          const void* hout;
          if (c->stacked) {
            hout = sp(c, c->X, ((size_t)Q * c->Nt + (size_t)q * N) * H);
          } else {
            TRY(full_stack(c, seqs[q], t, T));
            hout = c->cfg.n_cross ? c->X : sp(c, c->X, (size_t)c->Nt * H);
          }
          TRY(final_layer(c, b, hout, seqs[q].mod, DIT_K_FULL_OTHER, fused_euler ? lat(j) : nullptr, dsig));
        }
        TRY(step_rule(j, pair, fused_euler));
      }
    }

    for (int j = 0; j < S; ++j) {
      Lane& l = c->lanes[j];
      if (l.dec) {
        l.cnt += 1;
        l.t_last = t;
        l.acc = 0.0;
        l.i_last = l.i_new;
        c->stats.full_steps += 1;
      } else {
        c->stats.reuse_steps += 1;
      }
      l.i_prev = l.i_new;
      out[j].nfe = l.cnt;
      out[j].steps_done = t + 1;
    }
  }
  for (int j = 0; j < S; ++j)
    if (cur[j] != latents + j * NC)
      HIPCK(hipMemcpyAsync(latents + j * NC, cur[j], NC * sizeof(float), hipMemcpyDeviceToDevice, c->stream));
  HIPCK(hipStreamSynchronize(c->stream));
  if (p.policy != DIT_POLICY_THRESHOLD)
    for (int j = 0; j < S; ++j)
      if (c->lanes[j].cnt != B)
        return fail(c, DIT_EBUDGET, "realised NFE differs from the budget (sample " + std::to_string(j) + ")");
  return DIT_OK;
}

}  // namespace

// ====================================================================== C ABI
extern "C" {

dit_status dit_cache_create(const dit_model_config* cfg, const void* weights, size_t nbytes, void* hip_stream,
                            dit_cache** out) {
  g_create_error.clear();
  if (!cfg || !weights || !out) return fail(nullptr, DIT_EINVAL, "null argument");
  *out = nullptr;
  std::string why;
  dit_status st = validate(cfg, why);
  if (st != DIT_OK) return fail(nullptr, st, why);
  dit_cache* c = new dit_cache();
  c->cfg = *cfg;
  c->stream = (hipStream_t)hip_stream;
  c->bf16 = cfg->dtype == DIT_DTYPE_BF16;
  c->esz = c->bf16 ? 2 : 4;
  c->H = cfg->hidden; c->F = cfg->mlp_hidden; c->N = cfg->n_img; c->Nt = cfg->n_txt;
  c->L = cfg->n_cross ? cfg->n_img : cfg->n_img + cfg->n_txt;
  c->C = cfg->in_channels; c->nb = cfg->batch;
  c->stacked = c->bf16 && !cfg->n_cross;
  c->n_mod = 12 * c->H * cfg->n_double + 3 * c->H * cfg->n_single + (cfg->n_cross ? 6 * c->H : 0) + 2 * c->H;
  c->ldY = 4 * c->H + c->F;
  int dev = 0;
  if (hipGetDevice(&dev) == hipSuccess) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0) c->n_cu = n;
  }
  size_t elems = 0;
  layout(c, &elems);
  if (elems * c->esz != nbytes) {
    std::string m = "weight blob is " + std::to_string(nbytes) + " bytes, layout needs " +
                    std::to_string(elems * c->esz);
    delete c;
    return fail(nullptr, DIT_ESHAPE, m);
  }
  c->wbytes = nbytes;
  st = dalloc(c, &c->wdev, nbytes);
  if (st == DIT_OK) st = alloc_workspace(c);
  if (st == DIT_OK) {
    hipError_t e = hipMemcpyAsync(c->wdev, weights, nbytes, hipMemcpyHostToDevice, c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) st = fail(c, DIT_EHIP, std::string("weight upload: ") + hipGetErrorString(e));
  }
  if (st == DIT_OK && c->cand) st = upload_stream_stats(c, (const uint16_t*)weights);
  if (st != DIT_OK) {
    g_create_error = c->err;
    dit_cache_destroy(c);
    return st;
  }
  rebase(c);
  *out = c;
  return DIT_OK;
}

dit_status dit_cache_sample_batch(dit_cache* c, int32_t n_samples, float* latents, const void* text_emb,
                                  const float* gate_weights, size_t gate_len, const dit_sample_params* p,
                                  dit_schedule* out) {
  if (!c) return DIT_EINVAL;
  c->err.clear();
  if (!latents || !text_emb || !p || !out) return fail(c, DIT_EINVAL, "null argument");
  if (n_samples < 1) return fail(c, DIT_EINVAL, "need n_samples >= 1");
  for (int j = 0; j < n_samples; ++j) {
    if (!out[j].full) return fail(c, DIT_EINVAL, "null schedule array");
    out[j].nfe = 0;
    out[j].steps_done = 0;
  }
  if (p->T < 1 || p->B < 1 || p->B > p->T) return fail(c, DIT_EBUDGET, "need 1 <= B <= T");
  if (!(p->tau > 0.0 && p->tau < 1.0)) return fail(c, DIT_EINVAL, "tau must be in (0, 1)");
  if (p->indicator != DIT_INDICATOR_MODULATED && p->indicator != DIT_INDICATOR_PATCH)
    return fail(c, DIT_EINVAL, "bad indicator");
  if (!p->sigmas && !(p->shift > 0.0)) return fail(c, DIT_EINVAL, "shift must be > 0");
  if (p->sigmas)
    for (int i = 0; i <= p->T; ++i) {
      const double s = p->sigmas[i];
      // NaN fails every comparison; equal neighbours would make the UniPC step size zero
      if (!(s >= 0.0 && s <= 1.0) || (i > 0 && !(s < p->sigmas[i - 1])))
        return fail(c, DIT_EINVAL, "sigmas must lie in [0, 1] and decrease strictly");
    }
  if (p->policy != DIT_POLICY_GATE && p->policy != DIT_POLICY_STATIC && p->policy != DIT_POLICY_THRESHOLD)
    return fail(c, DIT_EINVAL, "bad policy");
  if (p->solver != DIT_SOLVER_EULER && p->solver != DIT_SOLVER_UNIPC) return fail(c, DIT_EINVAL, "bad solver");
  if (p->policy == DIT_POLICY_THRESHOLD && std::isnan(p->delta))
    return fail(c, DIT_EINVAL, "threshold delta is NaN");
  if (p->forced_mask)
    for (int j = 0; j < n_samples; ++j) {
      const uint8_t* fm = p->forced_mask + (size_t)j * p->T;
      int ones = 0;
      for (int t = 0; t < p->T; ++t) {
        if (fm[t] > 1) return fail(c, DIT_EINVAL, "forced mask entries must be 0/1");
        ones += fm[t];
      }
      if (fm[0] != 1) return fail(c, DIT_EINVAL, "forced mask needs m_0 = 1");
      if (p->policy != DIT_POLICY_THRESHOLD && ones != p->B)
        return fail(c, DIT_EINVAL, "forced mask needs exactly B ones");
    }
  GateMLP gate;
  if (p->policy == DIT_POLICY_GATE) TRY(parse_gate(c, gate_weights, gate_len, gate));
  const auto t0 = std::chrono::steady_clock::now();
  dit_status st = run_batch(c, n_samples, latents, text_emb, gate, *p, out);
  if (st != DIT_OK) hipStreamSynchronize(c->stream);
  collect_events(c);
  c->stats.sample_ms += std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
  c->stats.samples += (st == DIT_OK) ? n_samples : 0;
  return st;
}

dit_status dit_cache_sample_ex(dit_cache* c, float* latent, const void* text_emb, const float* gate_weights,
                               size_t gate_len, const dit_sample_params* p, dit_schedule* out) {
  return dit_cache_sample_batch(c, 1, latent, text_emb, gate_weights, gate_len, p, out);
}

dit_status dit_cache_sample(dit_cache* c, float* latent, const void* text_emb, int32_t T, int32_t B,
                            const float* gate_weights, size_t gate_len, dit_schedule* out) {
  dit_sample_params p{};
  p.T = T; p.B = B; p.sigmas = nullptr; p.shift = 1.0; p.tau = 0.5; p.guidance = 1.0;
  p.forced_mask = nullptr; p.indicator = DIT_INDICATOR_MODULATED;
  p.policy = DIT_POLICY_GATE; p.delta = 0.0; p.solver = DIT_SOLVER_EULER;
  return dit_cache_sample_ex(c, latent, text_emb, gate_weights, gate_len, &p, out);
}

dit_status dit_gate_logit(const float* gate_weights, size_t gate_len, const double* features, double* logit) {
  g_create_error.clear();
  if (!features || !logit) return fail(nullptr, DIT_EINVAL, "null argument");
  GateMLP g;
  TRY(parse_gate(nullptr, gate_weights, gate_len, g));
  *logit = gate_logit(g, features);
  return DIT_OK;
}

void dit_cache_destroy(dit_cache* c) {
  if (!c) return;
  if (c->stream) hipStreamSynchronize(c->stream);
  free_per_call(c);
  for (Lane& l : c->lanes) free_lane(l);
  void* ps[] = {c->wdev, c->xs, c->X, c->A, c->Y, c->vt, c->modq, c->yf, c->vel, c->ones,
                c->partials, c->cand, c->st_hi, c->st_lo};
  for (void* p : ps)
    if (p) hipFree(p);
  if (c->sums_host) hipHostFree(c->sums_host);
  if (c->ev_sums) hipEventDestroy(c->ev_sums);
  for (hipEvent_t e : c->ev_pool) hipEventDestroy(e);
  delete c;
}

const char* dit_cache_last_error(const dit_cache* c) {
  return c ? c->err.c_str() : g_create_error.c_str();
}

dit_status dit_cache_set_profiling(dit_cache* c, int32_t enable) {
  if (!c) return DIT_EINVAL;
  c->prof = enable != 0;
  return DIT_OK;
}

dit_status dit_cache_get_stats(const dit_cache* c, dit_stats* out) {
  if (!c || !out) return DIT_EINVAL;
  *out = c->stats;
  return DIT_OK;
}

dit_status dit_cache_reset_stats(dit_cache* c) {
  if (!c) return DIT_EINVAL;
  c->stats = dit_stats{};
  return DIT_OK;
}

// ---------------------------------------------------------------- components
dit_status dit_gemm_bf16(const dit_gemm_desc* d, void* hip_stream) {
  dit_cache* c = nullptr;
  if (!d || !d->A || !d->W || !d->C) return fail(c, DIT_EINVAL, "null argument");
  if (d->flags & ~(DIT_EPI_F32 | DIT_EPI_GATED_RES | DIT_EPI_SILU)) return fail(c, DIT_EINVAL, "bad flags");
  if ((d->flags & DIT_EPI_GATED_RES) && (!d->gate || (d->flags & DIT_EPI_F32)))
    return fail(c, DIT_EINVAL, "gated residual needs a gate and bf16 output");
  if (d->M < 0 || d->N < 0 || d->K < 1 || d->K % 8 || d->lda < d->K || d->ldw < d->K || d->gap < 0)
    return fail(c, DIT_ESHAPE, "bad GEMM shape");
  // the last output column is N - 1, plus the gap when it lies past gap_at
  if (d->ldc < (int64_t)d->N + (d->gap && d->gap_at < d->N ? d->gap : 0))
    return fail(c, DIT_ESHAPE, "ldc is smaller than the output row");
  if (d->rms_cols < 0 || d->rms_cols % 128) return fail(c, DIT_ESHAPE, "rms_cols must be a multiple of 128");
  GemmArgs g{};
  g.A = d->A; g.lda = d->lda; g.W = d->W; g.ldw = d->ldw; g.bias = d->bias;
  g.C = d->C; g.ldc = d->ldc; g.gate = d->gate; g.M = d->M; g.N = d->N; g.K = d->K;
  g.flags = d->flags; g.rms_cols = d->rms_cols;
  g.gelu_from = d->gelu_from; g.gap_at = d->gap ? d->gap_at : 0x7fffffff; g.gap = d->gap;
  int dev = 0, ncu = 256;
  hipGetDevice(&dev);
  hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
  hipStream_t s = (hipStream_t)hip_stream;
  HIPCK(dit::launch_gemm_bf16(&g, 1, s, ncu));
  HIPCK(hipStreamSynchronize(s));
  return DIT_OK;
}

dit_status dit_attention_bf16(const void* q, int64_t ldq, const void* k, int64_t ldk, const void* v, int64_t ldv,
                              void* o, int64_t ldo, int32_t Lq, int32_t Lk, int32_t heads, int32_t flags,
                              void* vt_ws, void* hip_stream) {
  dit_cache* c = nullptr;
  if (!q || !k || !v || !o || !vt_ws) return fail(c, DIT_EINVAL, "null argument");
  if (Lq < 1 || Lk < 1 || heads < 1) return fail(c, DIT_ESHAPE, "bad attention shape");
  if (flags & ~DIT_ATTN_BOUNDED_LOGITS) return fail(c, DIT_EINVAL, "bad attention flags");
  if (ldq < heads * 128 || ldk < heads * 128 || ldv < heads * 128 || ldo < heads * 128)
    return fail(c, DIT_ESHAPE, "row stride smaller than heads*128");
  hipStream_t s = (hipStream_t)hip_stream;
  HIPCK(dit::launch_transpose_v_bf16(v, ldv, vt_ws, Lk, heads, s));
  HIPCK(dit::launch_flash_attn_bf16(q, ldq, k, ldk, vt_ws, (int)rup(Lk, 64), o, ldo, Lq, Lk, heads,
                                    (flags & DIT_ATTN_BOUNDED_LOGITS) != 0, s));
  HIPCK(hipStreamSynchronize(s));
  return DIT_OK;
}

}  // extern "C"

// ------------------------------------------------------- allocation-free attention
// Transposed values of dit_attention_bf16_noalloc.  In host code `scratch`
// names a host-side stand-in, not device memory: kernels and copies take
// the address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) uint16_t scratch[DIT_NOALLOC_VT_MAX_ELEMS];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up once per device.
dit_status scratch_ptr(void** out) {
  dit_cache* c = nullptr;
  int dev = -1;
  HIPCK(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(c, DIT_EINVAL, "device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIPCK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(c, DIT_EHIP, "hipGetSymbolAddress returned no address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DIT_OK;
}
}  // namespace

extern "C" dit_status dit_attention_bf16_noalloc(const void* q, int64_t ldq, const void* k, int64_t ldk,
                                                 const void* v, int64_t ldv, void* o, int64_t ldo, int32_t Lq,
                                                 int32_t Lk, int32_t heads, int32_t flags, void* hip_stream) {
  dit_cache* c = nullptr;
  if (!q || !k || !v || !o) return fail(c, DIT_EINVAL, "null argument");
  if (Lq < 1 || Lk < 1 || heads < 1) return fail(c, DIT_ESHAPE, "bad attention shape");
  if (flags & ~DIT_ATTN_BOUNDED_LOGITS) return fail(c, DIT_EINVAL, "bad attention flags");
  if (ldq < heads * 128 || ldk < heads * 128 || ldv < heads * 128 || ldo < heads * 128)
    return fail(c, DIT_ESHAPE, "row stride smaller than heads*128");
  const size_t need = (size_t)heads * 128 * rup((size_t)Lk, 64);
  if (need > (size_t)DIT_NOALLOC_VT_MAX_ELEMS)
    return fail(c, DIT_ESHAPE, "heads * 128 * round_up(Lk, 64) = " + std::to_string(need) +
                                   " exceeds the allocation-free limit of " +
                                   std::to_string((size_t)DIT_NOALLOC_VT_MAX_ELEMS) + " elements");
  void* vt = nullptr;
  TRY(scratch_ptr(&vt));
  hipStream_t s = (hipStream_t)hip_stream;
  HIPCK(dit::launch_transpose_v_bf16(v, ldv, vt, Lk, heads, s));
  HIPCK(dit::launch_flash_attn_bf16(q, ldq, k, ldk, vt, (int)rup(Lk, 64), o, ldo, Lq, Lk, heads,
                                    (flags & DIT_ATTN_BOUNDED_LOGITS) != 0, s));
  HIPCK(hipStreamSynchronize(s));
  return DIT_OK;
}
