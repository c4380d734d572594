"""Random-init DiT backbones of the cached sampler (oracle; test infrastructure).

The paper treats the backbone as external (FLUX.1-dev, Qwen-Image, Wan2.1;
Sec. 4 setup) and caches the residual of the whole block stack.  These are
the shaped stand-ins the workloads use, written out in float64:

  LN        layer norm without affine parameters, eps 1e-6
  RMS       per-head RMS norm of q and k with unit gain, eps 1e-6
  GELU      tanh approximation
  attention softmax(q k^T / sqrt(d)) v per head, non-causal, exact softmax
  modulate  LN(x) * (1 + scale) + shift   (adaLN)

Every value is float64; ``rs`` rounds to the storage dtype S exactly where
the sampler stores a tensor in S (GEMM inputs and outputs, hidden states,
q/k/v, attention outputs).  Pinned: each primitive against torch's own
functional op, whole blocks against scalar brute force on tiny shapes and
against structural invariants (zero gate => identity, image-token
permutation equivariance).
"""
import math

import numpy as np

from .numerics import round_storage, storage_to_f64

LN_EPS = 1e-6
RMS_EPS = 1e-6


# ---------------------------------------------------------------- primitives

def layer_norm(x):
    mu = x.mean(axis=-1, keepdims=True)
    d = x - mu
    var = (d * d).mean(axis=-1, keepdims=True)
    return d / np.sqrt(var + LN_EPS)


def modulate(x, shift, scale):
    return layer_norm(x) * (1.0 + scale) + shift


def rms_heads(x, heads, head_dim):
    """RMS norm of every head_dim-wide slice of the last axis."""
    s = x.reshape(x.shape[:-1] + (heads, head_dim))
    r = np.sqrt((s * s).mean(axis=-1, keepdims=True) + RMS_EPS)
    return (s / r).reshape(x.shape)


def gelu_tanh(x):
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def silu(x):
    return x / (1.0 + np.exp(-x))


def attention(q, k, v, heads, head_dim, q_chunk=2048):
    """Exact softmax attention per head; q [Lq, H], k/v [Lk, H] -> [Lq, H]."""
    Lq = q.shape[0]
    out = np.empty((Lq, heads * head_dim))
    scale = 1.0 / math.sqrt(head_dim)
    for h in range(heads):
        sl = slice(h * head_dim, (h + 1) * head_dim)
        kh, vh = k[:, sl], v[:, sl]
        for lo in range(0, Lq, q_chunk):
            s = (q[lo:lo + q_chunk, sl] @ kh.T) * scale
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[lo:lo + q_chunk, sl] = p @ vh
    return out


def timestep_embedding(sigma, dim=256):
    """Sinusoidal embedding of 1000 * sigma: [cos(a f_k), sin(a f_k)],
    f_k = 10000^(-k / (dim/2))."""
    half = dim // 2
    f = np.exp(-math.log(10000.0) * np.arange(half) / half)
    a = 1000.0 * np.asarray(sigma, np.float64).reshape(-1, 1) * f
    return np.concatenate([np.cos(a), np.sin(a)], axis=1)


# ---------------------------------------------------------------- parameters

class Params:
    """Named storage tensors decoded to float64 on use."""

    def __init__(self, cfg, tensors):
        self.cfg = cfg
        self.t = tensors
        self.rs = round_storage(cfg.dtype)

    def __call__(self, name):
        return storage_to_f64(self.t[name], self.cfg.dtype)

    def linear(self, x, prefix):
        return x @ self(prefix + ".w").T + self(prefix + ".b")


def mod_offsets(cfg):
    """Start of each block's modulation chunk inside one step's vector."""
    H = cfg.hidden
    off = {}
    for i in range(cfg.n_double):
        off[("double", i, "img")] = 12 * H * i
        off[("double", i, "txt")] = 12 * H * i + 6 * H
    base = 12 * H * cfg.n_double
    for i in range(cfg.n_single):
        off[("single", i)] = base + 3 * H * i
    base += 3 * H * cfg.n_single
    if cfg.n_cross:
        off["cross_shared"] = base
        base += 6 * H
    off["final"] = base
    assert base + 2 * H == cfg.n_mod
    return off


def chunks(vec, start, n, H):
    return [vec[start + j * H: start + (j + 1) * H] for j in range(n)]


# ---------------------------------------------------------------- embeddings

def text_in(P, text_b):
    """txt = S(text . W_txt^T + b); text is already stored in S."""
    return P.rs(P.linear(text_b, "txt_in"))


def patch_embed(P, x):
    """h = S(S(x) . W_in^T + b_in); x is the float32 latent [N, C]."""
    return P.rs(P.linear(P.rs(x), "img_in"))


def vec_table(P, sigmas_t, text_b):
    """S(SiLU(vec_t)) for every step: [T, H].

    vec_t = MLP_time(S(temb(sigma_t))) (+ MLP_pool(S(mean_tokens(text))))
    with MLP = Linear -> SiLU (stored in S) -> Linear, vec stored in S."""
    cfg = P.cfg
    temb = P.rs(timestep_embedding(sigmas_t, cfg.time_dim))
    th = P.rs(silu(P.linear(temb, "time_in.0")))
    v = P.linear(th, "time_in.2")
    if cfg.pooled_text:
        pooled = P.rs(text_b.mean(axis=0, keepdims=True))
        ph = P.rs(silu(P.linear(pooled, "pool_in.0")))
        v = v + P.linear(ph, "pool_in.2")
    vec = P.rs(v)
    return P.rs(silu(vec))


def mod_table(P, silu_vec, row_chunk=1 << 16):
    """mod_t = SiLU(vec_t) . W_mod^T + b_mod, float64 [T, n_mod] (not rounded)."""
    cfg = P.cfg
    W = P.t["mod.w"]
    b = P("mod.b")
    out = np.empty((silu_vec.shape[0], cfg.n_mod))
    for lo in range(0, cfg.n_mod, row_chunk):
        hi = min(cfg.n_mod, lo + row_chunk)
        Wc = storage_to_f64(W[lo:hi], cfg.dtype)
        out[:, lo:hi] = silu_vec @ Wc.T + b[lo:hi]
    return out


# ---------------------------------------------------------------- blocks

def _qkv_split(P, y, H):
    cfg = P.cfg
    q = P.rs(rms_heads(y[:, :H], cfg.heads, cfg.head_dim))
    k = P.rs(rms_heads(y[:, H:2 * H], cfg.heads, cfg.head_dim))
    v = P.rs(y[:, 2 * H:3 * H])
    return q, k, v


def double_block(P, i, s_img, s_txt, mod):
    """MMDiT double-stream block: per-stream weights, joint attention over
    [txt; img], sequential attention then MLP, gated residuals."""
    cfg = P.cfg
    H = cfg.hidden
    off = mod_offsets(cfg)
    st = {"img": s_img, "txt": s_txt}
    m = {k: chunks(mod, off[("double", i, k)], 6, H) for k in st}
    qkv = {}
    for k in ("txt", "img"):
        sh1, sc1 = m[k][0], m[k][1]
        a = P.rs(modulate(st[k], sh1, sc1))
        qkv[k] = _qkv_split(P, P.linear(a, f"double.{i}.{k}.qkv"), H)
    q = np.concatenate([qkv["txt"][0], qkv["img"][0]])
    kk = np.concatenate([qkv["txt"][1], qkv["img"][1]])
    v = np.concatenate([qkv["txt"][2], qkv["img"][2]])
    o = P.rs(attention(q, kk, v, cfg.heads, cfg.head_dim))
    nt = s_txt.shape[0]
    o_s = {"txt": o[:nt], "img": o[nt:]}
    out = {}
    for k in ("txt", "img"):
        sh1, sc1, g1, sh2, sc2, g2 = m[k]
        p = f"double.{i}.{k}."
        s = P.rs(st[k] + g1 * P.linear(o_s[k], p + "o"))
        a2 = P.rs(modulate(s, sh2, sc2))
        u = P.rs(gelu_tanh(P.linear(a2, p + "mlp0")))
        out[k] = P.rs(s + g2 * P.linear(u, p + "mlp1"))
    return out["img"], out["txt"]


def single_block(P, i, x, mod):
    """Single-stream block on x = [txt; img]: one fused input projection to
    [q k v | mlp], attention and GELU in parallel, one fused output
    projection of [attn | GELU(mlp)], gated residual."""
    cfg = P.cfg
    H = cfg.hidden
    off = mod_offsets(cfg)
    sh, sc, g = chunks(mod, off[("single", i)], 3, H)
    a = P.rs(modulate(x, sh, sc))
    y = P.linear(a, f"single.{i}.l1")
    q, k, v = _qkv_split(P, y, H)
    u = P.rs(gelu_tanh(y[:, 3 * H:]))
    o = P.rs(attention(q, k, v, cfg.heads, cfg.head_dim))
    return P.rs(x + g * P.linear(np.concatenate([o, u], axis=1), f"single.{i}.l2"))


def cross_mod(P, i, mod):
    """Video block modulation: one shared 6H projection of the step plus a
    learned per-block offset: (shift1, scale1, gate1, shift2, scale2, gate2)."""
    cfg = P.cfg
    H = cfg.hidden
    off = mod_offsets(cfg)
    shared = mod[off["cross_shared"]: off["cross_shared"] + 6 * H]
    e = shared + P(f"cross.{i}.mod_offset")
    return [e[j * H:(j + 1) * H] for j in range(6)]


def cross_block(P, i, x, ctx, mod):
    """Video block: gated self-attention, ungated cross-attention to the
    text tokens (q from LN(x), k/v from the text), gated FFN."""
    cfg = P.cfg
    H = cfg.hidden
    sh1, sc1, g1, sh2, sc2, g2 = cross_mod(P, i, mod)
    p = f"cross.{i}."
    a = P.rs(modulate(x, sh1, sc1))
    q, k, v = _qkv_split(P, P.linear(a, p + "qkv"), H)
    o = P.rs(attention(q, k, v, cfg.heads, cfg.head_dim))
    x = P.rs(x + g1 * P.linear(o, p + "o"))
    c = P.rs(layer_norm(x))
    q2 = P.rs(rms_heads(P.linear(c, p + "xq"), cfg.heads, cfg.head_dim))
    kv = P.linear(ctx, p + "xkv")
    k2 = P.rs(rms_heads(kv[:, :H], cfg.heads, cfg.head_dim))
    v2 = P.rs(kv[:, H:])
    o2 = P.rs(attention(q2, k2, v2, cfg.heads, cfg.head_dim))
    x = P.rs(x + P.linear(o2, p + "xo"))
    a3 = P.rs(modulate(x, sh2, sc2))
    u = P.rs(gelu_tanh(P.linear(a3, p + "ffn0")))
    return P.rs(x + g2 * P.linear(u, p + "ffn1"))


def block_stack(P, h, txt, mod, blocks=None):
    """F(h): the whole block stack on one branch; returns the image rows.

    ``blocks`` optionally limits the run to a list of ("double"|"single"|
    "cross", i) for bounded timing samples."""
    cfg = P.cfg
    if blocks is None:
        blocks = ([("double", i) for i in range(cfg.n_double)]
                  + [("single", i) for i in range(cfg.n_single)]
                  + [("cross", i) for i in range(cfg.n_cross)])
    if cfg.n_cross:
        x = h
        for kind, i in blocks:
            x = cross_block(P, i, x, txt, mod)
        return x
    s_img, s_txt = h, txt
    x = None
    for kind, i in blocks:
        if kind == "double":
            s_img, s_txt = double_block(P, i, s_img, s_txt, mod)
        else:
            if x is None:
                x = np.concatenate([s_txt, s_img])
            x = single_block(P, i, x, mod)
    if x is None:
        return s_img
    return x[txt.shape[0]:]


def first_block_shift_scale(P, mod):
    """(shift, scale) of the first block's image-stream pre-attention adaLN."""
    cfg = P.cfg
    H = cfg.hidden
    off = mod_offsets(cfg)
    if cfg.n_double:
        sh, sc = chunks(mod, off[("double", 0, "img")], 2, H)
    elif cfg.n_single:
        sh, sc = chunks(mod, off[("single", 0)], 2, H)
    else:
        e = cross_mod(P, 0, mod)
        sh, sc = e[0], e[1]
    return sh, sc


def final_layer(P, h_out, mod):
    """v = S(modulate(h_out, shift_f, scale_f)) . W_out^T + b_out, kept in f32."""
    cfg = P.cfg
    H = cfg.hidden
    off = mod_offsets(cfg)
    sh, sc = chunks(mod, off["final"], 2, H)
    y = P.rs(modulate(h_out, sh, sc))
    v = P.linear(y, "final")
    return v.astype(np.float32).astype(np.float64)
