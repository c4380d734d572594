"""Workload registry and seeded synthetic inputs.

This module is shared by the CPU oracle, the tests and the benchmark.  It
holds shapes and random-number generation only: nothing in it computes any
part of the sampler (no normalisation, no attention, no gate, no pacing).

Every tensor is drawn from its own child stream
``SeedSequence([seed, stream, index])`` so that any single tensor can be
regenerated without drawing the ones before it.  Weights and biases are
N(0, std^2) with std = 0.02, the latent and the text embeddings N(0, 1),
the gate parameters N(0, 0.3^2).  For bf16 workloads every weight and the
text embeddings are rounded once, round-to-nearest-even, to bfloat16 and
kept as raw uint16 bit patterns: the device path and the oracle then read
bit-identical values.

The flat weight blob concatenates the tensors in ``weight_specs(cfg)``
order; every tensor is stored row-major, linear weights as ``[out, in]``.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

# Stream ids of the child seeds.
_W, _LATENT, _TEXT, _GATE = 0, 1, 2, 3


@dataclass(frozen=True)
class ModelConfig:
    name: str
    dtype: str              # storage dtype: "f32" or "bf16"
    n_double: int           # double-stream (MMDiT) blocks
    n_single: int           # single-stream blocks, after the double ones
    n_cross: int            # video blocks: self-attn + cross-attn + FFN
    hidden: int             # H
    heads: int
    head_dim: int
    mlp_hidden: int         # F
    in_channels: int        # C, latent channels per token
    ctx_dim: int            # width of the text embeddings
    n_img: int              # N, image / video latent tokens
    n_txt: int              # N_t, text tokens
    batch: int = 1          # 1, or 2 for a (cond, uncond) guidance pair
    pooled_text: bool = True  # vec also gets an MLP of the mean text token
    time_dim: int = 256
    weight_std: float = 0.02

    def __post_init__(self):
        assert self.dtype in ("f32", "bf16")
        assert self.heads * self.head_dim == self.hidden
        assert self.batch in (1, 2)
        assert (self.n_cross == 0) or (self.n_double == 0 and self.n_single == 0)
        assert self.n_double + self.n_single + self.n_cross >= 1

    @property
    def n_mod(self) -> int:
        """Width of the modulation projection of one step."""
        H = self.hidden
        n = 12 * H * self.n_double + 3 * H * self.n_single
        if self.n_cross:
            n += 6 * H
        return n + 2 * H


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelConfig
    T: int
    B: int
    shift: float
    guidance: float
    seed: int
    gate_widths: tuple = (8, 32, 16, 1)
    gate_std: float = 0.3
    note: str = ""
    solver: str = "euler"   # step rule: "euler", or "unipc" (the paper's Wan sampler)


def _m(**kw) -> ModelConfig:
    return ModelConfig(**kw)


# Paper-shaped workloads (random init).  Token counts follow the latent
# grids: FLUX 1024^2 -> 64x64 = 4096 tokens of 64 channels (2x2 patches of
# a 16-channel VAE latent), 2048^2 -> 16384; Wan 81 frames 480x832 ->
# 21x30x52 = 32760 tokens.
WORKLOADS = {
    "tiny": Workload(
        "tiny",
        _m(name="tiny", dtype="f32", n_double=0, n_single=2, n_cross=0,
           hidden=128, heads=4, head_dim=32, mlp_hidden=512, in_channels=16,
           ctx_dim=128, n_img=64, n_txt=16),
        T=10, B=5, shift=1.0, guidance=1.0, seed=0),
    "flux1024": Workload(
        "flux1024",
        _m(name="flux1024", dtype="bf16", n_double=19, n_single=38, n_cross=0,
           hidden=3072, heads=24, head_dim=128, mlp_hidden=12288,
           in_channels=64, ctx_dim=4096, n_img=4096, n_txt=512),
        T=28, B=10, shift=3.0, guidance=1.0, seed=42),
    "flux2048": Workload(
        "flux2048",
        _m(name="flux2048", dtype="bf16", n_double=19, n_single=38, n_cross=0,
           hidden=3072, heads=24, head_dim=128, mlp_hidden=12288,
           in_channels=64, ctx_dim=4096, n_img=16384, n_txt=512),
        T=50, B=10, shift=3.0, guidance=1.0, seed=42),
    "qwen_cfg": Workload(
        "qwen_cfg",
        _m(name="qwen_cfg", dtype="bf16", n_double=60, n_single=0, n_cross=0,
           hidden=3072, heads=24, head_dim=128, mlp_hidden=12288,
           in_channels=64, ctx_dim=3584, n_img=4096, n_txt=256, batch=2,
           pooled_text=False),
        T=50, B=20, shift=3.0, guidance=4.0, seed=42),
    "wan14b": Workload(
        "wan14b",
        _m(name="wan14b", dtype="bf16", n_double=0, n_single=0, n_cross=40,
           hidden=5120, heads=40, head_dim=128, mlp_hidden=13824,
           in_channels=64, ctx_dim=4096, n_img=32760, n_txt=512,
           pooled_text=False),
        T=50, B=12, shift=5.0, guidance=1.0, seed=42, solver="unipc"),
    # Small parity workloads: several GEMM / attention tiles and ragged tails,
    # still quick for the oracle.
    "small_bf16": Workload(
        "small_bf16",
        _m(name="small_bf16", dtype="bf16", n_double=2, n_single=2, n_cross=0,
           hidden=256, heads=2, head_dim=128, mlp_hidden=1024, in_channels=64,
           ctx_dim=96, n_img=200, n_txt=40),
        T=8, B=4, shift=3.0, guidance=1.0, seed=7),
    "small_f32": Workload(
        "small_f32",
        _m(name="small_f32", dtype="f32", n_double=2, n_single=2, n_cross=0,
           hidden=192, heads=3, head_dim=64, mlp_hidden=768, in_channels=16,
           ctx_dim=80, n_img=150, n_txt=21),
        T=8, B=3, shift=3.0, guidance=1.0, seed=11),
    "small_cfg_bf16": Workload(
        "small_cfg_bf16",
        _m(name="small_cfg_bf16", dtype="bf16", n_double=2, n_single=0, n_cross=0,
           hidden=256, heads=2, head_dim=128, mlp_hidden=1024, in_channels=64,
           ctx_dim=72, n_img=136, n_txt=24, batch=2, pooled_text=False),
        T=8, B=4, shift=3.0, guidance=4.0, seed=5),
    # Token counts that are multiples of 32: the stacked block stack gates
    # the residual of each sequence inside one GEMM launch.
    "small_seg_bf16": Workload(
        "small_seg_bf16",
        _m(name="small_seg_bf16", dtype="bf16", n_double=2, n_single=2, n_cross=0,
           hidden=256, heads=2, head_dim=128, mlp_hidden=1024, in_channels=64,
           ctx_dim=96, n_img=512, n_txt=128),
        T=8, B=4, shift=3.0, guidance=1.0, seed=13),
    # Shapes the column-sliced step kernel does not take (H not a multiple
    # of 256; 32 latent channels): the row-tiled fused kernels run instead.
    "small_w384_bf16": Workload(
        "small_w384_bf16",
        _m(name="small_w384_bf16", dtype="bf16", n_double=1, n_single=1, n_cross=0,
           hidden=384, heads=3, head_dim=128, mlp_hidden=1536, in_channels=64,
           ctx_dim=96, n_img=176, n_txt=40),
        T=8, B=4, shift=3.0, guidance=1.0, seed=17),
    "small_c32_bf16": Workload(
        "small_c32_bf16",
        _m(name="small_c32_bf16", dtype="bf16", n_double=1, n_single=1, n_cross=0,
           hidden=256, heads=2, head_dim=128, mlp_hidden=1024, in_channels=32,
           ctx_dim=96, n_img=184, n_txt=40),
        T=8, B=4, shift=3.0, guidance=1.0, seed=19),
    # Fewer image tokens than one 32-token tile of the column-sliced step
    # kernel (a single ragged tile), single sample and guidance pair.
    "micro_bf16": Workload(
        "micro_bf16",
        _m(name="micro_bf16", dtype="bf16", n_double=1, n_single=1, n_cross=0,
           hidden=256, heads=2, head_dim=128, mlp_hidden=1024, in_channels=64,
           ctx_dim=64, n_img=7, n_txt=5),
        T=8, B=4, shift=3.0, guidance=1.0, seed=23),
    "micro_cfg_bf16": Workload(
        "micro_cfg_bf16",
        _m(name="micro_cfg_bf16", dtype="bf16", n_double=2, n_single=0, n_cross=0,
           hidden=512, heads=4, head_dim=128, mlp_hidden=2048, in_channels=64,
           ctx_dim=64, n_img=33, n_txt=6, batch=2, pooled_text=False),
        T=8, B=3, shift=3.0, guidance=4.0, seed=29),
    "small_cross_bf16": Workload(
        "small_cross_bf16",
        _m(name="small_cross_bf16", dtype="bf16", n_double=0, n_single=0, n_cross=2,
           hidden=256, heads=2, head_dim=128, mlp_hidden=864, in_channels=64,
           ctx_dim=64, n_img=210, n_txt=30, pooled_text=False),
        T=8, B=3, shift=5.0, guidance=1.0, seed=9),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def reduced(w: Workload, *, n_double=None, n_single=None, n_cross=None,
            T=None, B=None, name=None) -> Workload:
    """Same widths and token counts with fewer blocks / steps."""
    m = w.model
    m2 = dataclasses.replace(
        m,
        n_double=m.n_double if n_double is None else n_double,
        n_single=m.n_single if n_single is None else n_single,
        n_cross=m.n_cross if n_cross is None else n_cross,
        name=name or m.name + "_reduced")
    return dataclasses.replace(w, model=m2, T=w.T if T is None else T,
                               B=w.B if B is None else B, name=m2.name)


# ---------------------------------------------------------------- weights

def weight_specs(cfg: ModelConfig):
    """[(name, shape)] in blob order."""
    H, F, C, X = cfg.hidden, cfg.mlp_hidden, cfg.in_channels, cfg.ctx_dim
    s = [("img_in.w", (H, C)), ("img_in.b", (H,)),
         ("txt_in.w", (H, X)), ("txt_in.b", (H,)),
         ("time_in.0.w", (H, cfg.time_dim)), ("time_in.0.b", (H,)),
         ("time_in.2.w", (H, H)), ("time_in.2.b", (H,))]
    if cfg.pooled_text:
        s += [("pool_in.0.w", (H, X)), ("pool_in.0.b", (H,)),
              ("pool_in.2.w", (H, H)), ("pool_in.2.b", (H,))]
    s += [("mod.w", (cfg.n_mod, H)), ("mod.b", (cfg.n_mod,))]
    for i in range(cfg.n_double):
        for st in ("img", "txt"):
            p = f"double.{i}.{st}."
            s += [(p + "qkv.w", (3 * H, H)), (p + "qkv.b", (3 * H,)),
                  (p + "o.w", (H, H)), (p + "o.b", (H,)),
                  (p + "mlp0.w", (F, H)), (p + "mlp0.b", (F,)),
                  (p + "mlp1.w", (H, F)), (p + "mlp1.b", (H,))]
    for i in range(cfg.n_single):
        p = f"single.{i}."
        s += [(p + "l1.w", (3 * H + F, H)), (p + "l1.b", (3 * H + F,)),
              (p + "l2.w", (H, H + F)), (p + "l2.b", (H,))]
    for i in range(cfg.n_cross):
        p = f"cross.{i}."
        s += [(p + "mod_offset", (6 * H,)),
              (p + "qkv.w", (3 * H, H)), (p + "qkv.b", (3 * H,)),
              (p + "o.w", (H, H)), (p + "o.b", (H,)),
              (p + "xq.w", (H, H)), (p + "xq.b", (H,)),
              (p + "xkv.w", (2 * H, H)), (p + "xkv.b", (2 * H,)),
              (p + "xo.w", (H, H)), (p + "xo.b", (H,)),
              (p + "ffn0.w", (F, H)), (p + "ffn0.b", (F,)),
              (p + "ffn1.w", (H, F)), (p + "ffn1.b", (H,))]
    s += [("final.w", (C, H)), ("final.b", (C,))]
    return s


def weight_count(cfg: ModelConfig) -> int:
    return int(sum(int(np.prod(sh)) for _, sh in weight_specs(cfg)))


def storage_np_dtype(cfg: ModelConfig):
    return np.uint16 if cfg.dtype == "bf16" else np.float32


_CHUNK = 1 << 22


def _bf16_bits_inplace(src32: np.ndarray, dst16: np.ndarray, tmp: np.ndarray):
    """float32 -> bfloat16 bits, round to nearest even (finite inputs)."""
    u = src32.view(np.uint32)
    t = tmp[: u.size]
    np.right_shift(u, 16, out=t)
    np.bitwise_and(t, 1, out=t)
    np.add(t, 0x7FFF, out=t)
    np.add(t, u, out=t)
    np.right_shift(t, 16, out=t)
    dst16[...] = t


def _fill_normal(dst: np.ndarray, seed_key, std: float, bf16: bool):
    """Fill a flat array (float32 or uint16-as-bf16) with N(0, std^2)."""
    rng = np.random.default_rng(np.random.SeedSequence(list(seed_key)))
    n = dst.size
    buf = np.empty(min(n, _CHUNK), np.float32)
    tmp = np.empty(min(n, _CHUNK), np.uint32) if bf16 else None
    for lo in range(0, n, _CHUNK):
        hi = min(n, lo + _CHUNK)
        b = buf[: hi - lo]
        rng.standard_normal(out=b, dtype=np.float32)
        if std != 1.0:
            np.multiply(b, np.float32(std), out=b)
        if bf16:
            _bf16_bits_inplace(b, dst[lo:hi], tmp)
        else:
            dst[lo:hi] = b


def _threads():
    n = os.environ.get("SYNTH_THREADS")
    if n:
        return max(1, int(n))
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:  # pragma: no cover
        return 4


@dataclass
class Weights:
    cfg: ModelConfig
    blob: np.ndarray                 # flat, uint16 (bf16 bits) or float32
    tensors: dict = field(default_factory=dict)   # name -> view into blob

    @property
    def nbytes(self) -> int:
        return int(self.blob.nbytes)


def make_weights(cfg: ModelConfig, seed: int) -> Weights:
    """Seeded N(0, weight_std^2) weights in blob order (bf16 bits or f32)."""
    specs = weight_specs(cfg)
    total = weight_count(cfg)
    dt = storage_np_dtype(cfg)
    blob = np.empty(total, dt)
    tensors, jobs, off = {}, [], 0
    for idx, (name, shape) in enumerate(specs):
        n = int(np.prod(shape))
        view = blob[off: off + n]
        tensors[name] = view.reshape(shape)
        jobs.append((view, (seed, _W, idx)))
        off += n
    bf16 = cfg.dtype == "bf16"
    big = [j for j in jobs if j[0].size >= _CHUNK]
    small = [j for j in jobs if j[0].size < _CHUNK]
    for v, k in small:
        _fill_normal(v, k, cfg.weight_std, bf16)
    if big:
        # Split big tensors into independent sub-streams so threads share work.
        tasks = []
        for v, k in big:
            for part, lo in enumerate(range(0, v.size, 16 * _CHUNK)):
                tasks.append((v[lo: lo + 16 * _CHUNK], tuple(k) + (part,)))
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(lambda a: _fill_normal(a[0], a[1], cfg.weight_std, bf16), tasks))
    return Weights(cfg, blob, tensors)


def make_weight_tensor(cfg: ModelConfig, seed: int, name: str) -> np.ndarray:
    """Regenerate one tensor of ``make_weights`` without drawing the rest."""
    specs = weight_specs(cfg)
    idx = [n for n, _ in specs].index(name)
    shape = specs[idx][1]
    n = int(np.prod(shape))
    out = np.empty(n, storage_np_dtype(cfg))
    bf16 = cfg.dtype == "bf16"
    if n >= _CHUNK:
        for part, lo in enumerate(range(0, n, 16 * _CHUNK)):
            _fill_normal(out[lo: lo + 16 * _CHUNK], (seed, _W, idx, part), cfg.weight_std, bf16)
    else:
        _fill_normal(out, (seed, _W, idx), cfg.weight_std, bf16)
    return out.reshape(shape)


# ----------------------------------------------------------------- inputs

def make_latent(cfg: ModelConfig, seed: int) -> np.ndarray:
    """x_0 ~ N(0, 1), float32 [N, C] (shared by both guidance branches)."""
    out = np.empty(cfg.n_img * cfg.in_channels, np.float32)
    _fill_normal(out, (seed, _LATENT, 0), 1.0, False)
    return out.reshape(cfg.n_img, cfg.in_channels)


def make_text(cfg: ModelConfig, seed: int) -> np.ndarray:
    """Text embeddings ~ N(0, 1) in storage dtype, [batch, N_t, ctx].

    Branch 0 is the conditional prompt, branch 1 (guidance only) an
    independent draw standing for the unconditional one."""
    bf16 = cfg.dtype == "bf16"
    out = np.empty(cfg.batch * cfg.n_txt * cfg.ctx_dim, storage_np_dtype(cfg))
    n1 = cfg.n_txt * cfg.ctx_dim
    for b in range(cfg.batch):
        _fill_normal(out[b * n1:(b + 1) * n1], (seed, _TEXT, b), 1.0, bf16)
    return out.reshape(cfg.batch, cfg.n_txt, cfg.ctx_dim)


def gate_param_count(widths) -> int:
    return int(sum(widths[i] * widths[i - 1] + widths[i] for i in range(1, len(widths))))


def make_gate_blob(widths=(8, 32, 16, 1), seed: int = 0, std: float = 0.3,
                   zscore=None) -> np.ndarray:
    """Self-describing float32 gate blob.

    Layout: [k, d_0 .. d_{k-1}, zflag, (mu[d_0], sd[d_0] if zflag),
    W_1, b_1, ..., W_{k-1}, b_{k-1}], W_l row-major [d_l, d_{l-1}].
    Parameters ~ N(0, std^2).  ``zscore`` = (mu, sd) arrays or None."""
    widths = tuple(int(w) for w in widths)
    n = gate_param_count(widths)
    params = np.empty(n, np.float32)
    _fill_normal(params, (seed, _GATE, 0), std, False)
    head = [float(len(widths))] + [float(w) for w in widths]
    if zscore is None:
        head.append(0.0)
        z = []
    else:
        mu, sd = (np.asarray(a, np.float32) for a in zscore)
        assert mu.shape == (widths[0],) and sd.shape == (widths[0],)
        head.append(1.0)
        z = list(mu) + list(sd)
    return np.concatenate([np.asarray(head + z, np.float32), params])


def make_branched_gate_blob(branches=((3, 8, 8), (3, 8, 8)), trunk=(16, 32, 1), seed: int = 0,
                            std: float = 0.3, zscore=None) -> np.ndarray:
    """Self-describing float32 blob of a branched gate (default: the Wan
    gate shape of App. A.2, 785 parameters).

    Layout: [-n, (k_j, widths_j) for each branch, k, trunk widths, zflag,
    (mu[D], sd[D] if zflag), branch parameters in branch order, trunk
    parameters], D = sum of the branch input widths; each network's
    parameters are W_1, b_1, W_2, b_2, ... with W_l row-major
    [d_l, d_{l-1}].
    Parameters ~ N(0, std^2).  ``zscore`` = (mu, sd) arrays or None."""
    branches = [tuple(int(w) for w in b) for b in branches]
    trunk = tuple(int(w) for w in trunk)
    n = sum(gate_param_count(b) for b in branches) + gate_param_count(trunk)
    params = np.empty(n, np.float32)
    _fill_normal(params, (seed, _GATE, 1), std, False)
    head = [-float(len(branches))]
    for b in branches + [trunk]:
        head += [float(len(b))] + [float(w) for w in b]
    d_in = sum(b[0] for b in branches)
    if zscore is None:
        head.append(0.0)
        z = []
    else:
        mu, sd = (np.asarray(a, np.float32) for a in zscore)
        assert mu.shape == (d_in,) and sd.shape == (d_in,)
        head.append(1.0)
        z = list(mu) + list(sd)
    return np.concatenate([np.asarray(head + z, np.float32), params])


def make_inputs(w: Workload):
    """(weights, latent, text, gate blob) of a workload, all seeded."""
    cfg = w.model
    return (make_weights(cfg, w.seed), make_latent(cfg, w.seed),
            make_text(cfg, w.seed), make_gate_blob(w.gate_widths, w.seed, w.gate_std))


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns (uint16) to float32."""
    return (bits.astype(np.uint32) << 16).view(np.float32)
