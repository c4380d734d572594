"""Pins of the oracle's conditioning and output plumbing: the per-step
vector table, the modulation table, the first block's (shift, scale) and the
final layer.

Two kinds of check, neither of which re-types the oracle's own code:

* torch compositions of library modules (``nn.Linear``, ``F.silu``,
  ``F.layer_norm``) loaded with the same blob tensors, on an f32 model where
  storing a value in S is torch's own float64 -> float32 conversion;
* modulation vectors whose every H-wide chunk holds its own chunk id, read
  back through the oracle's functions and compared with the chunk order the
  weight-blob comment of the C header states (double block i at 12 H i: image
  stream shift1, scale1, gate1, shift2, scale2, gate2, then the text stream;
  single block i at 12 H n_double + 3 H i: shift, scale, gate; video blocks:
  one shared 6 H chunk plus each block's offset; final layer: the last 2 H as
  shift, scale), and behavioural probes in which only one chunk is nonzero.
"""
import dataclasses

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import dit
from oracle.numerics import round_f32
from tests._nano import NANO, NANO_BF16, NANO_CROSS, inputs

# ---------------------------------------------------------------- helpers


def torch_linear(P, prefix):
    """nn.Linear holding the blob's tensor pair (float64)."""
    W = torch.from_numpy(P(prefix + ".w"))
    b = torch.from_numpy(P(prefix + ".b"))
    m = torch.nn.Linear(W.shape[1], W.shape[0], dtype=torch.float64)
    with torch.no_grad():
        m.weight.copy_(W)
        m.bias.copy_(b)
    return m


def f32(t):
    """Store in S for an f32 model: torch's own float64 -> float32 rounding."""
    return t.to(torch.float32).to(torch.float64)


def sinusoid(sigmas, dim):
    """Sinusoidal embedding of 1000 sigma (pinned by closed forms in the
    primitive tests; only the composition around it is checked here)."""
    return torch.from_numpy(dit.timestep_embedding(sigmas, dim))


def chunk_id_vector(cfg):
    """One step's modulation vector, chunk k (H wide) filled with k."""
    H = cfg.hidden
    return np.repeat(np.arange(cfg.n_mod // H, dtype=np.float64), H)


def header_chunks(cfg):
    """Chunk ids as the header's layout names them (not the oracle's table)."""
    ids, k = {}, 0
    for i in range(cfg.n_double):
        for stream in ("img", "txt"):
            for part in ("shift1", "scale1", "gate1", "shift2", "scale2", "gate2"):
                ids[("double", i, stream, part)] = k
                k += 1
    for i in range(cfg.n_single):
        for part in ("shift", "scale", "gate"):
            ids[("single", i, part)] = k
            k += 1
    if cfg.n_cross:
        for part in ("shift1", "scale1", "gate1", "shift2", "scale2", "gate2"):
            ids[("cross_shared", part)] = k
            k += 1
    ids[("final", "shift")] = k
    ids[("final", "scale")] = k + 1
    assert (k + 2) * cfg.hidden == cfg.n_mod
    return ids


NANO_SINGLE = dataclasses.replace(NANO, name="nano_single", n_double=0, n_single=2)
NANO_NOPOOL = dataclasses.replace(NANO, name="nano_nopool", pooled_text=False)

# ---------------------------------------------------------------- vec table


@pytest.mark.parametrize("cfg", [NANO, NANO_NOPOOL], ids=lambda c: c.name)
def test_vec_table_vs_torch_modules(cfg):
    w, _, text = inputs(cfg, seed=21)
    P = dit.Params(cfg, w.tensors)
    sig = np.array([1.0, 0.83, 0.41, 0.05])
    got = dit.vec_table(P, sig, P.rs(text[0].astype(np.float64)))
    t0, t2 = torch_linear(P, "time_in.0"), torch_linear(P, "time_in.2")
    with torch.no_grad():
        temb = f32(sinusoid(sig, cfg.time_dim))
        v = t2(f32(F.silu(t0(temb))))
        if cfg.pooled_text:
            p0, p2 = torch_linear(P, "pool_in.0"), torch_linear(P, "pool_in.2")
            pooled = f32(torch.from_numpy(text[0].astype(np.float64)).mean(dim=0, keepdim=True))
            v = v + p2(f32(F.silu(p0(pooled))))
        ref = f32(F.silu(f32(v))).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-6, atol=1e-7)
    # the SiLU of the output is applied: undoing it would give negative
    # values below -0.2785 (the minimum of SiLU), which must not occur
    assert got.min() >= -0.2785
    assert got.shape == (len(sig), cfg.hidden)


def test_vec_table_pooled_text_is_a_token_mean():
    cfg = NANO
    w, _, text = inputs(cfg, seed=22)
    P = dit.Params(cfg, w.tensors)
    sig = np.array([0.7])
    t = text[0].astype(np.float64)
    a = dit.vec_table(P, sig, t)
    b = dit.vec_table(P, sig, t[::-1].copy())          # token order is irrelevant
    np.testing.assert_array_equal(a, b)
    c = dit.vec_table(P, sig, t + 0.5)                  # content is not
    assert np.max(np.abs(a - c)) > 1e-4
    nop = dit.Params(NANO_NOPOOL, inputs(NANO_NOPOOL, seed=22)[0].tensors)
    np.testing.assert_array_equal(dit.vec_table(nop, sig, t), dit.vec_table(nop, sig, t + 0.5))


def test_vec_table_bf16_within_one_rounding():
    """bf16 model: torch rounds float64 -> bfloat16 through float32 (two
    roundings), the oracle once; the two agree to one bf16 ulp."""
    cfg = NANO_BF16
    w, _, text = inputs(cfg, seed=23)
    P = dit.Params(cfg, w.tensors)
    sig = np.array([1.0, 0.5, 0.02])
    t64 = P.rs(text[0].astype(np.float64)) if text.dtype != np.uint16 else (
        (text[0].astype(np.uint32) << 16).view(np.float32).astype(np.float64))
    got = dit.vec_table(P, sig, t64)

    def bf(x):
        return x.to(torch.bfloat16).to(torch.float64)

    t0, t2 = torch_linear(P, "time_in.0"), torch_linear(P, "time_in.2")
    p0, p2 = torch_linear(P, "pool_in.0"), torch_linear(P, "pool_in.2")
    with torch.no_grad():
        v = t2(bf(F.silu(t0(bf(sinusoid(sig, cfg.time_dim))))))
        v = v + p2(bf(F.silu(p0(bf(torch.from_numpy(t64).mean(dim=0, keepdim=True))))))
        ref = bf(F.silu(bf(v))).numpy()
    close = np.abs(got - ref) <= 2.0 ** -7 * np.abs(ref) + 1e-12
    assert close.mean() > 0.97, close.mean()
    assert np.abs(got - ref).max() <= 0.05 * np.abs(ref).max()

# ---------------------------------------------------------------- mod table


@pytest.mark.parametrize("cfg", [NANO, NANO_BF16, NANO_CROSS], ids=lambda c: c.name)
def test_mod_table_is_a_linear_of_silu_vec(cfg):
    w, _, _ = inputs(cfg, seed=24)
    P = dit.Params(cfg, w.tensors)
    sv = np.random.default_rng(3).standard_normal((5, cfg.hidden))
    got = dit.mod_table(P, sv, row_chunk=7)     # chunking must not matter
    with torch.no_grad():
        ref = torch_linear(P, "mod")(torch.from_numpy(sv)).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    assert got.shape == (5, cfg.n_mod)

# ---------------------------------------------------------------- chunk layout


@pytest.mark.parametrize("cfg", [NANO, NANO_SINGLE, NANO_CROSS], ids=lambda c: c.name)
def test_first_block_shift_scale_reads_the_header_chunks(cfg):
    w, _, _ = inputs(cfg, seed=25)
    P = dit.Params(cfg, w.tensors)
    ids = header_chunks(cfg)
    sh, sc = dit.first_block_shift_scale(P, chunk_id_vector(cfg))
    if cfg.n_double:
        want = (ids[("double", 0, "img", "shift1")], ids[("double", 0, "img", "scale1")])
        off = (0.0, 0.0)
    elif cfg.n_single:
        want = (ids[("single", 0, "shift")], ids[("single", 0, "scale")])
        off = (0.0, 0.0)
    else:
        want = (ids[("cross_shared", "shift1")], ids[("cross_shared", "scale1")])
        o = P("cross.0.mod_offset")
        off = (o[:cfg.hidden], o[cfg.hidden:2 * cfg.hidden])
    np.testing.assert_array_equal(sh, want[0] + off[0])
    np.testing.assert_array_equal(sc, want[1] + off[1])


@pytest.mark.parametrize("cfg", [NANO, NANO_BF16, NANO_CROSS], ids=lambda c: c.name)
def test_final_layer_vs_torch_and_header_chunks(cfg):
    w, _, _ = inputs(cfg, seed=26)
    P = dit.Params(cfg, w.tensors)
    rng = np.random.default_rng(4)
    h = P.rs(rng.standard_normal((7, cfg.hidden)) * 2 + 0.3)
    mod = rng.standard_normal(cfg.n_mod)
    ids = header_chunks(cfg)
    H = cfg.hidden
    shift = mod[ids[("final", "shift")] * H:(ids[("final", "shift")] + 1) * H]
    scale = mod[ids[("final", "scale")] * H:(ids[("final", "scale")] + 1) * H]
    got = dit.final_layer(P, h, mod)
    with torch.no_grad():
        y = F.layer_norm(torch.from_numpy(h), (H,), eps=1e-6) * (1 + torch.from_numpy(scale)) + torch.from_numpy(shift)
        y = torch.from_numpy(P.rs(y.numpy()))       # stored in S before the projection
        ref = round_f32(torch_linear(P, "final")(y).numpy())
    if cfg.dtype == "f32":
        np.testing.assert_allclose(got, ref, rtol=1e-6, atol=1e-7)
    else:
        np.testing.assert_allclose(got, ref, rtol=1e-5, atol=1e-6)
    # chunk roles: constant rows have LN = 0, so v = shift W^T + b whatever the
    # scale; rows of +-1 have LN = +-1, so v moves with (1 + scale)
    ids_vec = chunk_id_vector(cfg)
    flat = np.ones((2, H))
    v0 = dit.final_layer(P, flat, ids_vec)
    Wf, bf = P("final.w"), P("final.b")
    s_id, c_id = ids[("final", "shift")], ids[("final", "scale")]
    exp0 = round_f32(P.rs(np.full((1, H), float(s_id))) @ Wf.T + bf)
    np.testing.assert_allclose(v0, np.repeat(exp0, 2, axis=0), rtol=1e-12, atol=1e-12)
    pm = np.tile(np.array([1.0, -1.0]), H // 2)[None, :]
    v1 = dit.final_layer(P, pm, ids_vec)
    ln = pm / np.sqrt(1.0 + 1e-6)
    exp1 = round_f32(P.rs(ln * (1 + c_id) + s_id) @ Wf.T + bf)
    np.testing.assert_allclose(v1, exp1, rtol=1e-12, atol=1e-12)

# ---------------------------------------------------------------- block chunk roles


def _gates_off(cfg, ids):
    mod = np.random.default_rng(5).standard_normal(cfg.n_mod) * 0.5
    H = cfg.hidden
    for key, k in ids.items():
        if key[-1] in ("gate", "gate1", "gate2"):
            mod[k * H:(k + 1) * H] = 0.0
    return mod


def _set(mod, k, H, val):
    m = mod.copy()
    m[k * H:(k + 1) * H] = val
    return m


def test_double_block_chunk_roles():
    """With every gate off the block is the identity; switching one stream's
    gate on moves only that stream; a stream's shift1/scale1 act only when its
    gate1 is on, its shift2/scale2 only when its gate2 is on."""
    cfg = NANO
    w, _, _ = inputs(cfg, seed=27)
    P = dit.Params(cfg, w.tensors)
    rng = np.random.default_rng(6)
    h = P.rs(rng.standard_normal((cfg.n_img, cfg.hidden)))
    txt = P.rs(rng.standard_normal((cfg.n_txt, cfg.hidden)))
    ids = header_chunks(cfg)
    H = cfg.hidden
    base = _gates_off(cfg, ids)
    i0, t0 = dit.double_block(P, 0, h, txt, base)
    np.testing.assert_array_equal(i0, h)
    np.testing.assert_array_equal(t0, txt)
    for stream, other in (("img", "txt"), ("txt", "img")):
        for g in ("gate1", "gate2"):
            m = _set(base, ids[("double", 0, stream, g)], H, 0.7)
            out = dict(zip(("img", "txt"), dit.double_block(P, 0, h, txt, m)))
            ref = {"img": h, "txt": txt}
            assert np.max(np.abs(out[stream] - ref[stream])) > 1e-3, (stream, g)
            np.testing.assert_array_equal(out[other], ref[other])
        # gate1 on, gate2 off: shift1 matters, shift2 does not
        m = _set(base, ids[("double", 0, stream, "gate1")], H, 0.7)
        a = dit.double_block(P, 0, h, txt, m)
        b = dit.double_block(P, 0, h, txt, _set(m, ids[("double", 0, stream, "shift2")], H, 3.0))
        c = dit.double_block(P, 0, h, txt, _set(m, ids[("double", 0, stream, "scale2")], H, 3.0))
        d = dit.double_block(P, 0, h, txt, _set(m, ids[("double", 0, stream, "shift1")], H, 3.0))
        np.testing.assert_array_equal(a[0], b[0])
        np.testing.assert_array_equal(a[0], c[0])
        k = 0 if stream == "img" else 1
        assert np.max(np.abs(a[k] - d[k])) > 1e-3
        # gate2 on, gate1 off: shift2 / scale2 matter, shift1 does not
        m = _set(base, ids[("double", 0, stream, "gate2")], H, 0.7)
        a = dit.double_block(P, 0, h, txt, m)
        b = dit.double_block(P, 0, h, txt, _set(m, ids[("double", 0, stream, "shift1")], H, 3.0))
        e = dit.double_block(P, 0, h, txt, _set(m, ids[("double", 0, stream, "scale2")], H, 3.0))
        np.testing.assert_array_equal(a[k], b[k])
        assert np.max(np.abs(a[k] - e[k])) > 1e-3


def test_single_block_chunk_roles():
    cfg = NANO_SINGLE
    w, _, _ = inputs(cfg, seed=28)
    P = dit.Params(cfg, w.tensors)
    x = P.rs(np.random.default_rng(7).standard_normal((cfg.n_txt + cfg.n_img, cfg.hidden)))
    ids = header_chunks(cfg)
    H = cfg.hidden
    base = _gates_off(cfg, ids)
    for i in range(cfg.n_single):
        np.testing.assert_array_equal(dit.single_block(P, i, x, base), x)
        m = _set(base, ids[("single", i, "gate")], H, 0.7)
        a = dit.single_block(P, i, x, m)
        assert np.max(np.abs(a - x)) > 1e-3
        # the other block's chunks do not reach block i
        j = 1 - i
        b = dit.single_block(P, i, x, _set(m, ids[("single", j, "shift")], H, 3.0))
        np.testing.assert_array_equal(a, b)
        c = dit.single_block(P, i, x, _set(m, ids[("single", i, "shift")], H, 3.0))
        assert np.max(np.abs(a - c)) > 1e-3


def test_cross_block_chunk_roles():
    """Video blocks read the shared 6H chunk plus their own offset: a shift
    of the shared gate1 chunk by s equals the same shift of the offset."""
    cfg = NANO_CROSS
    w, _, _ = inputs(cfg, seed=29)
    P = dit.Params(cfg, w.tensors)
    rng = np.random.default_rng(8)
    x = P.rs(rng.standard_normal((cfg.n_img, cfg.hidden)))
    ctx = P.rs(rng.standard_normal((cfg.n_txt, cfg.hidden)))
    ids = header_chunks(cfg)
    H = cfg.hidden
    mod = rng.standard_normal(cfg.n_mod) * 0.3
    k = ids[("cross_shared", "gate1")]
    a = dit.cross_block(P, 1, x, ctx, _set(mod, k, H, mod[k * H:(k + 1) * H] + 0.25))
    off = w.tensors["cross.1.mod_offset"]
    saved = off.copy()
    off[2 * H:3 * H] = (off[2 * H:3 * H].astype(np.float64) + 0.25).astype(off.dtype)
    try:
        b = dit.cross_block(P, 1, x, ctx, mod)
    finally:
        off[...] = saved
    np.testing.assert_allclose(a, b, rtol=1e-6, atol=1e-6)
    # gate1 = gate2 = 0 in shared + offset: only the ungated cross-attention acts
    m = mod.copy()
    for g in ("gate1", "gate2"):
        kk = ids[("cross_shared", g)]
        j = 2 if g == "gate1" else 5
        m[kk * H:(kk + 1) * H] = -P("cross.1.mod_offset")[j * H:(j + 1) * H]
    y = dit.cross_block(P, 1, x, ctx, m)
    ctx2 = ctx * 1.5
    y2 = dit.cross_block(P, 1, x, ctx2, m)
    assert np.max(np.abs(y - y2)) > 1e-4          # the text still reaches x
