"""Block-level pins of the oracle: scalar brute force on tiny shapes and
structural invariants.  The brute force below walks explicit indices with
plain Python floats, so a transposed weight, a wrong split offset or a
wrong head slice in the vectorised oracle shows up as a mismatch."""
import math

import numpy as np
import pytest

from oracle import dit
from tests._nano import NANO, NANO_BF16, NANO_CROSS, inputs


# ------------------------------------------------------------ scalar helpers

def lin(x, W, b):  # x [n][k], W [o][k]
    return [[sum(x[i][kk] * W[o][kk] for kk in range(len(x[i]))) + b[o] for o in range(len(W))]
            for i in range(len(x))]


def ln_row(r):
    mu = sum(r) / len(r)
    var = sum((v - mu) ** 2 for v in r) / len(r)
    return [(v - mu) / math.sqrt(var + 1e-6) for v in r]


def mod_rows(x, sh, sc):
    return [[v * (1 + sc[j]) + sh[j] for j, v in enumerate(ln_row(r))] for r in x]


def rms_row(r, heads, d):
    out = []
    for h in range(heads):
        s = r[h * d:(h + 1) * d]
        m = math.sqrt(sum(v * v for v in s) / d + 1e-6)
        out += [v / m for v in s]
    return out


def gelu(v):
    return 0.5 * v * (1 + math.tanh(math.sqrt(2 / math.pi) * (v + 0.044715 * v ** 3)))


def attn(q, k, v, heads, d):
    out = [[0.0] * (heads * d) for _ in q]
    for h in range(heads):
        for i in range(len(q)):
            s = [sum(q[i][h * d + e] * k[j][h * d + e] for e in range(d)) / math.sqrt(d) for j in range(len(k))]
            mx = max(s)
            p = [math.exp(v_ - mx) for v_ in s]
            z = sum(p)
            for e in range(d):
                out[i][h * d + e] = sum(p[j] * v[j][h * d + e] for j in range(len(k))) / z
    return out


def rsm(P, rows):
    return P.rs(np.array(rows)).tolist()


def W(P, name):
    return P(name).tolist()


def split_qkv(P, y, H, cfg):
    q = rsm(P, [rms_row(r[:H], cfg.heads, cfg.head_dim) for r in y])
    k = rsm(P, [rms_row(r[H:2 * H], cfg.heads, cfg.head_dim) for r in y])
    v = rsm(P, [r[2 * H:3 * H] for r in y])
    return q, k, v


def brute_double(P, i, s_img, s_txt, mod):
    cfg, H = P.cfg, P.cfg.hidden
    base = {"img": 12 * H * i, "txt": 12 * H * i + 6 * H}
    st = {"img": s_img.tolist(), "txt": s_txt.tolist()}
    ch = {k: [mod[base[k] + j * H: base[k] + (j + 1) * H].tolist() for j in range(6)] for k in st}
    qkv = {}
    for k in st:
        a = rsm(P, mod_rows(st[k], ch[k][0], ch[k][1]))
        y = lin(a, W(P, f"double.{i}.{k}.qkv.w"), W(P, f"double.{i}.{k}.qkv.b"))
        qkv[k] = split_qkv(P, y, H, cfg)
    q = qkv["txt"][0] + qkv["img"][0]
    kk = qkv["txt"][1] + qkv["img"][1]
    v = qkv["txt"][2] + qkv["img"][2]
    o = rsm(P, attn(q, kk, v, cfg.heads, cfg.head_dim))
    nt = len(st["txt"])
    os_ = {"txt": o[:nt], "img": o[nt:]}
    out = {}
    for k in st:
        sh1, sc1, g1, sh2, sc2, g2 = ch[k]
        p = f"double.{i}.{k}."
        y = lin(os_[k], W(P, p + "o.w"), W(P, p + "o.b"))
        s = rsm(P, [[st[k][r][j] + g1[j] * y[r][j] for j in range(H)] for r in range(len(y))])
        a2 = rsm(P, mod_rows(s, sh2, sc2))
        u = rsm(P, [[gelu(v_) for v_ in r] for r in lin(a2, W(P, p + "mlp0.w"), W(P, p + "mlp0.b"))])
        y2 = lin(u, W(P, p + "mlp1.w"), W(P, p + "mlp1.b"))
        out[k] = rsm(P, [[s[r][j] + g2[j] * y2[r][j] for j in range(H)] for r in range(len(s))])
    return np.array(out["img"]), np.array(out["txt"])


def brute_single(P, i, x, mod):
    cfg, H = P.cfg, P.cfg.hidden
    base = 12 * H * cfg.n_double + 3 * H * i
    sh, sc, g = (mod[base + j * H: base + (j + 1) * H].tolist() for j in range(3))
    xl = x.tolist()
    a = rsm(P, mod_rows(xl, sh, sc))
    y = lin(a, W(P, f"single.{i}.l1.w"), W(P, f"single.{i}.l1.b"))
    q, k, v = split_qkv(P, y, H, cfg)
    u = rsm(P, [[gelu(v_) for v_ in r[3 * H:]] for r in y])
    o = rsm(P, attn(q, k, v, cfg.heads, cfg.head_dim))
    cat = [o[r] + u[r] for r in range(len(o))]
    y2 = lin(cat, W(P, f"single.{i}.l2.w"), W(P, f"single.{i}.l2.b"))
    return np.array(rsm(P, [[xl[r][j] + g[j] * y2[r][j] for j in range(H)] for r in range(len(xl))]))


def brute_cross(P, i, x, ctx, mod):
    cfg, H = P.cfg, P.cfg.hidden
    base = 12 * H * cfg.n_double + 3 * H * cfg.n_single
    off = P(f"cross.{i}.mod_offset")
    e = [[mod[base + j * H + c] + off[j * H + c] for c in range(H)] for j in range(6)]
    sh1, sc1, g1, sh2, sc2, g2 = e
    p = f"cross.{i}."
    xl = x.tolist()
    a = rsm(P, mod_rows(xl, sh1, sc1))
    q, k, v = split_qkv(P, lin(a, W(P, p + "qkv.w"), W(P, p + "qkv.b")), H, cfg)
    o = rsm(P, attn(q, k, v, cfg.heads, cfg.head_dim))
    y = lin(o, W(P, p + "o.w"), W(P, p + "o.b"))
    xl = rsm(P, [[xl[r][j] + g1[j] * y[r][j] for j in range(H)] for r in range(len(xl))])
    c = rsm(P, [ln_row(r) for r in xl])
    q2 = rsm(P, [rms_row(r, cfg.heads, cfg.head_dim) for r in lin(c, W(P, p + "xq.w"), W(P, p + "xq.b"))])
    kv = lin(ctx.tolist(), W(P, p + "xkv.w"), W(P, p + "xkv.b"))
    k2 = rsm(P, [rms_row(r[:H], cfg.heads, cfg.head_dim) for r in kv])
    v2 = rsm(P, [r[H:] for r in kv])
    o2 = rsm(P, attn(q2, k2, v2, cfg.heads, cfg.head_dim))
    y2 = lin(o2, W(P, p + "xo.w"), W(P, p + "xo.b"))
    xl = rsm(P, [[xl[r][j] + y2[r][j] for j in range(H)] for r in range(len(xl))])
    a3 = rsm(P, mod_rows(xl, sh2, sc2))
    u = rsm(P, [[gelu(v_) for v_ in r] for r in lin(a3, W(P, p + "ffn0.w"), W(P, p + "ffn0.b"))])
    y3 = lin(u, W(P, p + "ffn1.w"), W(P, p + "ffn1.b"))
    return np.array(rsm(P, [[xl[r][j] + g2[j] * y3[r][j] for j in range(H)] for r in range(len(xl))]))


def setup(cfg, seed=3):
    w, x, text = inputs(cfg, seed)
    P = dit.Params(cfg, w.tensors)
    rng = np.random.default_rng(seed)
    mod = rng.standard_normal(cfg.n_mod) * 0.5
    h = P.rs(rng.standard_normal((cfg.n_img, cfg.hidden)))
    txt = P.rs(rng.standard_normal((cfg.n_txt, cfg.hidden)))
    return P, mod, h, txt


@pytest.mark.parametrize("cfg", [NANO, NANO_BF16], ids=lambda c: c.name)
def test_double_block_vs_scalar_bruteforce(cfg):
    P, mod, h, txt = setup(cfg)
    a_img, a_txt = dit.double_block(P, 0, h, txt, mod)
    b_img, b_txt = brute_double(P, 0, h, txt, mod)
    tol = 1e-12 if cfg.dtype == "f32" else 0
    if cfg.dtype == "f32":
        np.testing.assert_allclose(a_img, b_img, rtol=1e-6, atol=1e-6)
        np.testing.assert_allclose(a_txt, b_txt, rtol=1e-6, atol=1e-6)
    else:
        # the same bf16 roundings: values agree except for rare 1-ulp flips
        assert np.mean(np.abs(a_img - b_img) <= np.abs(b_img) * 2 ** -7 + tol) > 0.99
        assert np.mean(np.abs(a_txt - b_txt) <= np.abs(b_txt) * 2 ** -7 + tol) > 0.99


@pytest.mark.parametrize("cfg", [NANO, NANO_BF16], ids=lambda c: c.name)
def test_single_block_vs_scalar_bruteforce(cfg):
    P, mod, h, txt = setup(cfg)
    x = np.concatenate([txt, h])
    a = dit.single_block(P, 0, x, mod)
    b = brute_single(P, 0, x, mod)
    if cfg.dtype == "f32":
        np.testing.assert_allclose(a, b, rtol=1e-6, atol=1e-6)
    else:
        assert np.mean(np.abs(a - b) <= np.abs(b) * 2 ** -7) > 0.99


def test_cross_block_vs_scalar_bruteforce():
    cfg = NANO_CROSS
    P, mod, h, txt = setup(cfg)
    a = dit.cross_block(P, 1, h, txt, mod)
    b = brute_cross(P, 1, h, txt, mod)
    np.testing.assert_allclose(a, b, rtol=1e-6, atol=1e-6)


def _zero_gates(cfg, mod):
    H = cfg.hidden
    mod = mod.copy()
    off = dit.mod_offsets(cfg)
    for i in range(cfg.n_double):
        for st in ("img", "txt"):
            b = off[("double", i, st)]
            mod[b + 2 * H: b + 3 * H] = 0
            mod[b + 5 * H: b + 6 * H] = 0
    for i in range(cfg.n_single):
        b = off[("single", i)]
        mod[b + 2 * H: b + 3 * H] = 0
    return mod


def test_zero_gate_blocks_are_identity():
    cfg = NANO
    P, mod, h, txt = setup(cfg)
    mz = _zero_gates(cfg, mod)
    a_img, a_txt = dit.double_block(P, 0, h, txt, mz)
    np.testing.assert_array_equal(a_img, h)
    np.testing.assert_array_equal(a_txt, txt)
    x = np.concatenate([txt, h])
    np.testing.assert_array_equal(dit.single_block(P, 0, x, mz), x)


def test_image_token_permutation_equivariance():
    cfg = NANO
    P, mod, h, txt = setup(cfg)
    perm = np.random.default_rng(0).permutation(cfg.n_img)
    out = dit.block_stack(P, h, txt, mod)
    out_p = dit.block_stack(P, h[perm], txt, mod)
    np.testing.assert_allclose(out_p, out[perm], rtol=1e-9, atol=1e-9)


def test_text_tokens_change_image_rows():
    """Joint attention: text reaches the image stream."""
    cfg = NANO
    P, mod, h, txt = setup(cfg)
    out = dit.block_stack(P, h, txt, mod)
    out2 = dit.block_stack(P, h, txt[::-1] * 2, mod)
    assert np.max(np.abs(out - out2)) > 1e-6
