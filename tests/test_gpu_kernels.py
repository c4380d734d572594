"""GPU parity of the full-step kernels (bf16 GEMM with its epilogues, flash
attention) against the oracle's primitives, through the C ABI.

Small shapes span several tiles and a ragged tail in every dimension; the
workload-sized cases run the exact launch shapes of the FLUX-1024 step and
compare sampled outputs computed one by one in float64."""
import numpy as np
import pytest

from oracle import dit
from oracle.numerics import round_bf16
from paper_2608_09231_amd import binding
from tests._gpu import assert_bf16_close, dev, host_bf16, rel_l2, torch_cuda

pytestmark = pytest.mark.gpu

RNG = np.random.default_rng(2024)


def bf16_bits(x):
    """float64 -> bf16 bit patterns of round_bf16(x) (exact)."""
    r = round_bf16(x).astype(np.float32)
    return (r.view(np.uint32) >> 16).astype(np.uint16)


def bits_to_f64(b):
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def make(shape, scale=1.0):
    b = bf16_bits(RNG.standard_normal(shape) * scale)
    return b, bits_to_f64(b)


@pytest.mark.parametrize("M,N,K", [(300, 392, 200), (37, 136, 64), (1, 8, 8), (513, 256, 3072)])
def test_gemm_store_and_bias(M, N, K):
    torch = torch_cuda()
    a_b, a = make((M, K))
    w_b, w = make((N, K), 0.05)
    b_b, b = make((N,), 0.1)
    out = torch.zeros((M, N), dtype=torch.int16, device="cuda")
    binding.gemm_bf16(dev(torch, a_b), dev(torch, w_b), dev(torch, b_b), out, M=M, N=N, K=K)
    assert_bf16_close(host_bf16(out), round_bf16(a @ w.T + b))


def test_gemm_epilogues_gelu_silu_f32():
    torch = torch_cuda()
    M, N, K = 260, 300, 136
    a_b, a = make((M, K))
    w_b, w = make((N, K), 0.1)
    b_b, b = make((N,), 0.1)
    y = a @ w.T + b
    out = torch.zeros((M, N), dtype=torch.int16, device="cuda")
    binding.gemm_bf16(dev(torch, a_b), dev(torch, w_b), dev(torch, b_b), out, M=M, N=N, K=K, gelu_from=100)
    ref = round_bf16(np.concatenate([y[:, :100], dit.gelu_tanh(y[:, 100:])], axis=1))
    assert_bf16_close(host_bf16(out), ref)
    binding.gemm_bf16(dev(torch, a_b), dev(torch, w_b), dev(torch, b_b), out, M=M, N=N, K=K,
                      flags=binding.EPI_SILU)
    assert_bf16_close(host_bf16(out), round_bf16(dit.silu(y)))
    of = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    binding.gemm_bf16(dev(torch, a_b), dev(torch, w_b), dev(torch, b_b), of, M=M, N=N, K=K,
                      flags=binding.EPI_F32)
    np.testing.assert_allclose(of.cpu().numpy(), y, rtol=1e-5, atol=1e-5)


def test_gemm_qkv_rms_and_gated_residual():
    torch = torch_cuda()
    M, H = 203, 256
    N, K = 3 * H + 512, H
    a_b, a = make((M, K))
    w_b, w = make((N, K), 0.05)
    b_b, b = make((N,), 0.1)
    y = a @ w.T + b
    ld = 4 * H + 512
    out = torch.zeros((M, ld), dtype=torch.int16, device="cuda")
    binding.gemm_bf16(dev(torch, a_b), dev(torch, w_b), dev(torch, b_b), out, M=M, N=N, K=K, ldc=ld,
                      rms_cols=2 * H, gelu_from=3 * H, gap_at=3 * H, gap=H)
    got = host_bf16(out)
    assert_bf16_close(got[:, :2 * H], round_bf16(dit.rms_heads(y[:, :2 * H], 2 * H // 128, 128)))
    assert_bf16_close(got[:, 2 * H:3 * H], round_bf16(y[:, 2 * H:3 * H]))
    assert_bf16_close(got[:, 4 * H:], round_bf16(dit.gelu_tanh(y[:, 3 * H:])))
    assert np.all(got[:, 3 * H:4 * H] == 0)          # the hole is left untouched
    # gated residual in place: C = S(C + g * (A W^T + b))
    N2 = H
    w2_b, w2 = make((N2, K), 0.05)
    b2_b, b2 = make((N2,), 0.1)
    c0_b, c0 = make((M, N2))
    g = RNG.standard_normal(N2).astype(np.float32)
    cbuf = dev(torch, c0_b)
    binding.gemm_bf16(dev(torch, a_b), dev(torch, w2_b), dev(torch, b2_b), cbuf, M=M, N=N2, K=K,
                      flags=binding.EPI_GATED_RES, gate=dev(torch, g))
    ref = round_bf16(c0 + g.astype(np.float64) * (a @ w2.T + b2))
    assert_bf16_close(host_bf16(cbuf), ref)


@pytest.mark.parametrize("gated", [False, True])
def test_gemm_ring_pipeline_ragged(gated):
    """256 x 256 tiles with the five-slice LDS ring (chosen for this shape:
    one full wave of 16 x 16 tiles), ragged M and N, K = 320 = five 64-deep
    slices (prologue, steady slices and the peeled tail); plain and gated
    residual epilogues against float64."""
    torch = torch_cuda()
    M, N, K = 3999, 3992, 320
    a_b, a = make((M, K))
    w_b, w = make((N, K), 0.05)
    b_b, b = make((N,), 0.1)
    y = a @ w.T + b
    if not gated:
        out = torch.zeros((M, N), dtype=torch.int16, device="cuda")
        binding.gemm_bf16(dev(torch, a_b), dev(torch, w_b), dev(torch, b_b), out, M=M, N=N, K=K)
        assert_bf16_close(host_bf16(out), round_bf16(y))
    else:
        c0_b, c0 = make((M, N))
        g = RNG.standard_normal(N).astype(np.float32)
        cbuf = dev(torch, c0_b)
        binding.gemm_bf16(dev(torch, a_b), dev(torch, w_b), dev(torch, b_b), cbuf, M=M, N=N, K=K,
                          flags=binding.EPI_GATED_RES, gate=dev(torch, g))
        assert_bf16_close(host_bf16(cbuf), round_bf16(c0 + g.astype(np.float64) * y))


def test_gemm_ring_rms_gelu_gap_ragged():
    """The ring kernel's store epilogue with the single-block projection's
    column roles at a ragged M: per-head RMS on the first 2 H columns, GELU
    on the MLP half, written past a hole of H columns."""
    torch = torch_cuda()
    M, H, F, K = 3999, 1024, 1024, 320
    N, ld = 3 * H + F, 4 * H + F
    a_b, a = make((M, K))
    w_b, w = make((N, K), 0.05)
    b_b, b = make((N,), 0.1)
    y = a @ w.T + b
    out = torch.zeros((M, ld), dtype=torch.int16, device="cuda")
    binding.gemm_bf16(dev(torch, a_b), dev(torch, w_b), dev(torch, b_b), out, M=M, N=N, K=K, ldc=ld,
                      rms_cols=2 * H, gelu_from=3 * H, gap_at=3 * H, gap=H)
    got = host_bf16(out)
    assert_bf16_close(got[:, :2 * H], round_bf16(dit.rms_heads(y[:, :2 * H], 2 * H // 128, 128)))
    assert_bf16_close(got[:, 2 * H:3 * H], round_bf16(y[:, 2 * H:3 * H]))
    assert_bf16_close(got[:, 4 * H:], round_bf16(dit.gelu_tanh(y[:, 3 * H:])))
    assert np.all(got[:, 3 * H:4 * H] == 0)


def attn_case(torch, Lq, Lk, heads, sample_rows=None):
    H = heads * 128
    q_b, q = make((Lq, H))
    k_b, k = make((Lk, H))
    v_b, v = make((Lk, H))
    o = torch.zeros((Lq, H), dtype=torch.int16, device="cuda")
    ws = torch.zeros(heads * 128 * ((Lk + 63) // 64 * 64), dtype=torch.int16, device="cuda")
    binding.attention_bf16(dev(torch, q_b), dev(torch, k_b), dev(torch, v_b), o, Lq=Lq, Lk=Lk, heads=heads,
                           ldq=H, ldk=H, ldv=H, ldo=H, vt_ws=ws)
    got = host_bf16(o)
    rows = np.arange(Lq) if sample_rows is None else sample_rows
    ref = round_bf16(dit.attention(q[rows], k, v, heads, 128))
    return got[rows], ref


@pytest.mark.parametrize("Lq,Lk,heads", [(200, 200, 2), (130, 33, 1), (1, 1, 1), (64, 300, 3)])
def test_attention_small_ragged(Lq, Lk, heads):
    torch = torch_cuda()
    got, ref = attn_case(torch, Lq, Lk, heads)
    assert rel_l2(got, ref) < 4e-3
    assert np.max(np.abs(got - ref)) <= 3 * 2.0 ** -8 * np.max(np.abs(ref))


def test_attention_flux1024_joint_shape_sampled():
    """FLUX-1024 joint attention: 4608 tokens, 24 heads; 96 sampled queries."""
    torch = torch_cuda()
    L, heads = 4096 + 512, 24
    rows = np.sort(RNG.choice(L, 96, replace=False))
    got, ref = attn_case(torch, L, L, heads, rows)
    assert rel_l2(got, ref) < 4e-3


def test_gemm_flux1024_single_block_shape_sampled():
    """Single-block input projection of FLUX-1024: [4608 x 3072] x [21504 x 3072]^T
    with the fused RMS / GELU / gap epilogue; 2048 sampled outputs per region."""
    torch = torch_cuda()
    M, H, F = 4608, 3072, 12288
    N, K = 3 * H + F, H
    a_b = bf16_bits(RNG.standard_normal((M, K)))
    w_b = bf16_bits(RNG.standard_normal((N, K)) * 0.02)
    b_b = bf16_bits(RNG.standard_normal(N) * 0.02)
    ld = 4 * H + F
    out = torch.zeros((M, ld), dtype=torch.int16, device="cuda")
    binding.gemm_bf16(dev(torch, a_b), dev(torch, w_b), dev(torch, b_b), out, M=M, N=N, K=K, ldc=ld,
                      rms_cols=2 * H, gelu_from=3 * H, gap_at=3 * H, gap=H)
    got = host_bf16(out)
    a, w, b = bits_to_f64(a_b), bits_to_f64(w_b), bits_to_f64(b_b)
    rows = RNG.choice(M, 16, replace=False)
    # q/k heads need the whole head row for the RMS norm: sample rows x heads
    for r in rows:
        y = a[r] @ w.T + b
        qk = round_bf16(dit.rms_heads(y[None, :2 * H], 2 * H // 128, 128))[0]
        assert_bf16_close(got[r, :2 * H], qk, frac_exact=0.8)
        assert_bf16_close(got[r, 2 * H:3 * H], round_bf16(y[2 * H:3 * H]), frac_exact=0.8)
        assert_bf16_close(got[r, 4 * H:], round_bf16(dit.gelu_tanh(y[3 * H:])), frac_exact=0.8)


@pytest.mark.parametrize("L,heads", [(4608, 24), (333, 2)])
def test_attention_bounded_logits_rms_normalised(L, heads):
    """The sampler's path: q and k leave a unit-gain RMS norm, so the kernel
    may replace the running max by a fixed shift (DIT_ATTN_BOUNDED_LOGITS)."""
    torch = torch_cuda()
    H = heads * 128
    def mk(n, norm):
        x = RNG.standard_normal((n, H)) * 3.0
        if norm:
            x = dit.rms_heads(x, heads, 128)
        b = bf16_bits(x)
        return b, bits_to_f64(b)
    q_b, q = mk(L, True)
    k_b, k = mk(L, True)
    v_b, v = mk(L, False)
    o = torch.zeros((L, H), dtype=torch.int16, device="cuda")
    ws = torch.zeros(heads * 128 * ((L + 63) // 64 * 64), dtype=torch.int16, device="cuda")
    binding.attention_bf16(dev(torch, q_b), dev(torch, k_b), dev(torch, v_b), o, Lq=L, Lk=L, heads=heads,
                           ldq=H, ldk=H, ldv=H, ldo=H, vt_ws=ws, flags=binding.ATTN_BOUNDED_LOGITS)
    got = host_bf16(o)
    rows = np.sort(RNG.choice(L, min(L, 64), replace=False))
    ref = round_bf16(dit.attention(q[rows], k, v, heads, 128))
    assert rel_l2(got[rows], ref) < 4e-3
