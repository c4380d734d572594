"""dit_attention_bf16_noalloc (the allocation-free attention entry point)
against dit_attention_bf16 with a caller-owned workspace: same kernels, so
the outputs must be bit-identical.  Two calls in a row on one device, the
second with fewer keys and queries than the first (the shared device array
keeps the first call's contents), both value-checked against the oracle's
attention on sampled rows; sizes beyond the limit are rejected on the host."""
import numpy as np
import pytest

from oracle import dit
from oracle.numerics import round_bf16
from paper_2608_09231_amd import binding
from tests._gpu import dev, host_bf16, rel_l2, torch_cuda

pytestmark = pytest.mark.gpu

RNG = np.random.default_rng(2024)


def bf16_bits(x):
    return (round_bf16(x).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


def bits_to_f64(b):
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def case(torch, L, heads, bounded):
    H = heads * 128

    def mk(norm):
        x = RNG.standard_normal((L, H)) * 2.0
        if norm:
            x = dit.rms_heads(x, heads, 128)
        b = bf16_bits(x)
        return b, bits_to_f64(b)
    (q_b, q), (k_b, k), (v_b, v) = mk(bounded), mk(bounded), mk(False)
    flags = binding.ATTN_BOUNDED_LOGITS if bounded else 0
    qd, kd, vd = dev(torch, q_b), dev(torch, k_b), dev(torch, v_b)
    o_ref = torch.zeros((L, H), dtype=torch.int16, device="cuda")
    ws = torch.zeros(heads * 128 * ((L + 63) // 64 * 64), dtype=torch.int16, device="cuda")
    binding.attention_bf16(qd, kd, vd, o_ref, Lq=L, Lk=L, heads=heads, ldq=H, ldk=H, ldv=H, ldo=H,
                           vt_ws=ws, flags=flags)
    o = torch.full((L, H), 0x7fc0, dtype=torch.int16, device="cuda")    # NaN pattern: every row written
    binding.attention_bf16_noalloc(qd, kd, vd, o, Lq=L, Lk=L, heads=heads, ldq=H, ldk=H, ldv=H, ldo=H,
                                   flags=flags)
    torch.cuda.synchronize()
    got = host_bf16(o)
    np.testing.assert_array_equal(o.cpu().numpy(), o_ref.cpu().numpy())
    rows = np.sort(RNG.choice(L, min(L, 48), replace=False))
    ref = round_bf16(dit.attention(q[rows], k, v, heads, 128))
    assert rel_l2(got[rows], ref) < 4e-3
    return got


def test_noalloc_attention_two_calls_shrinking():
    torch = torch_cuda()
    print("noalloc attention: L=4608 heads=24 (FLUX-1024 joint sequence), bounded", flush=True)
    case(torch, 4608, 24, True)
    print("noalloc attention: L=777 heads=3, unbounded", flush=True)
    case(torch, 777, 3, False)


def test_noalloc_attention_rejects_oversized():
    torch = torch_cuda()
    H = 24 * 128
    t = torch.zeros((8, H), dtype=torch.int16, device="cuda")
    with pytest.raises(binding.DitError) as e:
        binding.attention_bf16_noalloc(t, t, t, t, Lq=8, Lk=5441, heads=24, ldq=H, ldk=H, ldv=H, ldo=H)
    assert e.value.status == binding.DIT_ESHAPE
    assert "allocation-free limit" in str(e.value)
