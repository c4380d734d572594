"""Pins of the oracle's numeric primitives against independent library routines."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import dit
from oracle.numerics import round_bf16, round_f32, storage_to_f64

RNG = np.random.default_rng(1234)


def test_round_bf16_matches_torch_on_float32_inputs():
    x = np.concatenate([RNG.standard_normal(20000) * s for s in (1e-3, 0.02, 1.0, 37.0, 1e4)])
    x32 = x.astype(np.float32)
    ref = torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(round_bf16(x32.astype(np.float64)), ref)


@pytest.mark.parametrize("x,expect", [
    (1.0 + 2.0 ** -8, 1.0),                       # tie -> even (1.0)
    (1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -6),       # tie -> even (upper)
    (1.0 + 2.0 ** -8 + 2.0 ** -30, 1.0 + 2.0 ** -7),  # just above the tie
    (-(1.0 + 2.0 ** -8), -1.0),
    (3.0 * 2.0 ** 20, 3.0 * 2.0 ** 20),
    (0.0, 0.0),
])
def test_round_bf16_ties(x, expect):
    assert round_bf16(np.array([x]))[0] == expect


def test_round_bf16_from_float64_is_single_rounding():
    # 1 + 2^-8 + 2^-40 is above the bf16 tie, but float32 rounds it to the tie
    # itself: a two-step rounding would give 1.0, the direct one 1 + 2^-7.
    x = 1.0 + 2.0 ** -8 + 2.0 ** -40
    assert float(np.float32(x)) == 1.0 + 2.0 ** -8
    assert round_bf16(np.array([x]))[0] == 1.0 + 2.0 ** -7


def test_round_f32_and_bits_decode():
    x = RNG.standard_normal(100)
    np.testing.assert_array_equal(round_f32(x), x.astype(np.float32).astype(np.float64))
    bits = np.array([0x3F80, 0xBF80, 0x4049, 0x0000], np.uint16)
    np.testing.assert_array_equal(storage_to_f64(bits, "bf16"), [1.0, -1.0, 3.140625, 0.0])


def test_layer_norm_vs_torch():
    x = RNG.standard_normal((7, 96)) * 3 + 0.5
    ref = F.layer_norm(torch.from_numpy(x), (96,), eps=1e-6).numpy()
    np.testing.assert_allclose(dit.layer_norm(x), ref, rtol=1e-12, atol=1e-12)


def test_modulate_reduces_to_layer_norm():
    x = RNG.standard_normal((5, 32))
    z = np.zeros(32)
    np.testing.assert_array_equal(dit.modulate(x, z, z), dit.layer_norm(x))
    sh, sc = RNG.standard_normal(32), RNG.standard_normal(32)
    ref = F.layer_norm(torch.from_numpy(x), (32,), eps=1e-6).numpy() * (1 + sc) + sh
    np.testing.assert_allclose(dit.modulate(x, sh, sc), ref, rtol=1e-12, atol=1e-12)


def test_rms_heads_vs_torch():
    x = RNG.standard_normal((6, 4 * 32))
    ref = F.rms_norm(torch.from_numpy(x).reshape(6, 4, 32), (32,), eps=1e-6).reshape(6, 128).numpy()
    np.testing.assert_allclose(dit.rms_heads(x, 4, 32), ref, rtol=1e-12, atol=1e-12)


def test_gelu_and_silu_vs_torch():
    x = np.linspace(-8, 8, 1001)
    np.testing.assert_allclose(dit.gelu_tanh(x), F.gelu(torch.from_numpy(x), approximate="tanh").numpy(),
                               rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(dit.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("lq,lk", [(9, 9), (5, 13), (33, 7)])
def test_attention_vs_torch_sdpa(lq, lk):
    heads, d = 3, 16
    q, k, v = (RNG.standard_normal((n, heads * d)) for n in (lq, lk, lk))
    ref = F.scaled_dot_product_attention(
        torch.from_numpy(q).reshape(lq, heads, d).transpose(0, 1),
        torch.from_numpy(k).reshape(lk, heads, d).transpose(0, 1),
        torch.from_numpy(v).reshape(lk, heads, d).transpose(0, 1)).transpose(0, 1).reshape(lq, heads * d)
    np.testing.assert_allclose(dit.attention(q, k, v, heads, d, q_chunk=4), ref.numpy(), rtol=1e-10, atol=1e-12)


def test_timestep_embedding_closed_forms():
    e0 = dit.timestep_embedding(np.array([0.0]), 256)[0]
    np.testing.assert_array_equal(e0[:128], 1.0)
    np.testing.assert_array_equal(e0[128:], 0.0)
    sig = np.array([0.37, 0.9])
    e = dit.timestep_embedding(sig, 256)
    np.testing.assert_allclose(e[:, :128] ** 2 + e[:, 128:] ** 2, 1.0, atol=1e-14)
    # k = 0 has frequency 1 and k = 64 has 10000^-1/2 = 0.01
    np.testing.assert_allclose(e[:, 0], np.cos(1000 * sig), atol=1e-12)
    np.testing.assert_allclose(e[:, 128 + 64], np.sin(10 * sig), atol=1e-12)
