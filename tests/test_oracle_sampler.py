"""Whole-sampler pins of the oracle: closed forms, brute-force re-derivations
and invariants of Alg. 2 with plain residual reuse."""
import dataclasses

import numpy as np
import pytest

from oracle import dit, sample, sigma_schedule
from oracle.numerics import round_f32, storage_to_f64
from paper_2608_09231_amd import synth
from tests._nano import NANO, NANO_BF16, NANO_CFG, NANO_CROSS, inputs


def gate_for(cfg, seed=1):
    return synth.make_gate_blob((8, 32, 16, 1), seed=seed)


def const_gate(z):
    return lambda f: z


def test_sigma_schedule_closed_forms():
    s = sigma_schedule(10, 1.0)
    np.testing.assert_allclose(s, 1 - np.arange(11) / 10, atol=1e-15)
    s3 = sigma_schedule(28, 3.0)
    assert s3[0] == 1.0 and s3[-1] == 0.0
    assert np.all(np.diff(s3) < 0)
    u = 0.5
    assert np.isclose(sigma_schedule(2, 3.0)[1], 3 * u / (1 + 2 * u))


@pytest.mark.parametrize("cfg", [NANO, NANO_CROSS], ids=lambda c: c.name)
def test_zero_dit_closed_form(cfg):
    """All weights 0 except b_out: h = 0, r = 0, v = b_out, so
    x_T = x_0 + sum_t f32(dsigma_t) b_out  (= x_0 - b_out up to f32)."""
    w, x0, text = inputs(cfg)
    for k, v in w.tensors.items():
        v[...] = 0
    bout = np.linspace(-1, 1, cfg.in_channels).astype(np.float32)
    w.tensors["final.b"][...] = bout
    T, B = 9, 4
    res = sample(cfg, w.tensors, gate_for(cfg), x0, text, T, B, shift=3.0)
    sig = sigma_schedule(T, 3.0)
    x = x0.astype(np.float64)
    for t in range(T):
        x = round_f32(x + float(np.float32(sig[t + 1] - sig[t])) * bout.astype(np.float64))
    np.testing.assert_array_equal(res.x, x)
    np.testing.assert_allclose(res.x, x0 - bout, atol=1e-6)
    assert res.nfe == B
    # every indicator tensor is 0, so both relative distances are 0
    assert np.all(res.features[1:, 4:6] == 0)


def uncached_euler(cfg, w, x0, text, T, shift):
    """Plain Euler flow-matching sampler with a network call every step."""
    P = dit.Params(cfg, w.tensors)
    sig = sigma_schedule(T, shift)
    t64 = storage_to_f64(text[0], cfg.dtype)
    txt = dit.text_in(P, t64)
    mods = dit.mod_table(P, dit.vec_table(P, sig[:T], t64))
    x = round_f32(x0.astype(np.float64))
    for t in range(T):
        h = dit.patch_embed(P, x)
        v = dit.final_layer(P, dit.block_stack(P, h, txt, mods[t]), mods[t])
        x = round_f32(x + float(np.float32(sig[t + 1] - sig[t])) * v)
    return x


@pytest.mark.parametrize("cfg", [NANO, NANO_BF16, NANO_CROSS], ids=lambda c: c.name)
def test_full_budget_equals_uncached_sampler(cfg):
    w, x0, text = inputs(cfg)
    T = 6
    res = sample(cfg, w.tensors, gate_for(cfg), x0, text, T, T, shift=3.0)
    assert list(res.full) == [1] * T
    np.testing.assert_array_equal(res.x, uncached_euler(cfg, w, x0, text, T, 3.0))


def test_budget_one_brute_force():
    """B = 1: x_T = x_0 + sum_t dsigma_t Final(S(h_t + r_0)), r_0 from step 0."""
    cfg = NANO
    w, x0, text = inputs(cfg)
    T = 7
    res = sample(cfg, w.tensors, gate_for(cfg), x0, text, T, 1, shift=2.0)
    assert list(res.full) == [1] + [0] * (T - 1)
    P = dit.Params(cfg, w.tensors)
    t64 = storage_to_f64(text[0], cfg.dtype)
    sig = sigma_schedule(T, 2.0)
    txt = dit.text_in(P, t64)
    mods = dit.mod_table(P, dit.vec_table(P, sig[:T], t64))
    x = round_f32(x0.astype(np.float64))
    h0 = dit.patch_embed(P, x)
    r0 = P.rs(dit.block_stack(P, h0, txt, mods[0]) - h0)
    for t in range(T):
        h = dit.patch_embed(P, x)
        h_out = dit.block_stack(P, h, txt, mods[0]) if t == 0 else P.rs(h + r0)
        x = round_f32(x + float(np.float32(sig[t + 1] - sig[t])) * dit.final_layer(P, h_out, mods[t]))
    np.testing.assert_array_equal(res.x, x)


def test_constant_gates_give_closed_form_schedules():
    cfg = NANO
    w, x0, text = inputs(cfg)
    T, B = 10, 5
    pos = sample(cfg, w.tensors, None, x0, text, T, B, gate_fn=const_gate(2.0))
    neg = sample(cfg, w.tensors, None, x0, text, T, B, gate_fn=const_gate(-2.0))
    assert list(pos.full) == [1] * B + [0] * (T - B)
    assert list(neg.full) == [1] + [0] * (T - B) + [1] * (B - 1)
    assert list(neg.forced) == [1] + [0] * (T - B) + [1] * (B - 1)


def test_replay_of_own_schedule_is_bitwise_identical():
    cfg = NANO
    w, x0, text = inputs(cfg)
    T, B = 10, 5
    gated = sample(cfg, w.tensors, gate_for(cfg, 4), x0, text, T, B)
    replay = sample(cfg, w.tensors, gate_for(cfg, 4), x0, text, T, B, forced_mask=gated.full)
    np.testing.assert_array_equal(gated.full, replay.full)
    np.testing.assert_array_equal(gated.x, replay.x)
    np.testing.assert_array_equal(gated.logit[1:], replay.logit[1:])


def test_replay_rejects_invalid_masks():
    cfg = NANO
    w, x0, text = inputs(cfg)
    with pytest.raises(ValueError):
        sample(cfg, w.tensors, gate_for(cfg), x0, text, 5, 2, forced_mask=[0, 1, 1, 0, 0])
    with pytest.raises(ValueError):
        sample(cfg, w.tensors, gate_for(cfg), x0, text, 5, 2, forced_mask=[1, 1, 1, 0, 0])
    with pytest.raises(ValueError):
        sample(cfg, w.tensors, gate_for(cfg), x0, text, 5, 6)
    with pytest.raises(ValueError):
        sample(cfg, w.tensors, gate_for(cfg), x0, text, 5, 0)


def test_features_brute_force_and_reuse_invariant():
    cfg = NANO
    w, x0, text = inputs(cfg)
    T, B = 10, 5
    res = sample(cfg, w.tensors, gate_for(cfg, 2), x0, text, T, B, trace=True)
    ms = [m.ravel().tolist() for m in res.trace["m"]]
    c, t_last, acc = 1, 0, 0.0
    for t in range(1, T):
        def rel(a, b):
            num = sum(abs(x - y) for x, y in zip(a, b))
            den = sum(abs(y) for y in b)
            return num / den
        d_prev = rel(ms[t], ms[t - 1])
        d_last = rel(ms[t], ms[t_last])
        acc += d_prev
        expect = [B / T, (B - c) / B, (B - c) / (T - t), t - t_last, d_last, d_prev, t / T, acc]
        np.testing.assert_allclose(res.features[t], expect, rtol=1e-12, atol=0)
        if t - 1 == t_last:
            assert res.features[t, 4] == res.features[t, 5]
        if res.full[t]:
            c += 1
            t_last = t
            acc = 0.0
        else:
            # reuse keeps the residual cached at the last computed step
            np.testing.assert_array_equal(res.trace["r"][t][0], res.trace["r"][t_last][0])
    assert np.all(np.isnan(res.features[0])) and np.isnan(res.logit[0])


def test_guidance_reduces_to_single_branch():
    """g = 1 follows the conditional branch, g = 0 the unconditional one,
    with the shared schedule taken from the conditional indicator."""
    cfg = NANO_CFG
    w, x0, text = inputs(cfg)
    T, B = 7, 3
    one = dataclasses.replace(cfg, batch=1)
    for g, branch in ((1.0, 0), (0.0, 1)):
        pair = sample(cfg, w.tensors, gate_for(cfg), x0, text, T, B, guidance=g)
        solo = sample(one, w.tensors, gate_for(cfg), x0, text[branch:branch + 1], T, B,
                      forced_mask=pair.full)
        np.testing.assert_array_equal(pair.x, solo.x)
    # the indicator reads the conditional branch: with pooled text the two
    # branches modulate differently, and m_0 (same x_0) matches branch 0 only
    cfg_p = dataclasses.replace(cfg, pooled_text=True)
    wp, x0p, textp = inputs(cfg_p)
    one_p = dataclasses.replace(cfg_p, batch=1)
    pair = sample(cfg_p, wp.tensors, gate_for(cfg), x0p, textp, T, B, guidance=4.0, trace=True)
    cond = sample(one_p, wp.tensors, gate_for(cfg), x0p, textp[:1], T, B, trace=True)
    unc = sample(one_p, wp.tensors, gate_for(cfg), x0p, textp[1:], T, B, trace=True)
    np.testing.assert_array_equal(pair.trace["m"][0], cond.trace["m"][0])
    assert np.max(np.abs(pair.trace["m"][0] - unc.trace["m"][0])) > 0


def test_patch_indicator_option_uses_embedding():
    cfg = NANO
    w, x0, text = inputs(cfg)
    res = sample(cfg, w.tensors, gate_for(cfg), x0, text, 6, 3, indicator="patch", trace=True)
    np.testing.assert_array_equal(res.trace["m"][2], res.trace["h"][2])


def test_tiny_workload_runs_and_spends_budget():
    wl = synth.workload("tiny")
    w, x0, text, gate = synth.make_inputs(wl)
    res = sample(wl.model, w.tensors, gate, x0, text, wl.T, wl.B, shift=wl.shift)
    assert res.nfe == wl.B and res.full[0] == 1
    assert np.all(np.isfinite(res.x))


@pytest.mark.parametrize("cfg", [NANO, NANO_CROSS], ids=lambda c: c.name)
def test_unipc_zero_dit_is_exact(cfg):
    """UniPC integrates the constant velocity b_out exactly: x_T = x_0 - b_out."""
    w, x0, text = inputs(cfg)
    for k, v in w.tensors.items():
        v[...] = 0
    bout = np.linspace(-1, 1, cfg.in_channels).astype(np.float32)
    w.tensors["final.b"][...] = bout
    res = sample(cfg, w.tensors, gate_for(cfg), x0, text, 9, 4, shift=3.0, solver="unipc")
    np.testing.assert_allclose(res.x, x0.astype(np.float64) - bout, atol=2e-6)


@pytest.mark.parametrize("cfg", [NANO, NANO_BF16], ids=lambda c: c.name)
def test_unipc_full_budget_equals_standalone_unipc(cfg):
    """B = T: the sampler's UniPC wiring equals the standalone UniPC loop with a
    network call per step (same f32 storage points)."""
    from oracle.unipc import integrate
    w, x0, text = inputs(cfg)
    T = 7
    res = sample(cfg, w.tensors, gate_for(cfg), x0, text, T, T, shift=3.0, solver="unipc")
    P = dit.Params(cfg, w.tensors)
    sig = sigma_schedule(T, 3.0)
    t64 = storage_to_f64(text[0], cfg.dtype)
    txt = dit.text_in(P, t64)
    mods = dit.mod_table(P, dit.vec_table(P, sig[:T], t64))
    step = {"t": 0}

    def velocity(x, s):
        t = step["t"]
        assert s == sig[t]
        step["t"] += 1
        h = dit.patch_embed(P, x)
        return dit.final_layer(P, dit.block_stack(P, h, txt, mods[t]), mods[t])

    np.testing.assert_array_equal(res.x, integrate(velocity, x0, sig, rnd=round_f32))
