"""Pins of the oracle's alternative decision policies (Sec. 3): the static
schedule mu(B, T) and the online threshold rule, on the same sampler."""
import numpy as np
import pytest

from oracle import sample, static_schedule
from paper_2608_09231_amd import synth
from tests._nano import NANO, NANO_BF16, inputs

GATE = synth.make_gate_blob((8, 32, 16, 1), seed=1)


@pytest.mark.parametrize("T", range(1, 31))
def test_static_schedule_is_uniform(T):
    """m_0 = 1, exactly B ones, and every gap between consecutive computed
    steps (and from the last one to T) is floor(T/B) or ceil(T/B)."""
    for B in range(1, T + 1):
        m = static_schedule(B, T)
        assert m[0] == 1 and int(m.sum()) == B
        pos = np.flatnonzero(m)
        gaps = np.diff(np.append(pos, T))
        assert set(gaps.tolist()) <= {T // B, -(-T // B)}
        assert gaps.sum() == T
    assert static_schedule(T, T).all()
    assert static_schedule(1, T).tolist() == [1] + [0] * (T - 1)


@pytest.mark.parametrize("cfg", [NANO, NANO_BF16], ids=lambda c: c.name)
def test_static_policy_is_open_loop(cfg):
    """The schedule does not depend on the trajectory: two latents, two
    gates, one mask; and the run equals the gate policy replaying it."""
    w, x0, text = inputs(cfg)
    T, B = 9, 4
    a = sample(cfg, w.tensors, GATE, x0, text, T, B, policy="static")
    b = sample(cfg, w.tensors, synth.make_gate_blob((8, 32, 16, 1), seed=7), -2 * x0, text, T, B,
               policy="static")
    np.testing.assert_array_equal(a.full, static_schedule(B, T))
    np.testing.assert_array_equal(b.full, static_schedule(B, T))
    assert a.nfe == B and np.all(np.isnan(a.logit))
    r = sample(cfg, w.tensors, GATE, x0, text, T, B, forced_mask=static_schedule(B, T))
    np.testing.assert_array_equal(a.x, r.x)


@pytest.mark.parametrize("cfg", [NANO, NANO_BF16], ids=lambda c: c.name)
def test_threshold_policy_limits(cfg):
    """delta < 0 computes every step (the uncached sampler: same result as
    the gate policy at B = T); delta = inf computes only t = 0 (same as
    replaying 1 0...0 at B = 1)."""
    w, x0, text = inputs(cfg)
    T = 7
    every = sample(cfg, w.tensors, GATE, x0, text, T, 3, policy="threshold", delta=-1.0)
    assert every.nfe == T and every.full.all()
    np.testing.assert_array_equal(every.x, sample(cfg, w.tensors, GATE, x0, text, T, T).x)
    once = sample(cfg, w.tensors, GATE, x0, text, T, 3, policy="threshold", delta=np.inf)
    assert once.nfe == 1 and once.full.tolist() == [1] + [0] * (T - 1)
    one = np.zeros(T, np.uint8)
    one[0] = 1
    np.testing.assert_array_equal(once.x, sample(cfg, w.tensors, GATE, x0, text, T, 1, forced_mask=one).x)


def test_threshold_decisions_rederived_from_features():
    """Brute force: q_t = sum of the step changes f5 since the last computed
    step, recomputed from the recorded features; m_t = [q_t > delta]."""
    cfg = NANO
    w, x0, text = inputs(cfg)
    T = 12
    base = sample(cfg, w.tensors, GATE, x0, text, T, T, policy="threshold", delta=-1.0)
    delta = float(np.median(base.features[1:, 5])) * 1.5
    res = sample(cfg, w.tensors, GATE, x0, text, T, 4, policy="threshold", delta=delta)
    assert 1 < res.nfe < T
    q = 0.0
    for t in range(1, T):
        q += res.features[t, 5]
        assert np.isclose(res.features[t, 7], q, rtol=1e-12)
        assert res.logit[t] == res.features[t, 7]
        assert res.full[t] == (1 if q > delta else 0)
        if res.full[t]:
            q = 0.0
    # the budget rules do not apply: B only enters the features
    np.testing.assert_allclose(res.features[1:, 0], 4 / T)
