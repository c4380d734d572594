"""Pins of the oracle's gate (Eq. 1) and budget pacing (Alg. 2)."""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

from oracle import parse_gate_blob, decide, budget_features
from paper_2608_09231_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")


def test_gate_param_counts_match_paper():
    g = json.load(open(GOLDEN))
    # App. A.2: FLUX / Qwen gate 6->8->8->32->1 has 449 parameters
    assert synth.gate_param_count((6, 8, 8, 32, 1)) == g["gate_params_flux"]["value"]
    # App. A.2: Wan gate = two 3->8->8 branches fused by 16->32->1, 785 parameters
    branch = synth.gate_param_count((3, 8, 8))
    assert 2 * branch + synth.gate_param_count((16, 32, 1)) == g["gate_params_wan"]["value"]
    # the workloads' gate 8->32->16->1 has 833
    assert synth.gate_param_count((8, 32, 16, 1)) == 833
    for widths in ((6, 8, 8, 32, 1), (8, 32, 16, 1)):
        gate = parse_gate_blob(synth.make_gate_blob(widths, seed=1))
        assert gate.n_params == synth.gate_param_count(widths)


@pytest.mark.parametrize("widths,zs", [((8, 32, 16, 1), False), ((6, 8, 8, 32, 1), True)])
def test_gate_forward_vs_torch_sequential(widths, zs):
    rng = np.random.default_rng(5)
    z = None
    if zs:
        z = (rng.standard_normal(widths[0]).astype(np.float32),
             (0.5 + rng.random(widths[0])).astype(np.float32))
    blob = synth.make_gate_blob(widths, seed=9, zscore=z)
    gate = parse_gate_blob(blob)
    mods = []
    p = 1 + len(widths) + 1 + (2 * widths[0] if zs else 0)
    for i in range(1, len(widths)):
        lin = torch.nn.Linear(widths[i - 1], widths[i]).double()
        n = widths[i] * widths[i - 1]
        with torch.no_grad():
            lin.weight.copy_(torch.from_numpy(blob[p:p + n].astype(np.float64).reshape(widths[i], widths[i - 1])))
            p += n
            lin.bias.copy_(torch.from_numpy(blob[p:p + widths[i]].astype(np.float64)))
            p += widths[i]
        mods.append(lin)
        if i < len(widths) - 1:
            mods.append(torch.nn.ReLU())
    net = torch.nn.Sequential(*mods)
    for _ in range(20):
        f = rng.standard_normal(8) * 2
        u = f[: widths[0]]
        if zs:
            u = (u - z[0].astype(np.float64)) / z[1].astype(np.float64)
        ref = float(net(torch.from_numpy(u).reshape(1, -1)).detach()[0, 0])
        assert math.isclose(gate.logit(f), ref, rel_tol=1e-12, abs_tol=1e-12)


def _torch_mlp(blob, p, widths, last_relu):
    mods = []
    for i in range(1, len(widths)):
        lin = torch.nn.Linear(widths[i - 1], widths[i]).double()
        n = widths[i] * widths[i - 1]
        with torch.no_grad():
            lin.weight.copy_(torch.from_numpy(blob[p:p + n].astype(np.float64).reshape(widths[i], widths[i - 1])))
            p += n
            lin.bias.copy_(torch.from_numpy(blob[p:p + widths[i]].astype(np.float64)))
            p += widths[i]
        mods.append(lin)
        if i < len(widths) - 1 or last_relu:
            mods.append(torch.nn.ReLU())
    return torch.nn.Sequential(*mods), p


@pytest.mark.parametrize("zs", [False, True])
def test_branched_gate_vs_torch_modules(zs):
    """App. A.2 Wan gate: two 3->8->8 branches (budget state f0..f2 and
    trajectory state f3..f5), concatenated, fused by 16->32->1."""
    rng = np.random.default_rng(17)
    z = None
    if zs:
        z = (rng.standard_normal(6).astype(np.float32), (0.5 + rng.random(6)).astype(np.float32))
    blob = synth.make_branched_gate_blob(seed=3, zscore=z)
    gate = parse_gate_blob(blob)
    assert gate.n_params == json.load(open(GOLDEN))["gate_params_wan"]["value"]
    assert gate.d_in == 6
    # header: -2, (3; 3 8 8), (3; 3 8 8), (3; 16 32 1), zflag
    assert list(blob[:14]) == [-2, 3, 3, 8, 8, 3, 3, 8, 8, 3, 16, 32, 1, float(zs)]
    p = 14 + (12 if zs else 0)
    b1, p = _torch_mlp(blob, p, (3, 8, 8), True)
    b2, p = _torch_mlp(blob, p, (3, 8, 8), True)
    trunk, p = _torch_mlp(blob, p, (16, 32, 1), False)
    assert p == blob.size
    for _ in range(20):
        f = rng.standard_normal(8) * 2
        u = f[:6]
        if zs:
            u = (u - z[0].astype(np.float64)) / z[1].astype(np.float64)
        ut = torch.from_numpy(u).reshape(1, -1)
        ref = float(trunk(torch.cat([b1(ut[:, :3]), b2(ut[:, 3:])], dim=1)).detach()[0, 0])
        assert math.isclose(gate.logit(f), ref, rel_tol=1e-12, abs_tol=1e-12)


def test_branched_gate_blob_rejects_bad_headers():
    blob = synth.make_branched_gate_blob(seed=3)
    with pytest.raises(ValueError):
        parse_gate_blob(blob[:-1])
    bad = blob.copy()
    bad[10] = 15  # trunk input width != 8 + 8
    with pytest.raises(ValueError):
        parse_gate_blob(bad)
    bad = blob.copy()
    bad[0] = -2.5
    with pytest.raises(ValueError):
        parse_gate_blob(bad)
    big = synth.make_branched_gate_blob(branches=((5, 8), (4, 8)), seed=3)
    with pytest.raises(ValueError):  # 9 inputs > the 8 state features
        parse_gate_blob(big)


def test_gate_blob_rejects_bad_lengths():
    blob = synth.make_gate_blob((8, 32, 16, 1), seed=1)
    with pytest.raises(ValueError):
        parse_gate_blob(blob[:-1])
    bad = blob.copy()
    bad[4] = 2  # last width != 1
    with pytest.raises(ValueError):
        parse_gate_blob(bad)


def test_paper_constants_fixture():
    g = json.load(open(GOLDEN))
    # tau = 0.5 -> decision z > 0 (Alg. 2, Sec. 3.2 budget-exact inference)
    assert g["tau"]["value"] == 0.5
    # Tab. 3 quotes Qwen speed as T / NFE at T = 50
    for b, sp in g["qwen_speed"]["value"].items():
        assert round(50 / int(b), 2) == sp


def simulate(logits, B, T, tau=0.5):
    """Run the pacing rule over a given logit sequence (t = 1..T-1)."""
    m, forced, c = [1], [1], 1
    rows = []
    for t in range(1, T):
        f = budget_features(B, T, t, c)
        d, fr = decide(logits[t], B, T, t, c, tau)
        rows.append((f, d, fr))
        m.append(d)
        forced.append(fr)
        c += d
    return m, forced, rows


@settings(max_examples=400, deadline=None)
@given(T=st.integers(1, 60), data=st.data())
def test_pacing_invariants(T, data):
    B = data.draw(st.integers(1, T))
    logits = data.draw(st.lists(st.one_of(st.floats(-5, 5), st.just(float("nan")), st.just(0.0)),
                                min_size=T, max_size=T))
    m, forced, rows = simulate(logits, B, T)
    assert m[0] == 1 and forced[0] == 1
    assert sum(m) == B
    for (f, d, fr), z in zip(rows, logits[1:]):
        if f[2] >= 1:                    # spend remainder
            assert d == 1 and fr == 1
        elif f[1] == 0:                  # budget exhausted
            assert d == 0 and fr == 1
        else:                            # the gate decides: strict z > 0
            assert fr == 0
            assert d == (1 if z > 0 else 0)


@pytest.mark.parametrize("T,B", [(10, 5), (28, 10), (50, 12), (7, 1), (6, 6)])
def test_pacing_closed_forms(T, B):
    pos, _, _ = simulate([1.0] * T, B, T)
    assert pos == [1] * B + [0] * (T - B)
    neg, _, _ = simulate([-1.0] * T, B, T)
    assert neg == [1] + [0] * (T - B) + [1] * (B - 1)
    nan, _, _ = simulate([float("nan")] * T, B, T)
    assert nan == neg
    tie, _, _ = simulate([0.0] * T, B, T)       # sigma(0) = tau is not > tau
    assert tie == neg


def test_pacing_tau_shifts_threshold():
    T, B = 12, 5
    z = [0.5] * T
    hi, _, _ = simulate(z, B, T, tau=0.7)        # logit(0.7) = 0.847 > 0.5 -> reuse
    lo, _, _ = simulate(z, B, T, tau=0.3)
    assert hi == [1] + [0] * (T - B) + [1] * (B - 1)
    assert lo == [1] * B + [0] * (T - B)


def test_every_admissible_mask_is_reachable_tiny_budget():
    """T=10, B=5: a gate can realise each of the C(9,4) = 126 masks with
    m_0 = 1, and no other."""
    T, B = 10, 5
    seen = set()
    for mask in itertools.product([0, 1], repeat=T - 1):
        z = [0.0] + [1.0 if v else -1.0 for v in mask]
        m, _, _ = simulate(z, B, T)
        seen.add(tuple(m))
    assert len(seen) == math.comb(T - 1, B - 1)
    assert all(s[0] == 1 and sum(s) == B for s in seen)
