"""End-to-end GPU parity of the cached sampler against the oracle.

Protocol (the two sides can legitimately disagree only on decisions whose
gate logit is within 1e-3 of the threshold): run the device sampler with the
gate, replay its schedule in the oracle, then require (a) identical
decisions wherever the oracle's logit clears the margin, (b) NFE = B and
m_0 = 1, (c) final latents within rel-L2 1e-5 (f32) / 2e-2 (bf16), (d)
matching indicator sums and features.  Where no near-tie occurs, the
oracle's own gated run must give the identical schedule."""
import numpy as np
import pytest

from oracle import sample as oracle_sample
from paper_2608_09231_amd import binding, synth
from tests._gpu import check_logits, check_schedule_against_oracle, rel_l2, run_sampler, torch_cuda

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
SUM_TOL = {"f32": 1e-5, "bf16": 1e-3}
# f32 runs: the device logit within 1e-5 (1 + |z|) of the oracle's
LOGIT_F32 = 1e-5


def parity(name, *, T=None, B=None, indicator="modulated", tau=0.5, gate=None, policy="gate", delta=0.0,
           solver="euler", expect_schedule=None):
    torch = torch_cuda()
    w = synth.workload(name)
    cfg = w.model
    weights, x0, text, wgate = synth.make_inputs(w)
    gate = wgate if gate is None else gate
    T = T or w.T
    B = B or w.B
    pol = dict(policy=policy, delta=delta, solver=solver)
    x_gpu, sched, h = run_sampler(torch, w, weights, x0, text, gate, T=T, B=B, indicator=indicator, tau=tau,
                                  **pol)
    h.close()
    if policy != "threshold":
        assert sched.nfe == B and int(sched.full.sum()) == B
    assert sched.full[0] == 1 and int(sched.full.sum()) == sched.nfe
    ores = oracle_sample(cfg, weights.tensors, gate, x0, text, T, B, shift=w.shift, tau=tau,
                         guidance=w.guidance, forced_mask=sched.full, indicator=indicator, **pol)
    if policy == "threshold":
        check_schedule_against_oracle(sched, ores, margin=1e-2 * abs(delta), cut=delta)
    else:
        check_schedule_against_oracle(sched, ores)
    err = rel_l2(x_gpu, ores.x)
    assert err <= TOL[cfg.dtype], err
    # magnitude sums (|m_prev|, |m_last|) to SUM_TOL relative; the difference
    # sums carry the storage rounding of both tensors, so their error is bounded
    # relative to the magnitude sum of the same step, not to the difference
    got, ref = sched.sums[1:], ores.sums[1:]
    ok = np.all(np.isfinite(ref), axis=1)
    np.testing.assert_allclose(got[ok][:, [1, 3]], ref[ok][:, [1, 3]], rtol=SUM_TOL[cfg.dtype])
    for d, mcol in ((0, 1), (2, 3)):
        assert np.all(np.abs(got[ok][:, d] - ref[ok][:, d]) <= SUM_TOL[cfg.dtype] * ref[ok][:, mcol]), (d, got, ref)
    np.testing.assert_allclose(sched.features[1:, :4], ores.features[1:, :4], rtol=1e-12)
    np.testing.assert_allclose(sched.features[1:, 4:], ores.features[1:, 4:], rtol=10 * SUM_TOL[cfg.dtype])
    if policy == "gate":
        dz = check_logits(sched, ores, gate, LOGIT_F32 if cfg.dtype == "f32" else None)
        print(f"{name}: largest |z_dev - z_oracle| {dz:.2e}")
    elif policy == "threshold":
        # q_t is feature f7 itself
        np.testing.assert_array_equal(sched.logit[1:], sched.features[1:, 7].astype(np.float32))
    gated = oracle_sample(cfg, weights.tensors, gate, x0, text, T, B, shift=w.shift, tau=tau,
                          guidance=w.guidance, indicator=indicator, **pol)
    stat = ores.logit[1:] - (delta if policy == "threshold" else 0.0)
    if np.all(np.isnan(stat) | (np.abs(stat) > (1e-2 * abs(delta) if policy == "threshold" else 1e-3))):
        np.testing.assert_array_equal(sched.full, gated.full)
    if expect_schedule is not None:
        np.testing.assert_array_equal(gated.full, expect_schedule)
        np.testing.assert_array_equal(sched.full, expect_schedule)
    return sched, ores, err


def test_tiny_f32_parity():
    sched, ores, err = parity("tiny")
    print("tiny rel-L2", err, "schedule", sched.full.tolist())


def test_small_f32_parity():
    parity("small_f32")


def test_small_bf16_parity():
    sched, ores, err = parity("small_bf16")
    print("small_bf16 rel-L2", err, "schedule", sched.full.tolist())


def test_small_bf16_patch_indicator():
    parity("small_bf16", indicator="patch")


def test_small_cfg_bf16_parity():
    parity("small_cfg_bf16")


def test_small_cross_bf16_parity():
    parity("small_cross_bf16")


@pytest.mark.parametrize("name", ["micro_bf16", "micro_cfg_bf16"])
def test_fewer_tokens_than_one_tile(name):
    # 7 image tokens (one ragged 32-token tile), and 33 (a full tile plus one
    # token) as a guidance pair at H = 512 (four waves per work-group)
    parity(name)


@pytest.mark.parametrize("name", ["small_w384_bf16", "small_c32_bf16"])
def test_row_tiled_step_kernels_parity(name):
    # widths and channel counts outside the column-sliced kernel's: the
    # row-tiled fused kernels form the indicator and the reuse candidate
    parity(name)


def test_budget_edges_tiny():
    for T, B in ((1, 1), (6, 6), (7, 1)):
        parity("tiny", T=T, B=B)


def test_paper_flux_gate_with_zscore():
    """App. A.2's FLUX / Qwen gate shape 6-8-8-32-1 (449 parameters) with
    z-scored inputs: reads f0..f5 only."""
    mu = np.array([0.4, 0.5, 0.6, 2.0, 0.1, 0.05], np.float32)
    sd = np.array([0.2, 0.3, 0.4, 1.5, 0.1, 0.05], np.float32)
    gate = synth.make_gate_blob((6, 8, 8, 32, 1), seed=11, zscore=(mu, sd))
    parity("tiny", gate=gate)
    parity("small_bf16", gate=gate)


def test_wan_branched_gate():
    """App. A.2's Wan gate: two 3-8-8 branches (budget / trajectory state)
    fused by 16-32-1, 785 parameters, z-scored inputs; on the video
    cross-attention model."""
    mu = np.array([0.3, 0.5, 0.6, 2.0, 0.1, 0.05], np.float32)
    sd = np.array([0.1, 0.3, 0.4, 1.5, 0.1, 0.05], np.float32)
    gate = synth.make_branched_gate_blob(seed=5, zscore=(mu, sd))
    parity("tiny", gate=gate)
    parity("small_cross_bf16", gate=gate)


def _flip_cases():
    import json
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "flip_gates.json")
    with open(path) as f:
        data = json.load(f)
    return data


FLIP = _flip_cases()


def flip_gate(case):
    """The seeded gate of the case's shape with its output bias moved by beta
    (tests/golden/make_flip_gates.py chose beta with the oracle alone)."""
    z = (np.array(FLIP["zscore_mu"], np.float32), np.array(FLIP["zscore_sd"], np.float32))
    kind, seed, std = case["gate"], case["gate_seed"], case["gate_std"]
    if kind == "833":
        g = synth.make_gate_blob((8, 32, 16, 1), seed=seed, std=std)
    elif kind == "449z":
        g = synth.make_gate_blob((6, 8, 8, 32, 1), seed=seed, std=std, zscore=z)
    else:
        g = synth.make_branched_gate_blob(seed=seed, std=std, zscore=z)
    g[-1] = np.float32(g[-1] + np.float32(case["beta"]))
    return g


@pytest.mark.parametrize("cid", sorted(FLIP["cases"]))
def test_gate_vote_changes_sign(cid):
    """Alg. 2 driven by the gate itself: unforced steps vote compute and
    unforced steps vote reuse within one run, so the schedule is neither of
    the two closed forms a one-signed gate yields.  Device, the oracle's own
    gated run and the stored schedule agree bit for bit (every unforced
    logit is far from the threshold), and the logits agree by value."""
    case = FLIP["cases"][cid]
    T, B = case["T"], case["B"]
    sched, ores, err = parity(case["workload"], T=T, B=B, gate=flip_gate(case), expect_schedule=case["schedule"])
    closed = [np.r_[np.ones(B), np.zeros(T - B)], np.r_[1, np.zeros(T - B), np.ones(B - 1)]]
    assert not any(np.array_equal(sched.full, c) for c in closed)
    unforced = [t for t in range(1, T) if not sched.forced[t]]
    z = sched.logit[unforced]
    assert np.any(z > 0) and np.any(z < 0)
    print(cid, "schedule", sched.full.tolist(), "rel-L2", err)


def test_static_policy():
    from oracle import static_schedule
    for name in ("tiny", "small_bf16"):
        sched, _, _ = parity(name, policy="static", gate=np.zeros(0, np.float32))
        np.testing.assert_array_equal(sched.full, static_schedule(int(sched.nfe), len(sched.full)))


@pytest.mark.parametrize("name,delta", [("tiny", 0.05), ("small_bf16", 0.05), ("small_cfg_bf16", 0.07)])
def test_threshold_policy(name, delta):
    sched, ores, _ = parity(name, policy="threshold", delta=delta, gate=np.zeros(0, np.float32))
    print(name, "threshold", delta, "nfe", sched.nfe, "schedule", sched.full.tolist())


@pytest.mark.parametrize("name", ["tiny", "small_bf16", "small_cfg_bf16", "small_cross_bf16"])
def test_unipc_solver(name):
    """UniPC-2 predictor-corrector (the Wan sampler) in place of Euler."""
    sched, ores, err = parity(name, solver="unipc")
    print(name, "unipc rel-L2", err, "schedule", sched.full.tolist())


def test_forced_replay_and_determinism():
    torch = torch_cuda()
    w = synth.workload("small_bf16")
    weights, x0, text, gate = synth.make_inputs(w)
    x1, s1, h = run_sampler(torch, w, weights, x0, text, gate)
    x2, s2, _ = run_sampler(torch, w, weights, x0, text, gate, handle=h)
    x3, s3, _ = run_sampler(torch, w, weights, x0, text, gate, forced=s1.full, handle=h)
    h.close()
    np.testing.assert_array_equal(x1, x2)
    np.testing.assert_array_equal(s1.full, s2.full)
    np.testing.assert_array_equal(s1.sums[1:], s2.sums[1:])
    np.testing.assert_array_equal(x1, x3)


def test_error_paths_on_device():
    torch = torch_cuda()
    w = synth.workload("tiny")
    weights, x0, text, gate = synth.make_inputs(w)
    h = binding.DitCache(w.model, weights.blob)
    lat = torch.from_numpy(x0).cuda()
    txt = torch.from_numpy(text).cuda()
    for T, B in ((5, 0), (5, 6), (0, 0)):
        with pytest.raises(binding.DitError) as e:
            h.sample(lat, txt, gate, T, B)
        assert e.value.status == binding.DIT_EBUDGET
    with pytest.raises(binding.DitError) as e:
        h.sample(lat, txt, gate[:-1], 5, 2)
    assert e.value.status == binding.DIT_EINVAL
    with pytest.raises(binding.DitError) as e:
        h.sample(lat, txt, gate, 5, 2, forced_mask=[0, 1, 1, 0, 0])
    assert e.value.status == binding.DIT_EINVAL
    bad_gate = synth.make_branched_gate_blob(seed=5)
    bad_gate[10] = 15          # trunk input width != sum of branch outputs
    for g in (bad_gate, bad_gate[:-1], None):
        with pytest.raises(binding.DitError) as e:
            h.sample(lat, txt, g, 5, 2)
        assert e.value.status == binding.DIT_EINVAL
    with pytest.raises(binding.DitError) as e:
        h.sample(lat, txt, None, 5, 2, policy="threshold", delta=float("nan"))
    assert e.value.status == binding.DIT_EINVAL
    # the binding refuses buffers of the wrong size before the library reads them
    for kw in ({"sigmas": np.linspace(1.0, 0.0, 5)}, {"forced_mask": [1, 1, 0, 0]}):
        with pytest.raises(ValueError):
            h.sample(lat, txt, gate, 5, 2, **kw)
    for a, b in ((lat[:-1], txt), (lat.double(), txt), (lat, txt[:, :-1]), (lat.cpu(), txt)):
        with pytest.raises(ValueError):
            h.sample(a, b, gate, 5, 2)
    good = np.linspace(1.0, 0.0, 6)
    for sig in (good[::-1].copy(), np.r_[good[:3], good[2:5]], np.r_[1.5, good[1:]], np.r_[good[:5], np.nan]):
        with pytest.raises(binding.DitError) as e:
            h.sample(lat, txt, gate, 5, 2, sigmas=sig)
        assert e.value.status == binding.DIT_EINVAL
    bad = lat.clone()
    bad[3, 2] = float("nan")
    with pytest.raises(binding.DitError) as e:
        h.sample(bad, txt, gate, 5, 2)
    assert e.value.status == binding.DIT_ENONFINITE
    h.close()
