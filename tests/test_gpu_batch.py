"""Multi-prompt sampling (dit_cache_sample_batch): S samples in lockstep,
each with its own schedule, the computing ones' block stacks stacked into
shared launches.  Every sample is checked against the oracle run on that
sample alone (the problem is posed per prompt), under the same bar as the
single-sample parity tests, and against the library's own single-sample
path on the same inputs."""
import numpy as np
import pytest

from oracle import sample as oracle_sample
from paper_2608_09231_amd import binding, synth
from tests._gpu import check_logits, check_schedule_against_oracle, dev, rel_l2, torch_cuda

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
# stacked launches may pick other GEMM tiles than a lone sequence: same
# products, but e.g. the per-head RMS sum of squares in another order
SELF_TOL = {"f32": 1e-6, "bf16": 5e-3}

# Replay masks (T = 8, B = 4) whose per-step computing sets include all
# samples (t = 0), none (t = 6), a non-contiguous subset of three ({0, 1, 3},
# t = 1: gathered modulation vectors), an evenly spaced pair ({0, 2}, t = 5)
# and single samples.
MASKS = np.array([[1, 1, 0, 1, 0, 1, 0, 0],
                  [1, 1, 1, 0, 0, 0, 0, 1],
                  [1, 0, 1, 0, 1, 1, 0, 0],
                  [1, 1, 0, 0, 1, 0, 0, 1]], np.uint8)


def inputs(w, S):
    cfg = w.model
    weights, _, _, gate = synth.make_inputs(w)
    x0 = np.stack([synth.make_latent(cfg, w.seed + 101 * j) for j in range(S)])
    text = np.stack([synth.make_text(cfg, w.seed + 211 * j + 1) for j in range(S)])
    return weights, x0, text, gate


def run_batch(torch, h, w, x0, text, gate, T, B, **kw):
    lat = dev(torch, x0.astype(np.float32))
    txt = dev(torch, text)
    scheds = h.sample_batch(lat, txt, gate, T, B, shift=w.shift, guidance=w.guidance, **kw)
    torch.cuda.synchronize()
    return lat.cpu().numpy().astype(np.float64), scheds


def run_one(torch, h, w, x0, text, gate, T, B, **kw):
    lat = dev(torch, x0.astype(np.float32))
    txt = dev(torch, text)
    sched = h.sample(lat, txt, gate, T, B, shift=w.shift, guidance=w.guidance, **kw)
    torch.cuda.synchronize()
    return lat.cpu().numpy().astype(np.float64), sched


def check_batch(name, S, *, masks=None, solver="euler", T=None, B=None, gate=None):
    torch = torch_cuda()
    w = synth.workload(name)
    cfg = w.model
    T = T or w.T
    B = B or w.B
    weights, x0, text, wgate = inputs(w, S)
    gate = wgate if gate is None else gate
    h = binding.DitCache(cfg, weights.blob)
    try:
        xb, scheds = run_batch(torch, h, w, x0, text, gate, T, B, forced_masks=masks, solver=solver)
        singles = [run_one(torch, h, w, x0[j], text[j], gate, T, B, forced_mask=scheds[j].full, solver=solver)
                   for j in range(S)]
    finally:
        h.close()
    for j, s in enumerate(scheds):
        assert s.nfe == B and int(s.full.sum()) == B and s.full[0] == 1 and s.steps_done == T
        if masks is not None:
            np.testing.assert_array_equal(s.full, masks[j])
        ores = oracle_sample(cfg, weights.tensors, gate, x0[j], text[j], T, B, shift=w.shift,
                             guidance=w.guidance, forced_mask=s.full, solver=solver)
        if masks is None:
            check_schedule_against_oracle(s, ores)
        check_logits(s, ores, gate, 1e-5 if cfg.dtype == "f32" else None)
        err = rel_l2(xb[j], ores.x)
        assert err <= TOL[cfg.dtype], (j, err)
        xs, ss = singles[j]
        np.testing.assert_array_equal(ss.full, s.full)
        assert rel_l2(xb[j], xs) <= SELF_TOL[cfg.dtype], (j, rel_l2(xb[j], xs))
        np.testing.assert_allclose(s.features[1:, :4], ss.features[1:, :4], rtol=1e-12)
    return scheds


@pytest.mark.parametrize("name", ["tiny", "small_bf16", "small_seg_bf16", "small_cfg_bf16", "small_cross_bf16"])
def test_batch_replay_masks(name):
    check_batch(name, 4, masks=MASKS, T=8, B=4)


@pytest.mark.parametrize("name", ["small_bf16", "small_seg_bf16", "small_cfg_bf16"])
def test_batch_gated(name):
    check_batch(name, 3)


def test_batch_flip_gate():
    """A gate whose vote changes sign within a run: each prompt's lane paces
    its own budget, so the prompts' schedules are checked one by one."""
    from tests.test_gpu_sampler import FLIP, flip_gate
    case = FLIP["cases"]["small_bf16_833"]
    scheds = check_batch("small_bf16", 3, gate=flip_gate(case), T=case["T"], B=case["B"])
    print("flip-gate batch schedules", [s.full.tolist() for s in scheds])


def test_batch_unipc():
    check_batch("small_cfg_bf16", 3, solver="unipc")


def test_batch_sizes_on_one_handle():
    """Workspace grows with the batch and is reused by smaller ones: results
    do not depend on what the handle ran before."""
    torch = torch_cuda()
    w = synth.workload("small_seg_bf16")
    weights, x0, text, gate = inputs(w, 3)
    h = binding.DitCache(w.model, weights.blob)
    try:
        x1, s1 = run_one(torch, h, w, x0[0], text[0], gate, w.T, w.B)
        x3, s3 = run_batch(torch, h, w, x0, text, gate, w.T, w.B)
        fm = np.stack([s3[0].full, s3[1].full])
        x2, s2 = run_batch(torch, h, w, x0[:2], text[:2], gate, w.T, w.B, forced_masks=fm)
        x1b, s1b = run_one(torch, h, w, x0[0], text[0], gate, w.T, w.B)
    finally:
        h.close()
    np.testing.assert_array_equal(x1, x1b)
    np.testing.assert_array_equal(s1.full, s1b.full)
    for j in range(2):
        assert rel_l2(x2[j], x3[j]) <= SELF_TOL["bf16"]
        np.testing.assert_array_equal(s2[j].sums[1:2], s3[j].sums[1:2])


def test_batch_error_paths():
    torch = torch_cuda()
    w = synth.workload("small_bf16")
    weights, x0, text, gate = inputs(w, 2)
    h = binding.DitCache(w.model, weights.blob)
    try:
        lat = dev(torch, x0.astype(np.float32))
        txt = dev(torch, text)
        with pytest.raises(ValueError):
            h.sample_batch(lat, txt, gate, 8, 4, forced_masks=MASKS[:1])
        bad = MASKS[:2].copy()
        bad[1, 0] = 0
        with pytest.raises(binding.DitError) as e:
            h.sample_batch(lat, txt, gate, 8, 4, forced_masks=bad)
        assert e.value.status == binding.DIT_EINVAL
        lat[1, 5, 3] = float("nan")
        with pytest.raises(binding.DitError) as e:
            h.sample_batch(lat, txt, gate, 8, 4)
        assert e.value.status == binding.DIT_ENONFINITE
        assert "sample 1" in str(e.value)
        assert all(s.steps_done == 1 for s in e.value.schedule)
    finally:
        h.close()
