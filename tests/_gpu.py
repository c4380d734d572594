"""Helpers of the GPU parity tests (device buffers via torch, compare
functions).  Every expected value comes from the oracle."""
import numpy as np
import pytest

from paper_2608_09231_amd import binding, synth


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()      # fails loudly if the library is missing
    return torch


def dev(torch, a):
    """numpy -> cuda tensor (uint16 bf16 bits travel as int16)."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).cuda()


def host_bf16(t):
    """cuda int16 tensor of bf16 bits -> float64 numpy."""
    u = t.cpu().numpy().view(np.uint16)
    return (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def assert_bf16_close(got, ref, frac_exact=0.9, ulps=1, atol_rms=2.0 ** -10):
    """Every element within `ulps` bf16 ulps of the oracle's rounded value
    plus an absolute floor of `atol_rms` times the RMS of the reference: an
    f32 accumulator carries an absolute error proportional to the size of
    the summed terms, so an output that is small after cancellation can land
    a few of its own ulps away.  Most elements must be identical."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    floor = atol_rms * float(np.sqrt(np.mean(ref * ref)))
    tol = ulps * 2.0 ** -7 * np.abs(ref) + floor + 1e-30
    bad = np.abs(got - ref) > tol
    assert not bad.any(), (f"{bad.sum()} of {bad.size} beyond {ulps} ulp + floor; worst "
                           f"{np.max(np.abs(got - ref) / tol)} x tolerance")
    assert np.mean(got == ref) >= frac_exact, np.mean(got == ref)


def run_sampler(torch, w: synth.Workload, weights, x0, text, gate, *, T=None, B=None, forced=None,
                tau=0.5, indicator="modulated", handle=None, **kw):
    cfg = w.model
    h = handle or binding.DitCache(cfg, weights.blob)
    lat = dev(torch, x0.astype(np.float32))
    txt = dev(torch, text)
    sched = h.sample(lat, txt, gate, T or w.T, B or w.B, shift=w.shift, tau=tau,
                     guidance=w.guidance, forced_mask=forced, indicator=indicator, **kw)
    torch.cuda.synchronize()
    return lat.cpu().numpy().astype(np.float64), sched, h


def check_schedule_against_oracle(sched, ores, margin=1e-3, cut=0.0):
    """Decisions agree wherever the decision statistic (gate logit, or q_t of
    the threshold rule) is more than `margin` from its cutoff `cut`; counts
    are exact.  `ores` is the oracle replaying the device's schedule, so both
    sides see the same history."""
    T = len(sched.full)
    assert sched.full[0] == 1
    assert int(sched.full.sum()) == int(ores.nfe)
    for t in range(1, T):
        if ores.forced[t]:
            assert sched.forced[t] == 1
            continue
        z = ores.logit[t]
        if np.isnan(z):
            continue
        if abs(z - cut) > margin:
            assert sched.full[t] == (1 if z > cut else 0), (t, z, sched.logit[t])
