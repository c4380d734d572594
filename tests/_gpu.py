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


def gate_lipschitz(g):
    """Upper bound on |z(f) - z(f')| / |f - f'|_2 for a parsed oracle gate:
    the product of the layers' spectral norms (ReLU is 1-Lipschitz), times
    max 1/sd under z-scoring; parallel branches read disjoint inputs, so
    their concatenation is bounded by the largest branch bound."""
    def net(layers):
        L = 1.0
        for W, _ in layers:
            L *= float(np.linalg.norm(W, 2))
        return L
    L = net(g.layers)
    if g.branches:
        L *= max(net(layers) for _, layers in g.branches)
    if g.sd is not None:
        L *= float(np.max(1.0 / np.abs(g.sd)))
    return L


def check_logits(sched, ores, gate_blob, f32_bound=None):
    """The gate's logit at every unforced-or-forced step t >= 1.

    (a) The host gate is Eq. 1's network: the oracle's gate evaluated on the
        device's own recorded features reproduces the device's logit up to
        the float32 storage of the logit.
    (b) Against the oracle's replay: |z_dev - z_ref| is at most the gate's
        Lipschitz bound times the distance of the two feature vectors (both
        sides evaluate the same network), plus the float32 storage; with
        ``f32_bound`` also at most f32_bound (1 + |z|).
    Returns the largest |z_dev - z_ref|."""
    from oracle import parse_gate_blob
    g = parse_gate_blob(gate_blob)
    L = gate_lipschitz(g)
    worst = 0.0
    for t in range(1, len(sched.full)):
        z_dev = float(sched.logit[t])
        z_own = g.logit(sched.features[t])
        assert abs(z_dev - z_own) <= 1e-6 * (1.0 + abs(z_own)), (t, z_dev, z_own)
        z_ref = float(ores.logit[t])
        dz = abs(z_dev - z_ref)
        df = float(np.linalg.norm(sched.features[t, :g.d_in] - ores.features[t, :g.d_in]))
        assert dz <= L * df + 1e-6 * (1.0 + abs(z_ref)), (t, z_dev, z_ref, L, df)
        if f32_bound is not None:
            assert dz <= f32_bound * (1.0 + abs(z_ref)), (t, z_dev, z_ref)
        worst = max(worst, dz)
    return worst


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
