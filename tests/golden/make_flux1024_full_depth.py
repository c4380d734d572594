"""Write tests/golden/flux1024_full_depth.json: the oracle's gated sample of
the FLUX-1024 workload at its full depth (19 double + 38 single blocks,
H 3072, 4096 image + 512 text tokens) on a short schedule (T = 4, B = 2:
two passes through the whole block stack, two residual reuses).

The float64 oracle needs about 17-21 s per full-width block on eight host
cores, so the whole T = 28 schedule (10 full evaluations of 57 blocks) would
take hours; two full evaluations take about 40 minutes and still carry the
bf16 rounding of the device path through every block of the stack.

Stored: the schedule, the gate logits, forced flags, state features and
indicator sums of every step, the final latent x_T and the displacement
x_T - x_0 at every 256th element (1024 values each), and their full L2
norms.  Only the oracle and the seeded input generators are called.  Run
from the repository root:
    python tests/golden/make_flux1024_full_depth.py
"""
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import sample  # noqa: E402
from paper_2608_09231_amd import synth  # noqa: E402

T, B = 4, 2
STRIDE = 256
OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "flux1024_full_depth.json")


def _nan_to_none(a):
    return [None if not np.isfinite(v) else float(v) for v in np.asarray(a, np.float64).ravel()]


def main():
    w = synth.reduced(synth.workload("flux1024"), T=T, B=B, name="flux1024_full_depth")
    cfg = w.model
    t0 = time.time()
    weights, x0, text, gate = synth.make_inputs(w)
    print(f"inputs ready ({time.time() - t0:.0f} s)", flush=True)
    res = sample(cfg, weights.tensors, gate, x0, text, T, B, shift=w.shift, guidance=w.guidance,
                 solver=w.solver)
    print(f"oracle done ({time.time() - t0:.0f} s): schedule {res.full.tolist()}", flush=True)
    x = np.asarray(res.x, np.float64).ravel()
    dx = x - np.asarray(x0, np.float64).ravel()
    out = {
        "note": "oracle (float64) gated sample of flux1024 at full depth, T = 4, B = 2; "
                "written by tests/golden/make_flux1024_full_depth.py",
        "workload": "flux1024", "n_double": cfg.n_double, "n_single": cfg.n_single,
        "T": T, "B": B, "shift": w.shift, "solver": w.solver, "seed": w.seed,
        "full": res.full.astype(int).tolist(), "forced": res.forced.astype(int).tolist(),
        "logit": _nan_to_none(res.logit), "nfe": int(res.nfe),
        "features": [_nan_to_none(r) for r in res.features],
        "sums": [_nan_to_none(r) for r in res.sums],
        "stride": STRIDE,
        "x_sample": [float(v) for v in x[::STRIDE]],
        "dx_sample": [float(v) for v in dx[::STRIDE]],
        "x_norm": float(np.linalg.norm(x)), "dx_norm": float(np.linalg.norm(dx)),
    }
    with open(OUT, "w") as f:
        json.dump(out, f, indent=0)
    print(f"wrote {OUT}", flush=True)


if __name__ == "__main__":
    main()
