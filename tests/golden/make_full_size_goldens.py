"""Write the full-size oracle goldens of tests/golden/:

  flux1024_full_depth.json  FLUX-1024 at its full depth (19 double + 38 single
                            blocks, H 3072, 4096 image + 512 text tokens),
                            T = 4, B = 2: two passes through the whole block
                            stack, two residual reuses (about 36 minutes);
  wan14b_full_tokens.json   the Wan block at its full width and token count
                            (one video block, H 5120, 32760 video tokens, 512
                            text tokens) with the workload's UniPC step rule,
                            T = 3, B = 2 (about 25 minutes);
  qwen_cfg_full_depth.json  the Qwen-Image guidance pair at its full depth (60
                            double blocks, H 3072, 4096 image + 256 text
                            tokens, both branches, guidance 4), T = 3, B = 2
                            (about 80 minutes).

The float64 oracle needs about 17-21 s per full-width FLUX block and about six
minutes per Wan block at 32760 tokens on eight host cores, so these runs are
stored rather than recomputed by the GPU tests.

Stored per case: the schedule, the gate logits, forced flags, state features
and indicator sums of every step, the final latent x_T and the displacement
x_T - x_0 at every k-th element (k = 256 for FLUX, 2048 for Wan: about 1024
values each), and their full L2 norms.
Only the oracle and the seeded input generators are called.  Run from the
repository root (no argument: every case):
    python tests/golden/make_full_size_goldens.py [case ...]
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

HERE = os.path.dirname(os.path.abspath(__file__))

# case -> (workload, reduction of synth.reduced, sampling stride of the stored latents)
CASES = {
    "flux1024_full_depth": ("flux1024", dict(T=4, B=2), 256),
    "wan14b_full_tokens": ("wan14b", dict(T=3, B=2, n_cross=1), 2048),
    "qwen_cfg_full_depth": ("qwen_cfg", dict(T=3, B=2), 256),
}


def workload(case):
    """The seeded workload of a case (shared with the GPU tests)."""
    name, kw, _ = CASES[case]
    return synth.reduced(synth.workload(name), name=case, **kw)


def _nan_to_none(a):
    return [None if not np.isfinite(v) else float(v) for v in np.asarray(a, np.float64).ravel()]


def make(case):
    w = workload(case)
    cfg = w.model
    t0 = time.time()
    weights, x0, text, gate = synth.make_inputs(w)
    print(f"{case}: inputs ready ({time.time() - t0:.0f} s)", flush=True)
    res = sample(cfg, weights.tensors, gate, x0, text, w.T, w.B, shift=w.shift, guidance=w.guidance,
                 solver=w.solver)
    print(f"{case}: oracle done ({time.time() - t0:.0f} s): schedule {res.full.tolist()}", flush=True)
    x = np.asarray(res.x, np.float64).ravel()
    dx = x - np.asarray(x0, np.float64).ravel()
    stride = CASES[case][2]
    out = {
        "note": f"oracle (float64) gated sample of {case}; written by tests/golden/make_full_size_goldens.py",
        "workload": CASES[case][0], "n_double": cfg.n_double, "n_single": cfg.n_single,
        "n_cross": cfg.n_cross, "n_img": cfg.n_img,
        "T": w.T, "B": w.B, "shift": w.shift, "solver": w.solver, "seed": w.seed,
        "full": res.full.astype(int).tolist(), "forced": res.forced.astype(int).tolist(),
        "logit": _nan_to_none(res.logit), "nfe": int(res.nfe),
        "features": [_nan_to_none(r) for r in res.features],
        "sums": [_nan_to_none(r) for r in res.sums],
        "stride": stride,
        "x_sample": [float(v) for v in x[::stride]],
        "dx_sample": [float(v) for v in dx[::stride]],
        "x_norm": float(np.linalg.norm(x)), "dx_norm": float(np.linalg.norm(dx)),
    }
    path = os.path.join(HERE, case + ".json")
    with open(path, "w") as f:
        json.dump(out, f, indent=0)
    print(f"wrote {path}", flush=True)


if __name__ == "__main__":
    for c in sys.argv[1:] or list(CASES):
        make(c)
