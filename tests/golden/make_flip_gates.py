"""Write tests/golden/flip_gates.json: gates whose vote changes sign within a run.

A seeded random gate keeps one sign over a whole small run, so Alg. 2 then
yields one of the two closed-form schedules (all votes compute: ones first;
all votes reuse: one compute, then the forced tail).  This script shifts the
gate's output bias by a constant beta and keeps, for each case, the beta
for which the ORACLE's own gated run

  * has unforced steps voting compute and unforced steps voting reuse
    (so the schedule is decided by the gate, not by the budget rules), and
  * keeps every unforced logit as far from the threshold as possible
    (the largest smallest margin over a grid of beta).

Only the oracle and the seeded input generators are called.  Run from the
repository root:  python tests/golden/make_flip_gates.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import sample  # noqa: E402
from paper_2608_09231_amd import synth  # noqa: E402

MU6 = [0.4, 0.5, 0.6, 2.0, 0.1, 0.05]
SD6 = [0.2, 0.3, 0.4, 1.5, 0.1, 0.05]

# (case id, workload, gate kind, T, B); gate seeds and parameter std are searched
CASES = [
    ("tiny_833", "tiny", "833", 10, 5),
    ("tiny_449z", "tiny", "449z", 10, 5),
    ("tiny_785z", "tiny", "785z", 10, 5),
    ("small_bf16_833", "small_bf16", "833", 8, 4),
    ("small_bf16_449z", "small_bf16", "449z", 8, 4),
    ("small_cfg_bf16_833", "small_cfg_bf16", "833", 8, 4),
    ("small_cross_bf16_785z", "small_cross_bf16", "785z", 8, 3),
    ("small_cross_bf16_833", "small_cross_bf16", "833", 8, 3),
]
SEEDS = (1, 2, 3, 4, 5)
STDS = (0.3, 1.0)


def base_gate(kind, seed, std):
    z = (np.array(MU6, np.float32), np.array(SD6, np.float32))
    if kind == "833":
        return synth.make_gate_blob((8, 32, 16, 1), seed=seed, std=std)
    if kind == "449z":
        return synth.make_gate_blob((6, 8, 8, 32, 1), seed=seed, std=std, zscore=z)
    if kind == "785z":
        return synth.make_branched_gate_blob(seed=seed, std=std, zscore=z)
    raise ValueError(kind)


def shifted(blob, beta):
    """The gate with its output bias (the blob's last value) moved by beta."""
    g = blob.copy()
    g[-1] = np.float32(g[-1] + np.float32(beta))
    return g


def unforced_margins(res):
    z = np.array([res.logit[t] for t in range(1, len(res.full)) if not res.forced[t]])
    return z


def search(case):
    cid, wname, kind, T, B = case
    w = synth.workload(wname)
    weights, x0, text, _ = synth.make_inputs(w)
    run = lambda g: sample(w.model, weights.tensors, g, x0, text, T, B, shift=w.shift,  # noqa: E731
                           guidance=w.guidance)
    best = None
    for std in STDS:
        for seed in SEEDS:
            blob = base_gate(kind, seed, std)
            r0 = run(blob)
            lo, hi = float(np.nanmin(r0.logit)) - 0.5, float(np.nanmax(r0.logit)) + 0.5
            for beta in np.round(-np.linspace(lo, hi, 41), 4):
                res = run(shifted(blob, beta))
                z = unforced_margins(res)
                if not (np.any(z > 0) and np.any(z < 0)):
                    continue
                m = float(np.min(np.abs(z)))
                if best is None or m > best[0]:
                    best = (m, seed, std, float(beta), res)
    if best is None:
        raise SystemExit(f"{cid}: no beta flips the vote")
    m, seed, std, beta, res = best
    print(f"{cid}: seed {seed} std {std} beta {beta:+.4f} margin {m:.4f} schedule "
          f"{''.join(map(str, res.full))} forced {''.join(map(str, res.forced))}", flush=True)
    return {"workload": wname, "gate": kind, "gate_seed": seed, "gate_std": std, "T": T, "B": B,
            "beta": beta, "min_unforced_margin": round(m, 6), "schedule": [int(v) for v in res.full],
            "forced": [int(v) for v in res.forced]}


def main():
    out = {"note": ("gates whose vote changes sign within a run: the seeded gate of the named shape "
                    "with beta added to its output bias; schedules are the oracle's own gated runs "
                    "(written by tests/golden/make_flip_gates.py)"),
           "zscore_mu": MU6, "zscore_sd": SD6, "cases": {}}
    for case in CASES:
        out["cases"][case[0]] = search(case)
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "flip_gates.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")


if __name__ == "__main__":
    main()
