#!/usr/bin/env python3
"""Benchmark: budget-aware cached sampling on one MI355X.

Default workload: the Wan2.1-14B-shaped video DiT (40 blocks, H 5120, 40 x
128 heads, FFN 13824, 32760 video tokens + 512 text tokens, bf16, random
init), T = 50 UniPC steps at budget B = 12 -- the largest single-GPU
workload.  ``--workload flux1024`` (and flux2048, qwen_cfg, ...) runs the
others with the same kernels.

One bench step = one whole sample (T denoising steps: B full evaluations and
T - B residual reuses, gate decisions included).  `value` is denoising
steps per second (T / seconds per sample) with all inputs resident in HBM;
samples/s is reported beside it.  The roofline object covers the dominant
kernel class of the workload (the one with the most time: attention for
Wan, the block-stack GEMMs for FLUX-1024), timed live with HIP events on the
sampler's stream during the timed samples: achieved = algorithmic FLOPs of
the class (2 M N K per GEMM, 4 Lq Lk H per attention) / its summed event
time, which is the algorithmic FLOPs per launch over the average launch.

    python bench.py [--gpus 1] [--steps 3] [--warmup 1] [--workload wan14b]
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(w, rows=2048, q_sample=256):
    """Time the CPU oracle (as it stands) on a bounded sample of the same
    workload and extrapolate to one whole sample.

    Per block kind, the oracle's block runs once at `rows` image tokens (all
    text tokens, full width); its attention runs once for `q_sample` query
    rows against the full key count.  The attention time per query-key pair
    (beta) separates the block's time into a part linear in the sequence
    length L (alpha L) and self-attention (beta L^2), which extrapolate to
    the full L.  The per-step pass (embed, indicator, final layer, step
    rule) runs on the same `rows` tokens and scales with the token count; the
    modulation table is timed on the 1-block model and scaled by the
    modulation width."""
    import dataclasses

    from oracle import dit
    from oracle.numerics import round_f32, storage_to_f64
    from oracle.sampler import rel_l1_sums, sigma_schedule
    from paper_2608_09231_amd import synth

    cfg = w.model
    n_s = min(rows, cfg.n_img)
    small = dataclasses.replace(cfg, n_double=min(1, cfg.n_double), n_single=min(1, cfg.n_single),
                                n_cross=min(1, cfg.n_cross), name=cfg.name + "_1blk")
    weights = synth.make_weights(small, w.seed)
    x0 = synth.make_latent(small, w.seed)
    text = synth.make_text(small, w.seed)
    P = dit.Params(small, weights.tensors)
    sig = sigma_schedule(w.T, w.shift)
    t0 = time.perf_counter()
    t64 = storage_to_f64(text[0], small.dtype)
    txt = dit.text_in(P, t64)
    mods = dit.mod_table(P, dit.vec_table(P, sig[:w.T], t64))
    t_once = (time.perf_counter() - t0) * cfg.n_mod / small.n_mod
    x = round_f32(x0[:n_s].astype(np.float64))
    mod = mods[0]
    t0 = time.perf_counter()
    h = dit.patch_embed(P, x)
    sh0, sc0 = dit.first_block_shift_scale(P, mod)
    m = P.rs(dit.modulate(h, sh0, sc0))
    rel_l1_sums(m, m)
    rel_l1_sums(m, m)
    h_out = P.rs(h + h)
    v = dit.final_layer(P, h_out, mod)
    x = round_f32(x + 0.01 * v)
    t_common = (time.perf_counter() - t0) * cfg.n_img / n_s

    # attention time per query-key pair, full key count
    joint = cfg.n_cross == 0
    L_full = cfg.n_img + (cfg.n_txt if joint else 0)
    L_s = n_s + (cfg.n_txt if joint else 0)
    rng = np.random.default_rng(0)
    qs = P.rs(rng.standard_normal((q_sample, cfg.hidden)))
    kv = P.rs(rng.standard_normal((L_full, cfg.hidden)))
    t0 = time.perf_counter()
    dit.attention(qs, kv, kv, cfg.heads, cfg.head_dim)
    beta = (time.perf_counter() - t0) / (q_sample * L_full)

    hs = h
    t_blocks = 0.0
    parts = []
    for kind, count in (("double", cfg.n_double), ("single", cfg.n_single), ("cross", cfg.n_cross)):
        if not count:
            continue
        t0 = time.perf_counter()
        if kind == "double":
            dit.double_block(P, 0, hs, txt, mod)
        elif kind == "single":
            dit.single_block(P, 0, np.concatenate([txt, hs]), mod)
        else:
            dit.cross_block(P, 0, hs, txt, mod)
        t_s = time.perf_counter() - t0
        alpha = max(t_s - beta * L_s * L_s, 0.0) / L_s
        t_full = alpha * L_full + beta * L_full * L_full
        t_blocks += t_full * count
        parts.append(f"{kind} {t_s:.2f} s at {L_s} rows -> {t_full:.1f} s at {L_full}")
    nb = cfg.batch
    t_step_full = t_common + nb * t_blocks
    t_reuse = t_common
    t_sample = t_once + w.B * t_step_full + (w.T - w.B) * t_reuse
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count()
    threads = int(os.environ.get("OMP_NUM_THREADS", cores))
    return {
        "value": w.T / t_sample,
        "unit": "denoising steps/s",
        "cores": min(cores, threads),
        "kind": "oracle",
        "sample": (f"float64 NumPy oracle, extrapolated: one block of each kind of the {cfg.name} model at "
                   f"full width on {n_s} image tokens ({'; '.join(parts)}), its attention on {q_sample} "
                   f"queries x {L_full} keys (time per query-key pair {beta * 1e9:.2f} ns), one "
                   f"per-step pass on the same tokens and the 1-block modulation table; to {cfg.n_double}+{cfg.n_single}+"
                   f"{cfg.n_cross} blocks, T={w.T}, B={w.B}: {t_sample:.1f} s per sample"),
        "seconds_per_sample": t_sample,
    }


def kernel_traffic(kernel, workload, source):
    """HBM-side bytes per launch of `kernel` from the committed rocprofv3
    counter summary profiles/<kernel>_<workload>_hbm_traffic.md, or None when
    it does not cover this workload or `source` changed since the counters
    were taken."""
    import hashlib
    import re

    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_hbm_traffic.md")
    src = os.path.join(ROOT, "paper_2608_09231_amd", "csrc", source)
    try:
        txt = open(path).read()
        m = re.search(r"```json\n(.*?)\n```", txt, flags=re.S)
        data = json.loads(m.group(1))
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    except (OSError, AttributeError, ValueError):
        return None
    if data.get("source_sha256_16") != sha:
        return None
    return data["traffic_bytes_per_launch"]


def multi_prompt(h, w, lat0, args, ms_single):
    """P prompts (own latents and texts) through dit_cache_sample_batch: each
    keeps its own schedule, the computing ones share the block-stack
    launches.  Timed like the single-sample leg (same step and warmup
    counts, inputs resident)."""
    import torch

    from paper_2608_09231_amd import synth
    cfg = w.model
    P = args.prompts
    xs = np.stack([synth.make_latent(cfg, w.seed + 101 * j) for j in range(P)])
    ts = np.stack([synth.make_text(cfg, w.seed + 211 * j + 1) for j in range(P)])
    gate = synth.make_gate_blob(w.gate_widths, w.seed, w.gate_std)
    lats0 = torch.from_numpy(xs).cuda()
    txts = torch.from_numpy(ts.view(np.int16) if ts.dtype == np.uint16 else ts).cuda()
    lats = lats0.clone()

    def one():
        lats.copy_(lats0)
        return h.sample_batch(lats, txts, gate, w.T, w.B, shift=w.shift, guidance=w.guidance, solver=w.solver)

    for _ in range(args.warmup):
        one()
    torch.cuda.synchronize()
    h.reset_stats()
    t0 = time.perf_counter()
    for i in range(args.steps):
        scheds = one()
        log(f"[bench] multi-prompt batch {i + 1}/{args.steps} done at {time.perf_counter() - t0:.1f} s")
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    st = h.stats()
    full = np.stack([s.full for s in scheds])
    per_step = full.sum(axis=0)
    log(f"[bench] multi-prompt: {args.steps} x {P} samples in {dt:.3f} s; computing samples per step "
        f"{''.join(map(str, per_step.tolist()))}")
    ms_batch = dt / args.steps * 1e3
    return {
        "prompts": P,
        "samples_per_s": P / (ms_batch * 1e-3),
        "steps_per_s": P * w.T / (ms_batch * 1e-3),
        "ms_per_batch": ms_batch,
        "speedup_vs_one_at_a_time": P * ms_single / ms_batch,
        "stacked_steps": int((per_step > 0).sum()),
        "mean_samples_per_stacked_step": float(per_step[per_step > 0].mean()),
        "host_gate_ms_per_batch": st["host_gate_ms"] / max(args.steps, 1),
        "data": "prompt j: latent seed + 101 j, text seed + 211 j + 1; one gate for all",
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="wan14b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="time without per-kernel events")
    ap.add_argument("--prompts", type=int, default=0,
                    help="multi-prompt leg: this many prompts sampled together (0 or 1: skip)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one plain 256 MiB device-to-device copy first (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the sampler has no multi-GPU path "
              "(one sample's steps are sequential; samples are independent).", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2608_09231_amd import binding, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    w = synth.workload(args.workload)
    cfg = w.model
    log(f"[bench] generating {cfg.name} weights ({synth.weight_count(cfg) / 1e9:.2f} B params)")
    t0 = time.time()
    weights = synth.make_weights(cfg, w.seed)
    x0 = synth.make_latent(cfg, w.seed)
    text = synth.make_text(cfg, w.seed)
    gate = synth.make_gate_blob(w.gate_widths, w.seed, w.gate_std)
    log(f"[bench] inputs ready in {time.time() - t0:.1f} s; uploading")
    if args.copy_calibration:
        n = 64 << 20                     # 64 Mi float32 = 256 MiB read + 256 MiB written
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy: {n * 4} bytes read, {n * 4} bytes written")
        del src, dst
    stream = torch.cuda.current_stream()
    h = binding.DitCache(cfg, weights.blob, stream)
    del weights
    lat0 = torch.from_numpy(x0).cuda()
    txt = torch.from_numpy(text.view(np.int16) if text.dtype == np.uint16 else text).cuda()
    lat = lat0.clone()

    def one():
        lat.copy_(lat0)
        return h.sample(lat, txt, gate, w.T, w.B, shift=w.shift, guidance=w.guidance, solver=w.solver)

    for i in range(args.warmup):
        s = one()
        log(f"[bench] warmup {i}: schedule {''.join(map(str, s.full.tolist()))}")
    torch.cuda.synchronize()
    h.set_profiling(not args.no_profile)
    h.reset_stats()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        s = one()
        # one line per sample (a host print after the sample has drained)
        log(f"[bench] timed sample {i + 1}/{args.steps} done at {time.perf_counter() - t0:.1f} s")
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    st = h.stats()
    h.set_profiling(False)
    log(f"[bench] timed {args.steps} samples in {dt:.3f} s; schedule {''.join(map(str, s.full.tolist()))}")
    log(f"[bench] stats {json.dumps(st)}")

    ms_per_sample = dt / args.steps * 1e3
    ms = st["ms"]
    work = st["work"]
    gemm_tflops = work["gemm"] / (ms["gemm"] * 1e-3) / 1e12 if ms["gemm"] else 0.0
    attn_tflops = work["attn"] / (ms["attn"] * 1e-3) / 1e12 if ms["attn"] else 0.0
    reuse_gbs = work["reuse"] / (ms["reuse"] * 1e-3) / 1e9 if ms["reuse"] else 0.0
    ind_gbs = work["indicator"] / (ms["indicator"] * 1e-3) / 1e9 if ms["indicator"] else 0.0
    # dominant kernel class: the MFMA class with the most event time
    dom = "attn" if ms["attn"] > ms["gemm"] else "gemm"
    dom_kernel = {"gemm": ("gemm_bf16_ring_kernel", "bf16 GEMM (block-stack linear layers)", "gemm_bf16.hip"),
                  "attn": ("flash_attn_pipe_kernel", "bf16 flash attention (self- and cross-attention)",
                           "attention.hip")}[dom]
    launches = max(st["launches"][dom], 1)
    dom_tflops = work[dom] / (ms[dom] * 1e-3) / 1e12 if ms[dom] else 0.0
    out = {
        "metric": "denoising steps/s at budget B/T",
        "value": w.T / (ms_per_sample * 1e-3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_sample,
        "step_unit": f"one sample = {w.T} denoising steps at B={w.B} (gate decisions included)",
        "samples_per_s": 1e3 / ms_per_sample,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded N(0,1) latent and text embeddings, N(0,0.02) random-init weights, N(0,0.3) gate)",
        "config": {"workload": cfg.name, "T": w.T, "B": w.B, "solver": w.solver,
                   "blocks": (f"{cfg.n_cross} video (self-attn, cross-attn, FFN)" if cfg.n_cross
                              else f"{cfg.n_double} double + {cfg.n_single} single"),
                   "hidden": cfg.hidden, "heads": cfg.heads, "img_tokens": cfg.n_img, "txt_tokens": cfg.n_txt,
                   "mlp_hidden": cfg.mlp_hidden, "batch": cfg.batch, "gate": "-".join(map(str, w.gate_widths))},
        "roofline": {
            "bound": "mfma",
            "kernel": f"{dom_kernel[0]}: {dom_kernel[1]}",
            "achieved": dom_tflops,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": dom_tflops / PEAK_BF16_TFLOPS,
            "traffic": kernel_traffic(dom_kernel[0], cfg.name, dom_kernel[2]),
            "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
            "avg_launch_us": ms[dom] * 1e3 / launches,
            "flops_per_launch": work[dom] / launches,
        },
        "kernels": {
            "gemm_tflops": gemm_tflops,
            "gemm_frac_bf16_peak": gemm_tflops / PEAK_BF16_TFLOPS,
            "attention_tflops": attn_tflops,
            "attention_frac_bf16_peak": attn_tflops / PEAK_BF16_TFLOPS,
            "reuse_path_gbs": reuse_gbs,
            "indicator_gbs": ind_gbs,
            # streaming kernels together (indicator every step + reuse steps): algorithmic
            # bytes over their event time, against the 8 TB/s HBM peak
            "streaming_hbm_frac": ((work["indicator"] + work["reuse"]) / ((ms["indicator"] + ms["reuse"]) * 1e-3)
                                   / (PEAK_HBM_GBS * 1e9)) if (ms["indicator"] + ms["reuse"]) else 0.0,
            "ms_per_sample_by_class": {k: v / max(args.steps, 1) for k, v in ms.items()},
            "host_gate_ms_per_sample": st["host_gate_ms"] / max(args.steps, 1),
            "full_steps": st["full_steps"], "reuse_steps": st["reuse_steps"],
        },
        "paper_context": ("paper (one RTX 4090, precision not stated; context only): Wan2.1-T2V-1.3B 832x480, 65 "
                          "frames, 50-step UniPC: 184.40 s full compute, BAG B=15 55.76 s (3.31x) (Tab. 2); "
                          "FLUX.1-dev 1024^2, T=50: 31.13 s full, BAG B=9 5.99 s (Tab. 1)"),
    }
    if args.prompts > 1:
        out["multi_prompt"] = multi_prompt(h, w, lat0, args, ms_per_sample)
    h.close()
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        t0 = time.time()
        cb = cpu_baseline(w)
        log(f"[bench] cpu baseline done in {time.time() - t0:.1f} s")
        out["cpu_baseline"] = {k: cb[k] for k in ("value", "unit", "cores", "kind", "sample")}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
