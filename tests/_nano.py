"""Very small model configs for fast oracle tests."""
import dataclasses

import numpy as np

from paper_2608_09231_amd import synth

NANO = synth.ModelConfig(name="nano", dtype="f32", n_double=1, n_single=1, n_cross=0,
                         hidden=16, heads=2, head_dim=8, mlp_hidden=32, in_channels=4,
                         ctx_dim=8, n_img=6, n_txt=3)
NANO_CROSS = synth.ModelConfig(name="nano_cross", dtype="f32", n_double=0, n_single=0,
                               n_cross=2, hidden=16, heads=2, head_dim=8, mlp_hidden=24,
                               in_channels=4, ctx_dim=8, n_img=5, n_txt=3, pooled_text=False)
NANO_CFG = dataclasses.replace(NANO, name="nano_cfg", batch=2, pooled_text=False, n_single=0)
NANO_BF16 = dataclasses.replace(NANO, name="nano_bf16", dtype="bf16")


def inputs(cfg, seed=3, weight_scale=None):
    w = synth.make_weights(cfg, seed)
    if weight_scale is not None:
        # test-only rescaling of every tensor (keeps the storage dtype)
        for k, v in w.tensors.items():
            if cfg.dtype == "f32":
                v[...] = (v * weight_scale).astype(np.float32)
    return w, synth.make_latent(cfg, seed), synth.make_text(cfg, seed)
