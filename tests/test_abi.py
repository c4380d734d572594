"""C-ABI checks that need no GPU: the library loads, exports every symbol
the headers declare, and rejects bad configurations before touching the
device."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2608_09231_amd import binding, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for h in ("dit_cache.h", "dit_kernels.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        for m in re.finditer(r"^\s*(?:const\s+)?\w+\s*\**\s*(dit_\w+)\s*\(", src, flags=re.M):
            names.add(m.group(1))
    return names


def test_library_exports_every_declared_symbol():
    lib = binding.load()
    decl = declared_functions()
    assert decl == set(binding.EXPORTS)
    for n in decl:
        assert getattr(lib, n) is not None


def _create(cfg_c, blob):
    lib = binding.load()
    h = C.c_void_p()
    st = lib.dit_cache_create(C.byref(cfg_c), blob.ctypes.data_as(C.c_void_p), blob.nbytes, None, C.byref(h))
    return st, lib.dit_cache_last_error(None).decode()


def test_create_rejects_bad_configs_without_gpu():
    wl = synth.workload("tiny")
    cfg = binding.model_config_c(wl.model)
    blob = np.zeros(4, np.float32)
    bad = binding.model_config_c(wl.model)
    bad.abi_version = 99
    assert _create(bad, blob)[0] == binding.DIT_EINVAL
    bad = binding.model_config_c(wl.model)
    bad.heads = 3
    assert _create(bad, blob)[0] == binding.DIT_ESHAPE
    bad = binding.model_config_c(wl.model)
    bad.batch = 3
    assert _create(bad, blob)[0] == binding.DIT_ESHAPE
    bad = binding.model_config_c(synth.workload("small_bf16").model)
    bad.head_dim, bad.heads = 64, 4
    assert _create(bad, blob)[0] == binding.DIT_ESHAPE
    st, msg = _create(cfg, blob)                      # wrong blob size
    assert st == binding.DIT_ESHAPE and "bytes" in msg


def test_null_arguments():
    lib = binding.load()
    assert lib.dit_cache_create(None, None, 0, None, None) == binding.DIT_EINVAL
    assert lib.dit_cache_sample(None, None, None, 1, 1, None, 0, None) == binding.DIT_EINVAL
    assert lib.dit_cache_sample_batch(None, 2, None, None, None, 0, None, None) == binding.DIT_EINVAL
    assert lib.dit_cache_set_profiling(None, 1) == binding.DIT_EINVAL
    assert lib.dit_gemm_bf16(None, None) == binding.DIT_EINVAL


def test_blob_size_matches_layout():
    for name in ("tiny", "small_bf16", "small_cross_bf16", "flux1024", "wan14b", "qwen_cfg"):
        cfg = synth.workload(name).model
        n = synth.weight_count(cfg)
        # the C library computes the same total; check via the error message
        blob = np.zeros(1, np.uint16 if cfg.dtype == "bf16" else np.float32)
        st, msg = _create(binding.model_config_c(cfg), blob)
        assert st == binding.DIT_ESHAPE
        assert msg.endswith(str(n * (2 if cfg.dtype == "bf16" else 4))), (name, msg)


def test_noalloc_attention_rejects_oversized_on_the_host():
    """The size check of the allocation-free attention runs before any
    device call (no GPU needed; nothing is launched)."""
    lib = binding.load()
    fake = C.c_void_p(0x1000)
    H = 24 * 128
    st = lib.dit_attention_bf16_noalloc(fake, H, fake, H, fake, H, fake, H, 8, 5441, 24, 0, None)
    assert st == binding.DIT_ESHAPE
    assert "allocation-free limit" in lib.dit_cache_last_error(None).decode()
    st = lib.dit_attention_bf16_noalloc(None, H, fake, H, fake, H, fake, H, 8, 8, 24, 0, None)
    assert st == binding.DIT_EINVAL


def test_gemm_rejects_bad_shapes_on_the_host():
    """The GEMM entry point checks its shape and strides before any device
    call (no GPU needed; nothing is launched)."""
    lib = binding.load()
    fake = 0x1000

    def desc(**kw):
        d = dict(A=fake, lda=256, W=fake, ldw=256, bias=None, C=fake, ldc=512, M=64, N=512, K=256,
                 flags=0, gate=None, rms_cols=0, gelu_from=512, gap_at=0, gap=0)
        d.update(kw)
        return binding.GemmDescC(**d)

    for kw in ({"K": 250, "lda": 256, "ldw": 256}, {"lda": 128}, {"ldw": 128}, {"ldc": 511},
               {"ldc": 600, "gap_at": 256, "gap": 128}, {"gap": -1}, {"rms_cols": 100}):
        d = desc(**kw)
        assert lib.dit_gemm_bf16(C.byref(d), None) == binding.DIT_ESHAPE, kw
    for kw in ({"flags": 8}, {"flags": binding.EPI_GATED_RES}, {"C": None}):
        d = desc(**kw)
        assert lib.dit_gemm_bf16(C.byref(d), None) == binding.DIT_EINVAL, kw


# ---------------------------------------------------------------- host gate

def _gates():
    from tests.test_gpu_sampler import FLIP, flip_gate
    mu = np.array([0.4, 0.5, 0.6, 2.0, 0.1, 0.05], np.float32)
    sd = np.array([0.2, 0.3, 0.4, 1.5, 0.1, 0.05], np.float32)
    gates = [synth.make_gate_blob((8, 32, 16, 1), seed=0),
             synth.make_gate_blob((8, 32, 16, 1), seed=3, std=1.0),
             synth.make_gate_blob((6, 8, 8, 32, 1), seed=11, zscore=(mu, sd)),
             synth.make_branched_gate_blob(seed=5, zscore=(mu, sd)),
             synth.make_branched_gate_blob(seed=2)]
    gates += [flip_gate(c) for c in FLIP["cases"].values()]
    return gates


def test_host_gate_matches_the_oracle_gate():
    """dit_gate_logit (the gate the sampler evaluates between launches) is
    Eq. 1's network as the oracle reads it, for the plain, z-scored and
    branched blobs, on random states around the workloads' feature ranges."""
    from oracle import parse_gate_blob
    rng = np.random.default_rng(9)
    for blob in _gates():
        g = parse_gate_blob(blob)
        for _ in range(40):
            f = np.r_[rng.uniform(0, 1, 3), rng.integers(1, 12), rng.uniform(0, 0.5, 2), rng.uniform(0, 1),
                      rng.uniform(0, 2)]
            z = binding.gate_logit(blob, f)
            ref = g.logit(f)
            assert abs(z - ref) <= 1e-12 * (1 + abs(ref)), (z, ref)


def test_host_gate_rejects_malformed_blobs():
    good = synth.make_gate_blob((8, 32, 16, 1), seed=0)
    bad = [good[:-1], np.r_[good, 0.0], good[:3]]
    b = good.copy(); b[0] = 1.5; bad.append(b)                 # fractional layer count
    b = good.copy(); b[4] = 2; bad.append(b)                   # output width != 1
    b = good.copy(); b[1] = 9; bad.append(b)                   # more than 8 inputs
    br = synth.make_branched_gate_blob(seed=5)
    b = br.copy(); b[10] = 15; bad.append(b)                   # trunk input != branch outputs
    b = br.copy(); b[0] = -20; bad.append(b)                   # branch count
    f = np.zeros(8)
    for blob in bad:
        with pytest.raises(binding.DitError) as e:
            binding.gate_logit(blob, f)
        assert e.value.status == binding.DIT_EINVAL
    with pytest.raises(binding.DitError):
        binding.gate_logit(np.zeros(0, np.float32), f)


# ------------------------------------------------- sanitized host driver

_SAN_SCRIPT = r"""
import ctypes as C, sys
import numpy as np
sys.path.insert(0, sys.argv[2])
from paper_2608_09231_amd import binding, synth
lib = binding.load(sys.argv[1])
rng = np.random.default_rng(0)
# gate parsing on valid, truncated and randomly corrupted blobs
blobs = [synth.make_gate_blob((8, 32, 16, 1), seed=0), synth.make_gate_blob((6, 8, 8, 32, 1), seed=1),
         synth.make_branched_gate_blob(seed=5)]
f = np.linspace(0.1, 0.8, 8)
out = C.c_double()
n_ok = 0
for base in blobs:
    for trial in range(400):
        b = base.copy()
        if trial % 4 == 1:
            b = b[: rng.integers(0, b.size)]
        elif trial % 4 == 2:
            i = rng.integers(0, min(b.size, 16))
            b[i] = rng.choice([-3.0, -1.0, 0.0, 1.0, 2.5, 7.0, 9.0, 1e9, -1e9, np.nan, np.inf])
        elif trial % 4 == 3:
            b = np.r_[b, rng.standard_normal(rng.integers(1, 5)).astype(np.float32)]
        b = np.ascontiguousarray(b, np.float32)
        st = lib.dit_gate_logit(b.ctypes.data_as(C.c_void_p) if b.size else None, b.size,
                                f.ctypes.data_as(C.c_void_p), C.byref(out))
        assert st in (0, -1), st
        n_ok += st == 0
        lib.dit_cache_last_error(None)
# configuration checks of create (no device memory is touched before they pass)
wl = synth.workload("tiny")
for field, val in (("abi_version", 99), ("heads", 3), ("hidden", -1), ("batch", 3), ("n_cross", 2),
                   ("dtype", 7), ("head_dim", 0), ("n_img", 0)):
    cfg = binding.model_config_c(wl.model)
    setattr(cfg, field, val)
    h = C.c_void_p()
    blob = np.zeros(4, np.float32)
    st = lib.dit_cache_create(C.byref(cfg), blob.ctypes.data_as(C.c_void_p), blob.nbytes, None, C.byref(h))
    assert st < 0, (field, st)
    assert len(lib.dit_cache_last_error(None)) > 0
fake = C.c_void_p(0x1000)
assert lib.dit_attention_bf16_noalloc(fake, 3072, fake, 3072, fake, 3072, fake, 3072, 8, 5441, 24, 0, None) < 0
print("SANITIZED-OK", n_ok)
"""


def test_host_driver_under_address_and_ub_sanitizers(tmp_path):
    """The host driver built with AddressSanitizer and UBSan (host code
    only) runs the device-free entry points -- gate parsing on valid,
    truncated and corrupted blobs, create's configuration checks, the
    allocation-free attention's size check -- without a sanitizer report."""
    import subprocess
    import sys

    from paper_2608_09231_amd import build
    lib = build.build_sanitized()
    rt = build.sanitizer_runtime()
    if not os.path.exists(rt):
        pytest.skip("no AddressSanitizer runtime")
    script = tmp_path / "san.py"
    script.write_text(_SAN_SCRIPT)
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, str(script), lib, ROOT], capture_output=True, text=True, env=env,
                       timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "SANITIZED-OK" in r.stdout
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-4000:]
