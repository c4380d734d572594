"""Build libdit_cache.so for gfx950 with hipcc (in-tree).

    python -m paper_2608_09231_amd.build [--debug | --sanitize]

Every source is compiled on each call (objects under ``_build/``), then
linked into ``paper_2608_09231_amd/libdit_cache.so``.  ``--sanitize`` builds
``_build/sanitize/libdit_cache_sanitized.so`` instead: the host driver
(``dit_cache.cpp``) with AddressSanitizer and UndefinedBehaviorSanitizer on
its host code only (device code is compiled as usual), linked with the other
objects of the last normal build.  Load it with the AddressSanitizer runtime
preloaded (``sanitizer_runtime()``).
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libdit_cache.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = os.environ.get("DIT_OFFLOAD_ARCH", "gfx950")

SOURCES = ["dit_cache.cpp", "gemm_bf16.hip", "gemm_f32.hip", "attention.hip", "stream_kernels.hip",
           "reuse_kernels.hip", "step_stream.hip"]

COMMON = [
    f"--offload-arch={ARCH}", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function", "-Wno-unused-value", "-Wno-unused-result",
    # packed f32 arithmetic stays off for all device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _compile(src, opt):
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC, *COMMON, opt, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in (r.stderr or "").splitlines()
                    if "packed-fp32-ops" not in l and l.strip())
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err:
        sys.stderr.write(err + "\n")
    return obj


def build(debug: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    opt = "-O1" if debug else "-O3"
    with ThreadPoolExecutor(len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, opt), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    os.replace(tmp, LIB)
    return LIB


SAN_DIR = os.path.join(BUILD, "sanitize")
SAN_LIB = os.path.join(SAN_DIR, "libdit_cache_sanitized.so")
# host-side sanitizers only: each -fsanitize= follows -Xarch_host
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=undefined"]


def sanitizer_runtime() -> str:
    """Path of the AddressSanitizer runtime of hipcc's clang (to preload)."""
    clang = os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang"
    r = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    return r.stdout.strip()


def build_sanitized() -> str:
    objs = [os.path.join(BUILD, s + ".o") for s in SOURCES if s != "dit_cache.cpp"]
    if not all(os.path.exists(o) for o in objs):
        build()
    os.makedirs(SAN_DIR, exist_ok=True)
    obj = os.path.join(SAN_DIR, "dit_cache.cpp.o")
    cmd = [HIPCC, *COMMON, "-O1", "-g", *SAN_FLAGS, "-x", "hip", "-c", os.path.join(CSRC, "dit_cache.cpp"), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for the sanitized host driver:\n" + r.stderr)
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *SAN_FLAGS, obj, *objs, "-o", SAN_LIB]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    return SAN_LIB


if __name__ == "__main__":
    if "--sanitize" in sys.argv:
        print(build_sanitized())
    else:
        print(build(debug="--debug" in sys.argv))
