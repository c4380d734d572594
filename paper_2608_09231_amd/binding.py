"""ctypes binding of libdit_cache.so (argument marshalling only).

Every tensor operation of the sampler runs in the library's HIP kernels;
this module converts Python / torch arguments into the C structs and
pointers of ``include/dit_cache.h`` and ``include/dit_kernels.h``.  Loading
fails loudly when the library has not been built: there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdit_cache.so")

DIT_OK, DIT_EINVAL, DIT_ENOMEM, DIT_EHIP, DIT_ESHAPE, DIT_EBUDGET, DIT_ENONFINITE = 0, -1, -2, -3, -4, -5, -6
STATUS_NAMES = {0: "DIT_OK", -1: "DIT_EINVAL", -2: "DIT_ENOMEM", -3: "DIT_EHIP", -4: "DIT_ESHAPE",
                -5: "DIT_EBUDGET", -6: "DIT_ENONFINITE"}
DTYPE_F32, DTYPE_BF16 = 0, 1
INDICATOR_MODULATED, INDICATOR_PATCH = 0, 1
EPI_STORE, EPI_F32, EPI_GATED_RES, EPI_SILU = 0, 1, 2, 4
ABI_VERSION = 4
POLICIES = {"gate": 0, "static": 1, "threshold": 2}
SOLVERS = {"euler": 0, "unipc": 1}
N_FEATURES = 8
K_CLASSES = ["gemm", "attn", "indicator", "reuse", "full_other", "once"]

# Every symbol the headers declare.
EXPORTS = ["dit_cache_create", "dit_cache_sample", "dit_cache_sample_ex", "dit_cache_sample_batch",
           "dit_gate_logit", "dit_cache_destroy",
           "dit_cache_last_error", "dit_cache_set_profiling", "dit_cache_get_stats",
           "dit_cache_reset_stats", "dit_gemm_bf16", "dit_attention_bf16", "dit_attention_bf16_noalloc"]


class ModelConfigC(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "abi_version", "dtype", "n_double", "n_single", "n_cross", "hidden", "heads", "head_dim",
        "mlp_hidden", "in_channels", "ctx_dim", "time_dim", "n_img", "n_txt", "batch", "pooled_text")]


class SampleParamsC(C.Structure):
    _fields_ = [("T", C.c_int32), ("B", C.c_int32), ("sigmas", C.POINTER(C.c_double)),
                ("shift", C.c_double), ("tau", C.c_double), ("guidance", C.c_double),
                ("forced_mask", C.POINTER(C.c_uint8)), ("indicator", C.c_int32),
                ("policy", C.c_int32), ("delta", C.c_double), ("solver", C.c_int32)]


class ScheduleC(C.Structure):
    _fields_ = [("full", C.POINTER(C.c_uint8)), ("logit", C.POINTER(C.c_float)),
                ("forced", C.POINTER(C.c_uint8)), ("features", C.POINTER(C.c_double)),
                ("sums", C.POINTER(C.c_double)), ("nfe", C.c_int32), ("steps_done", C.c_int32)]


class StatsC(C.Structure):
    _fields_ = [("ms", C.c_double * 6), ("work", C.c_double * 6), ("launches", C.c_int64 * 6),
                ("host_gate_ms", C.c_double), ("sample_ms", C.c_double), ("samples", C.c_int64),
                ("full_steps", C.c_int64), ("reuse_steps", C.c_int64)]


class GemmDescC(C.Structure):
    _fields_ = [("A", C.c_void_p), ("lda", C.c_int64), ("W", C.c_void_p), ("ldw", C.c_int64),
                ("bias", C.c_void_p), ("C", C.c_void_p), ("ldc", C.c_int64),
                ("M", C.c_int32), ("N", C.c_int32), ("K", C.c_int32), ("flags", C.c_int32),
                ("gate", C.c_void_p), ("rms_cols", C.c_int32), ("gelu_from", C.c_int32),
                ("gap_at", C.c_int32), ("gap", C.c_int32)]


class DitError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None


def load(path: str = LIB_PATH):
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FileNotFoundError(
            f"{path} is missing: build it with `python -m paper_2608_09231_amd.build`")
    lib = C.CDLL(path)
    vp, sz = C.c_void_p, C.c_size_t
    lib.dit_cache_create.argtypes = [C.POINTER(ModelConfigC), vp, sz, vp, C.POINTER(vp)]
    lib.dit_cache_sample.argtypes = [vp, vp, vp, C.c_int32, C.c_int32, vp, sz, C.POINTER(ScheduleC)]
    lib.dit_cache_sample_ex.argtypes = [vp, vp, vp, vp, sz, C.POINTER(SampleParamsC), C.POINTER(ScheduleC)]
    lib.dit_cache_sample_batch.argtypes = [vp, C.c_int32, vp, vp, vp, sz, C.POINTER(SampleParamsC),
                                           C.POINTER(ScheduleC)]
    lib.dit_gate_logit.argtypes = [vp, sz, vp, vp]
    lib.dit_cache_destroy.argtypes = [vp]
    lib.dit_cache_destroy.restype = None
    lib.dit_cache_last_error.argtypes = [vp]
    lib.dit_cache_last_error.restype = C.c_char_p
    lib.dit_cache_set_profiling.argtypes = [vp, C.c_int32]
    lib.dit_cache_get_stats.argtypes = [vp, C.POINTER(StatsC)]
    lib.dit_cache_reset_stats.argtypes = [vp]
    lib.dit_gemm_bf16.argtypes = [C.POINTER(GemmDescC), vp]
    lib.dit_attention_bf16.argtypes = [vp, C.c_int64, vp, C.c_int64, vp, C.c_int64, vp, C.c_int64,
                                       C.c_int32, C.c_int32, C.c_int32, C.c_int32, vp, vp]
    lib.dit_attention_bf16_noalloc.argtypes = [vp, C.c_int64, vp, C.c_int64, vp, C.c_int64, vp, C.c_int64,
                                               C.c_int32, C.c_int32, C.c_int32, C.c_int32, vp]
    for n in EXPORTS:
        f = getattr(lib, n)
        if n not in ("dit_cache_destroy", "dit_cache_last_error"):
            f.restype = C.c_int
    _lib = lib
    return lib


def _check(status, handle=None):
    if status != DIT_OK:
        msg = _lib.dit_cache_last_error(handle).decode()
        raise DitError(status, msg)


def _stream_ptr(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def model_config_c(cfg) -> ModelConfigC:
    return ModelConfigC(ABI_VERSION, DTYPE_BF16 if cfg.dtype == "bf16" else DTYPE_F32,
                        cfg.n_double, cfg.n_single, cfg.n_cross, cfg.hidden, cfg.heads, cfg.head_dim,
                        cfg.mlp_hidden, cfg.in_channels, cfg.ctx_dim, cfg.time_dim, cfg.n_img,
                        cfg.n_txt, cfg.batch, int(cfg.pooled_text))


@dataclass
class Schedule:
    full: np.ndarray
    logit: np.ndarray
    forced: np.ndarray
    features: np.ndarray
    sums: np.ndarray
    nfe: int
    steps_done: int


class DitCache:
    """Handle of dit_cache_create; ``sample`` wraps dit_cache_sample_ex."""

    def __init__(self, cfg, weights_blob: np.ndarray, stream=None):
        lib = load()
        self.cfg = cfg
        self._stream = stream
        blob = np.ascontiguousarray(weights_blob)
        h = C.c_void_p()
        c = model_config_c(cfg)
        st = lib.dit_cache_create(C.byref(c), blob.ctypes.data_as(C.c_void_p), blob.nbytes,
                                  _stream_ptr(stream), C.byref(h))
        if st != DIT_OK:
            raise DitError(st, lib.dit_cache_last_error(None).decode())
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            _lib.dit_cache_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check_io(self, latents, text_embs, S):
        """The library reads S x [N, C] f32 latents and S x [batch, N_t, ctx]
        text embeddings in the storage dtype through raw device pointers:
        check that the tensors hold exactly that."""
        cfg = self.cfg
        esz = 2 if cfg.dtype == "bf16" else 4
        for t, name, n, size in ((latents, "latent", S * cfg.n_img * cfg.in_channels, 4),
                                 (text_embs, "text_emb", S * cfg.batch * cfg.n_txt * cfg.ctx_dim, esz)):
            if not getattr(t, "is_cuda", False):
                raise ValueError(f"{name} must be a device tensor")
            if not t.is_contiguous() or t.numel() != n or t.element_size() != size:
                raise ValueError(f"{name} must be contiguous with {n} elements of {size} bytes")
        if not latents.is_floating_point():
            raise ValueError("latent must be float32")

    @staticmethod
    def _params(T, B, sigmas, shift, tau, guidance, forced_mask, indicator, policy, delta, solver, S=1):
        sig = None if sigmas is None else np.ascontiguousarray(sigmas, np.float64)
        fm = None if forced_mask is None else np.ascontiguousarray(forced_mask, np.uint8)
        # the library reads T + 1 sigmas and T mask entries per sample
        if sig is not None and sig.size != int(T) + 1:
            raise ValueError(f"sigmas must hold T + 1 = {int(T) + 1} values")
        if fm is not None and fm.size != S * int(T):
            raise ValueError(f"forced mask must hold {S} x T = {S * int(T)} entries")
        p = SampleParamsC(int(T), int(B),
                          sig.ctypes.data_as(C.POINTER(C.c_double)) if sig is not None else None,
                          float(shift), float(tau), float(guidance),
                          fm.ctypes.data_as(C.POINTER(C.c_uint8)) if fm is not None else None,
                          INDICATOR_PATCH if indicator == "patch" else INDICATOR_MODULATED,
                          POLICIES[policy], float(delta), SOLVERS[solver])
        return p, (sig, fm)  # the arrays stay alive with the struct

    @staticmethod
    def _schedules(S, T):
        arrs = [(np.zeros(T, np.uint8), np.zeros(T, np.float32), np.zeros(T, np.uint8),
                 np.zeros(T * N_FEATURES, np.float64), np.zeros(T * 4, np.float64)) for _ in range(S)]
        cs = (ScheduleC * S)()
        for j, (full, logit, forced, feats, sums) in enumerate(arrs):
            cs[j] = ScheduleC(full.ctypes.data_as(C.POINTER(C.c_uint8)),
                              logit.ctypes.data_as(C.POINTER(C.c_float)),
                              forced.ctypes.data_as(C.POINTER(C.c_uint8)),
                              feats.ctypes.data_as(C.POINTER(C.c_double)),
                              sums.ctypes.data_as(C.POINTER(C.c_double)), 0, 0)
        return arrs, cs

    @staticmethod
    def _results(arrs, cs, T):
        return [Schedule(full, logit, forced, feats.reshape(T, N_FEATURES), sums.reshape(T, 4),
                         cs[j].nfe, cs[j].steps_done)
                for j, (full, logit, forced, feats, sums) in enumerate(arrs)]

    def _raise(self, st, res):
        err = DitError(st, _lib.dit_cache_last_error(self._h).decode())
        err.schedule = res
        raise err

    def sample(self, latent, text_emb, gate_blob, T, B, *, sigmas=None, shift=1.0, tau=0.5,
               guidance=1.0, forced_mask=None, indicator="modulated", policy="gate",
               delta=0.0, solver="euler") -> Schedule:
        """latent: torch f32 cuda [N, C] (in place); text_emb: torch cuda
        storage-dtype [batch, N_t, ctx] (bf16 workloads: int16/uint16 bits
        or torch.bfloat16); policy "gate" | "static" | "threshold" (the
        latter two do not read gate_blob, which may be None); solver
        "euler" | "unipc"."""
        self._check_io(latent, text_emb, 1)
        gate = np.ascontiguousarray(gate_blob if gate_blob is not None else [], np.float32)
        arrs, cs = self._schedules(1, T)
        p, keep = self._params(T, B, sigmas, shift, tau, guidance, forced_mask, indicator, policy, delta, solver)
        st = _lib.dit_cache_sample_ex(self._h, C.c_void_p(latent.data_ptr()),
                                      C.c_void_p(text_emb.data_ptr()),
                                      gate.ctypes.data_as(C.c_void_p) if gate.size else None, gate.size,
                                      C.byref(p), cs)
        res = self._results(arrs, cs, T)[0]
        if st != DIT_OK:
            self._raise(st, res)
        return res

    def sample_batch(self, latents, text_embs, gate_blob, T, B, *, sigmas=None, shift=1.0, tau=0.5,
                     guidance=1.0, forced_masks=None, indicator="modulated", policy="gate",
                     delta=0.0, solver="euler") -> list:
        """dit_cache_sample_batch: latents torch f32 cuda [S, N, C] (in
        place), text_embs [S, batch, N_t, ctx] in the storage dtype,
        forced_masks None or [S, T]; one Schedule per sample."""
        S = int(latents.shape[0])
        if S != int(text_embs.shape[0]):
            raise ValueError("latents and text_embs disagree on the number of samples")
        if forced_masks is not None and np.shape(forced_masks) != (S, T):
            raise ValueError("forced_masks must be [n_samples, T]")
        self._check_io(latents, text_embs, S)
        gate = np.ascontiguousarray(gate_blob if gate_blob is not None else [], np.float32)
        arrs, cs = self._schedules(S, T)
        p, keep = self._params(T, B, sigmas, shift, tau, guidance, forced_masks, indicator, policy, delta,
                               solver, S)
        st = _lib.dit_cache_sample_batch(self._h, S, C.c_void_p(latents.data_ptr()),
                                         C.c_void_p(text_embs.data_ptr()),
                                         gate.ctypes.data_as(C.c_void_p) if gate.size else None, gate.size,
                                         C.byref(p), cs)
        res = self._results(arrs, cs, T)
        if st != DIT_OK:
            self._raise(st, res)
        return res

    def set_profiling(self, on: bool):
        _check(_lib.dit_cache_set_profiling(self._h, int(on)), self._h)

    def reset_stats(self):
        _check(_lib.dit_cache_reset_stats(self._h), self._h)

    def stats(self) -> dict:
        s = StatsC()
        _check(_lib.dit_cache_get_stats(self._h, C.byref(s)), self._h)
        return {"ms": {k: s.ms[i] for i, k in enumerate(K_CLASSES)},
                "work": {k: s.work[i] for i, k in enumerate(K_CLASSES)},
                "launches": {k: s.launches[i] for i, k in enumerate(K_CLASSES)},
                "host_gate_ms": s.host_gate_ms, "sample_ms": s.sample_ms, "samples": s.samples,
                "full_steps": s.full_steps, "reuse_steps": s.reuse_steps}


def gemm_bf16(A, W, bias, Cout, *, M, N, K, lda=None, ldw=None, ldc=None, flags=EPI_STORE,
              gate=None, rms_cols=0, gelu_from=None, gap_at=0, gap=0, stream=None):
    """dit_gemm_bf16 on torch cuda tensors (bf16 data as torch.bfloat16 or int16)."""
    lib = load()
    d = GemmDescC(A.data_ptr(), lda if lda is not None else K, W.data_ptr(),
                  ldw if ldw is not None else K, bias.data_ptr() if bias is not None else None,
                  Cout.data_ptr(), ldc if ldc is not None else N, M, N, K, flags,
                  gate.data_ptr() if gate is not None else None, rms_cols,
                  gelu_from if gelu_from is not None else 0x7FFFFFFF, gap_at, gap)
    st = lib.dit_gemm_bf16(C.byref(d), _stream_ptr(stream))
    _check(st, None)


ATTN_BOUNDED_LOGITS = 1


def attention_bf16(q, k, v, o, *, Lq, Lk, heads, ldq, ldk, ldv, ldo, vt_ws, flags=0, stream=None):
    lib = load()
    st = lib.dit_attention_bf16(q.data_ptr(), ldq, k.data_ptr(), ldk, v.data_ptr(), ldv,
                                o.data_ptr(), ldo, Lq, Lk, heads, flags, vt_ws.data_ptr(), _stream_ptr(stream))
    _check(st, None)


NOALLOC_VT_MAX_ELEMS = 16 * 1024 * 1024


def attention_bf16_noalloc(q, k, v, o, *, Lq, Lk, heads, ldq, ldk, ldv, ldo, flags=0, stream=None):
    """dit_attention_bf16_noalloc: the library's own device array holds the
    transposed values (no workspace argument, nothing allocated)."""
    lib = load()
    st = lib.dit_attention_bf16_noalloc(q.data_ptr(), ldq, k.data_ptr(), ldk, v.data_ptr(), ldv,
                                        o.data_ptr(), ldo, Lq, Lk, heads, flags, _stream_ptr(stream))
    _check(st, None)


def gate_logit(gate_blob, features) -> float:
    """dit_gate_logit: the library's host gate on one 8-feature state."""
    lib = load()
    gate = np.ascontiguousarray(gate_blob, np.float32)
    f = np.ascontiguousarray(np.asarray(features, np.float64).reshape(-1)[:N_FEATURES])
    if f.size < N_FEATURES:
        f = np.concatenate([f, np.zeros(N_FEATURES - f.size)])
    out = C.c_double()
    st = lib.dit_gate_logit(gate.ctypes.data_as(C.c_void_p) if gate.size else None, gate.size,
                            f.ctypes.data_as(C.c_void_p), C.byref(out))
    _check(st, None)
    return out.value
