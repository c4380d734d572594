"""Storage-precision rounding (oracle; test infrastructure only).

The paper fixes no precision.  The workloads fix a storage dtype S (fp32 or
bf16); the oracle computes every value in float64 and rounds it to S only
where the sampler stores a tensor in S.  ``round_bf16`` is round to nearest,
ties to even, from the exact float64 value (no intermediate float32 step).
Pinned against torch's float32->bfloat16 conversion and hand-worked ties.
"""
import numpy as np


def round_f32(x):
    return np.asarray(x, np.float64).astype(np.float32).astype(np.float64)


def round_bf16(x):
    """Nearest bfloat16 value (8 significant bits), ties to even.

    Values are assumed finite and inside the normal bf16 range (our
    activations never reach 2**-126 or 2**127 in magnitude)."""
    x = np.asarray(x, np.float64)
    m, e = np.frexp(x)                  # x = m * 2**e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def round_storage(dtype: str):
    if dtype == "bf16":
        return round_bf16
    if dtype == "f32":
        return round_f32
    raise ValueError(dtype)


def storage_to_f64(a, dtype: str):
    """Decode storage arrays: uint16 bf16 bit patterns or float32."""
    a = np.asarray(a)
    if dtype == "bf16":
        assert a.dtype == np.uint16
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)
