"""bfloat16 <-> float64 for the oracle (test infrastructure only).

The model computes in bfloat16 except the position adjustment (Section 4,
inference setup).  Cached and recomputed K/V, queries and outputs are
therefore bfloat16; the oracle reads them exactly as float64 and, where it
must produce a bfloat16 tensor (the adjusted cache), rounds to nearest with
ties to even.
"""
import numpy as np


def bf16_to_f64(bits) -> np.ndarray:
    """Exact value of bfloat16 bit patterns (uint16) as float64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def f64_to_bf16(x) -> np.ndarray:
    """Round float64 values to bfloat16, nearest with ties to even.

    Done directly from float64 (no float32 step, so no double rounding):
    the significand is scaled to 8 bits and rounded with ``np.rint``
    (ties to even).  Values must be finite and, if non-zero, of magnitude
    at least 2**-126 and below the largest bfloat16 (3.39e38); the inputs
    of this project never leave that range, and anything else raises.
    """
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)):
        raise ValueError("f64_to_bf16: non-finite input")
    nz = x != 0
    if np.any(np.abs(x[nz]) < 2.0 ** -126):
        raise ValueError("f64_to_bf16: subnormal bfloat16 range not supported")
    m, e = np.frexp(x)                      # x = m * 2**e, 0.5 <= |m| < 1
    r = np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)   # 8 significant bits
    if np.any(np.abs(r) > 3.3895313892515355e38):
        raise ValueError("f64_to_bf16: overflow")
    # r is exactly representable in bfloat16, hence in float32
    return (r.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
