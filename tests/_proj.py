"""The bound a projection GEMM result must meet (tests only).

kvc_projection sums exact bf16 products in float32 on the matrix cores and
rounds once to bf16 after adding the residual in float32.  Against the
exact value (the oracle's projection, float64):
    |gpu - exact| <= 2^-8 |exact| + (k/16 + 4) 2^-23 (sum_e |a_e w_e| + |residual|)
one bf16 rounding (8 significant bits) plus the float32 roundings of the
accumulation (one per 16 terms along k, each at most 2^-24 of the running
magnitude, doubled) and of the residual sum.
"""
import numpy as np

import oracle


def projection_close(got_bits, a, w, rows=None, residual=None):
    """got_bits: bf16 [m, n]; a [n_a, k], w [n, k] ([out, in]); bf16 bits or floats."""
    want = oracle.projection(a, w, rows=rows, residual=residual)
    a64 = oracle.bf16_to_f64(a) if np.asarray(a).dtype == np.uint16 else np.asarray(a, dtype=np.float64)
    w64 = oracle.bf16_to_f64(w) if np.asarray(w).dtype == np.uint16 else np.asarray(w, dtype=np.float64)
    if rows is not None:
        rows = np.asarray(rows, dtype=np.int64)
        ok = (rows >= 0) & (rows < a64.shape[0])
        a64 = np.where(ok[:, None], a64[np.where(ok, rows, 0)], 0.0)
    mag = np.abs(a64) @ np.abs(w64).T
    if residual is not None:
        r64 = oracle.bf16_to_f64(residual) if np.asarray(residual).dtype == np.uint16 else residual
        mag = mag + np.abs(r64)
    k = w64.shape[1]
    bound = 2.0 ** -8 * np.abs(want) + (k / 16 + 4) * 2.0 ** -23 * mag
    err = np.abs(oracle.bf16_to_f64(got_bits) - want)
    return bool(np.all(err <= bound)), float(np.max(err - bound))
