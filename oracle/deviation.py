"""Per-token key deviation at the check layer (test infrastructure only).

Paper: CacheBlend picks the tokens to recompute where the keys of the
concatenated cache differ most from keys computed with full attention at
the first layer (Section 2); the paper ranks tokens by the squared
differences of the key entries, as LMCache implements it (Section 3.2),
after the cached keys have been moved to their new positions.

Definition used here: for row r,
    d[r] = sum over kv heads h and channels e of (k_fresh[r,h,e] - k_cached[r,h,e])**2
with the exact real sum rounded once to float64.  Both inputs are bfloat16.
"""
from fractions import Fraction
import math

import numpy as np

from .bf16 import bf16_to_f64


def _two_sum_err(a, b):
    """Rounding error of a + b (Knuth's TwoSum, exact in float64)."""
    s = a + b
    bb = s - a
    return (a - (s - bb)) + (b - bb)


def key_deviation(k_cached_shifted, k_fresh) -> np.ndarray:
    """Exactly rounded squared key deviation per row (float64 [n]).

    k_cached_shifted, k_fresh: bfloat16 bits (uint16) [n, Hkv, D].

    Each difference and square is computed in float64 and checked to be
    exact (TwoSum error zero; square of at most 26 significant bits); the
    exact terms are then summed with ``math.fsum``, which returns the
    correctly rounded sum.  A row with any inexact term is summed in exact
    rational arithmetic instead (``fractions.Fraction``) and rounded once.
    """
    a = bf16_to_f64(k_fresh)
    b = bf16_to_f64(k_cached_shifted)
    assert a.shape == b.shape
    n = a.shape[0]
    a = a.reshape(n, -1)
    b = b.reshape(n, -1)
    t = a - b
    exact = _two_sum_err(a, -b) == 0
    m, _ = np.frexp(t)
    mant = np.ldexp(np.abs(m), 53).astype(np.int64)      # 53-bit integer significand
    exact &= (mant & ((1 << 27) - 1)) == 0              # <= 26 bits -> square exact
    sq = t * t
    row_exact = exact.all(axis=1)
    out = np.empty(n, dtype=np.float64)
    for r in range(n):
        if row_exact[r]:
            out[r] = math.fsum(sq[r].tolist())
        else:
            acc = Fraction(0)
            for x, y in zip(a[r].tolist(), b[r].tolist()):
                dxy = Fraction(x) - Fraction(y)
                acc += dxy * dxy
            out[r] = float(acc)      # int/int -> float is correctly rounded
    return out
