"""Recompute count and top-k token selection (test infrastructure only).

Paper: CacheBlend recomputes a fixed fraction (15 %) of the tokens, those
with the largest key deviation (Section 3.1, Section 3.2).  The tokens of
the final chunk (instruction and question) are new and always computed
(Section 4 setup: they are prefilled, not reused), so the candidates are the
reused rows only.

Readings fixed here (the paper does not spell them out):
* k = floor(ratio * n_reused), with the product taken in IEEE float64;
* equal deviations are ordered by the lower row first;
* the selected rows are returned in ascending row order, followed by the
  query rows n_reused .. N-1.
"""
import math

import numpy as np


def recompute_count(ratio: float, n_reused: int) -> int:
    """k = floor(ratio * n_reused) (float64 product); -1 if ratio not in [0, 1]."""
    ratio = float(ratio)
    if not (0.0 <= ratio <= 1.0):       # also rejects NaN
        return -1
    return int(math.floor(ratio * float(n_reused)))


def select_topk(d, k: int) -> np.ndarray:
    """Rows of the k largest d (ties: lower row first), ascending, int64.

    np.lexsort sorts by the last key first: primary key -d (largest d
    first), secondary key the row index (lower row first).
    """
    d = np.asarray(d, dtype=np.float64)
    n = d.shape[0]
    assert 0 <= k <= n
    rows = np.arange(n, dtype=np.int64)
    d0 = np.where(d == 0.0, 0.0, d)      # -0.0 and +0.0 are equal
    order = np.lexsort((rows, -d0))
    return np.sort(order[:k])


def selection(d, k: int, n_reused: int, n_rows: int) -> np.ndarray:
    """Selected reused rows (top-k by d) followed by every query row."""
    top = select_topk(np.asarray(d)[:n_reused], k)
    return np.concatenate([top, np.arange(n_reused, n_rows, dtype=np.int64)])
