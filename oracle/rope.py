"""RoPE position adjustment of reused chunk keys (test infrastructure only).

Paper: a precomputed chunk cache is built at the chunk's own positions; when
chunks are concatenated, each chunk's keys are moved to the positions they
take in the new context (Section 1; Section 2, PIE's positional alignment
for RoPE), after the per-chunk caches are merged into one buffer (Section
3.4).  This adjustment runs in higher precision than the bfloat16 model
(Section 4, inference setup).

RoPE (Su et al.) in the half-split form of the Llama models the paper uses:
for a head vector x of size D and position p, pair (x[j], x[j + D/2]) is
rotated by the angle p * f_j with f_j = theta ** (-2 j / D), j < D/2.
Rotations by angles a and b compose to a rotation by a + b, so moving a key
cached at position p to p + delta is one rotation by delta * f_j.
"""
import numpy as np

from .bf16 import bf16_to_f64


def inv_freq(head_dim: int, theta: float, override=None) -> np.ndarray:
    """f_j = theta ** (-2 j / D) for j < D/2, float64 (or a caller's table).

    ``override`` stands for a model whose RoPE rescales the frequencies
    (Llama-3.1 scaling, YaRN for Qwen2.5 in Section 4.1).
    """
    if override is not None:
        f = np.asarray(override, dtype=np.float64)
        assert f.shape == (head_dim // 2,)
        return f
    j = np.arange(head_dim // 2, dtype=np.float64)
    return np.float64(theta) ** (-(2.0 * j) / head_dim)


def rope_rotate(x, pos, freqs) -> np.ndarray:
    """Rotate every head vector of row r by the angles pos[r] * f_j.

    x: [rows, heads, D] float64, pos: [rows] (integers, may be negative).
    Returns float64 [rows, heads, D]:
      out[j]       = x[j] cos(a_j) - x[j + D/2] sin(a_j)
      out[j + D/2] = x[j + D/2] cos(a_j) + x[j] sin(a_j)
    """
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    h = D // 2
    ang = np.asarray(pos, dtype=np.float64)[:, None] * np.asarray(freqs)[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    a, b = x[..., :h], x[..., h:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def chunk_row0(chunk_len) -> np.ndarray:
    """First row of each reused chunk in the concatenated context (int64)."""
    cl = np.asarray(chunk_len, dtype=np.int64)
    return np.concatenate([[0], np.cumsum(cl)[:-1]]).astype(np.int64)


def chunk_delta(chunk_len, old_pos0=None) -> np.ndarray:
    """Position shift of each chunk: new first position minus cached one.

    The new position of row r is r.  A chunk cache is computed on its own,
    so by default its first token sits at position 0 (old_pos0 = 0); the
    first chunk then keeps its positions (delta 0), which is the prefix
    caching case of Section 1.
    """
    r0 = chunk_row0(chunk_len)
    if old_pos0 is None:
        return r0
    return r0 - np.asarray(old_pos0, dtype=np.int64)


def rope_shift(k_cached, chunk_len, freqs, old_pos0=None) -> np.ndarray:
    """Move every reused chunk's cached keys to their new positions.

    k_cached: bfloat16 bits (uint16) or float64, [n_reused, Hkv, D], the
    chunks concatenated in order.  Returns float64 [n_reused, Hkv, D]: the
    rows of chunk i rotated by delta_i * f_j.  Values are untouched.
    """
    k = np.asarray(k_cached)
    kf = bf16_to_f64(k) if k.dtype == np.uint16 else np.asarray(k, dtype=np.float64)
    cl = np.asarray(chunk_len, dtype=np.int64)
    assert kf.shape[0] == int(cl.sum())
    delta_per_row = np.repeat(chunk_delta(cl, old_pos0), cl)
    return rope_rotate(kf, delta_per_row, freqs)
