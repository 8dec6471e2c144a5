"""Test-side construction of bfloat16 inputs from the seeded raw draws.

The raw draws come from ``workloads`` (random numbers only).  The model's
positional encoding of cached keys (chunk-local positions), recomputed keys
and queries (global positions) is applied here with the oracle's RoPE, and
the results rounded to bfloat16 with the oracle's rounding.  Nothing here
comes from the HIP library.
"""
import numpy as np

import workloads as W
from oracle import inv_freq, rope_rotate, f64_to_bf16


def local_positions(w):
    return np.concatenate([np.arange(L, dtype=np.int64) for L in w.chunk_len]
                          + [np.arange(w.n_reused, w.n_rows, dtype=np.int64)])


def build(w, seed=0, layer=0, q_rows=None, with_q=True):
    """bf16 bit arrays of one layer: k_src, v_cache, k_fresh, v_fresh, q (all N rows
    unless ``q_rows`` is given)."""
    raw = W.draw_raw(w, seed, layer, q_rows=q_rows, parts=("k", "v", "q") if with_q else ("k", "v"))
    f = inv_freq(w.head_dim, w.rope_theta)
    N = w.n_rows
    pos_local = local_positions(w)
    if w.chunk_old_pos0 is not None:
        # cached keys were encoded starting at old_pos0 of their chunk
        off = np.repeat(np.asarray(w.chunk_old_pos0, dtype=np.int64), w.chunk_len)
        pos_local = pos_local.copy()
        pos_local[:w.n_reused] += off
    glob = np.arange(N, dtype=np.int64)
    out = {}
    out["k_src"] = f64_to_bf16(rope_rotate(raw["k_raw"], pos_local, f))
    out["k_fresh"] = f64_to_bf16(rope_rotate(raw["k_raw"].astype(np.float64) + raw["k_noise"], glob, f))
    out["v_cache"] = W.f32_to_bf16_bits(raw["v"])
    out["v_fresh"] = W.f32_to_bf16_bits(raw["v"] + raw["v_noise"])
    z = w.zero_rows
    if len(z):
        # separator slots: cached K/V all zero (recomputed K/V as drawn)
        out["k_src"][z] = 0
        out["v_cache"][z] = 0
    if with_q:
        rows = glob if q_rows is None else np.asarray(q_rows, dtype=np.int64)
        out["q"] = f64_to_bf16(rope_rotate(raw["q_raw"], rows, f))
    return out


def build_q(w, rows, seed=0, layer=0):
    """bf16 bits of the queries of the given rows only (global positions)."""
    raw = W.draw_raw(w, seed, layer, q_rows=rows, parts=("q",))
    f = inv_freq(w.head_dim, w.rope_theta)
    return f64_to_bf16(rope_rotate(raw["q_raw"], np.asarray(rows, dtype=np.int64), f))
