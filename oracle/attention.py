"""Causal GQA attention of sparse queries (test infrastructure only).

Paper: in the recompute stage only the selected tokens' queries are
evaluated, against the whole concatenated cache, with a custom mask
(Section 4 setup); the mask must be causal by the tokens' original
positions -- without it a selected token attends to keys after it and
quality drops (Limitations, item 1).  Recomputing every token is plain
causal attention (Section 4 setup, the fully recomputed layer).

Definition, for selected query i at position p_i and query head h with
kv head g = h // (Hq / Hkv) (grouped-query attention as in Llama):
    s_j  = scale * <q[i,h], k[j,g]>          for keys j = 0 .. p_i
    O    = sum_j softmax(s)_j v[j,g]
    LSE  = log sum_j exp(s_j)
The softmax is evaluated in float64 with its maximum subtracted.
"""
import numpy as np

from .bf16 import bf16_to_f64


def _f64(x):
    x = np.asarray(x)
    return bf16_to_f64(x) if x.dtype == np.uint16 else x.astype(np.float64)


def sparse_query_attention(q, pos, k, v, n_q_heads: int, n_kv_heads: int,
                           scale=None, rows=None):
    """O [n_sel, Hq, D] and LSE [n_sel, Hq] in float64.

    q: [n_sel, Hq, D]; pos: [n_sel] int; k, v: [n_kv, Hkv, D]; bfloat16 bits
    (uint16) or floats.  ``rows`` restricts the evaluation to a subset of
    the queries (their outputs are returned in that order).  A query with
    no visible key (p_i < 0) gets O = 0 and LSE = -inf.
    """
    q = _f64(q)
    k = _f64(k)
    v = _f64(v)
    pos = np.asarray(pos, dtype=np.int64)
    n_sel, Hq, D = q.shape
    assert Hq == n_q_heads and n_q_heads % n_kv_heads == 0
    G = n_q_heads // n_kv_heads
    n_kv = k.shape[0]
    if scale is None or scale == 0:
        scale = 1.0 / np.sqrt(D)
    idx = np.arange(n_sel) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.zeros((len(idx), Hq, D))
    lse = np.full((len(idx), Hq), -np.inf)
    for o, i in enumerate(idx):
        p = int(min(pos[i], n_kv - 1))
        if p < 0:
            continue
        for g in range(n_kv_heads):
            qg = q[i, g * G:(g + 1) * G, :]            # [G, D]
            kg = k[: p + 1, g, :]                      # [p+1, D]
            vg = v[: p + 1, g, :]
            s = (qg @ kg.T) * scale                    # [G, p+1]
            m = s.max(axis=1, keepdims=True)
            e = np.exp(s - m)
            z = e.sum(axis=1, keepdims=True)
            out[o, g * G:(g + 1) * G, :] = (e @ vg) / z
            lse[o, g * G:(g + 1) * G] = (m + np.log(z))[:, 0]
    return out, lse


def causal_attention(q, k, v, n_q_heads: int, n_kv_heads: int, scale=None):
    """Plain causal attention of every row: sparse attention with p_i = i."""
    n = np.asarray(q).shape[0]
    return sparse_query_attention(q, np.arange(n), k, v, n_q_heads, n_kv_heads, scale)
