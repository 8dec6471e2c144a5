"""One layer of the selective-recompute prefill (test infrastructure only).

Paper, Section 3.4 and Section 4 setup: per layer the reused chunk caches
are merged into one buffer and moved to their new positions; at the check
layer the keys of all tokens are recomputed, compared with the adjusted
cache, and the tokens with the largest deviation are selected (Section
3.2); the selected tokens' recomputed K/V replace the cached ones and only
their attention is evaluated, causally by position, against the whole
blended cache.  Later layers reuse the selection.

Readings fixed here:
* rows [0, n_reused) hold the reused chunks in order; rows [n_reused, N)
  are the query chunk, always recomputed;
* the adjusted cache is stored in bfloat16 (round to nearest even);
* rows that are not selected keep the adjusted cached K/V even at the
  check layer (ratio 0 leaves the reused cache as adjusted);
* at the check layer the fresh Q/K/V cover all N rows; at a reuse layer
  they cover only the selected rows, in selection order.
"""
import numpy as np

from .bf16 import f64_to_bf16
from .rope import inv_freq as _inv_freq, rope_shift
from .deviation import key_deviation
from .select import recompute_count, selection
from .attention import sparse_query_attention


def blend_prefill_layer(chunk_len, n_query, n_q_heads, n_kv_heads, rope_theta,
                        k_src, v_cache, q_fresh, k_fresh, v_fresh,
                        is_check_layer: bool, ratio: float, sel=None,
                        old_pos0=None, freqs=None, attn_rows=None):
    """Returns a dict with the adjusted and blended cache, selection and output.

    k_src: bfloat16 bits [N, Hkv, D]; rows [0, n_reused) are the cached
    keys at their chunk-local positions (rows beyond are ignored).
    v_cache: bfloat16 bits [N, Hkv, D].
    q_fresh/k_fresh/v_fresh: bfloat16 bits, [N, ...] at the check layer,
    [n_sel, ...] (selection order) otherwise; ``sel`` is required then.
    ``attn_rows`` evaluates the attention for a subset of selected rows.

    Keys of the result: k_shift (bf16 bits [n_reused, Hkv, D]), dev
    (float64 [n_reused] or None), sel (int64 [n_sel]), k_cache, v_cache
    (bf16 bits [N, Hkv, D]), out (float64 [n_sel or len(attn_rows), Hq, D]),
    lse (float64).
    """
    cl = np.asarray(chunk_len, dtype=np.int64)
    n_r = int(cl.sum())
    N = n_r + int(n_query)
    D = np.asarray(k_src).shape[-1]
    f = _inv_freq(D, rope_theta) if freqs is None else np.asarray(freqs)

    k_shift = f64_to_bf16(rope_shift(np.asarray(k_src)[:n_r], cl, f, old_pos0))
    k_cache = np.array(k_src, dtype=np.uint16, copy=True)[:N]
    k_cache[:n_r] = k_shift
    v_out = np.array(v_cache, dtype=np.uint16, copy=True)[:N]

    dev = None
    if is_check_layer:
        k = recompute_count(ratio, n_r)
        if k < 0:
            raise ValueError("ratio outside [0, 1]")
        if k == n_r:
            sel = np.arange(N, dtype=np.int64)   # everything recomputed: causal
        else:
            dev = key_deviation(k_shift, np.asarray(k_fresh)[:n_r])
            sel = selection(dev, k, n_r, N)
        src = sel                                 # fresh tensors are full [N]
    else:
        sel = np.asarray(sel, dtype=np.int64)
        src = np.arange(len(sel))                 # fresh tensors are compact
    k_cache[sel] = np.asarray(k_fresh)[src]
    v_out[sel] = np.asarray(v_fresh)[src]
    q_sel = np.asarray(q_fresh)[src]
    out, lse = sparse_query_attention(q_sel, sel, k_cache, v_out, n_q_heads,
                                      n_kv_heads, rows=attn_rows)
    return dict(k_shift=k_shift, dev=dev, sel=sel, k_cache=k_cache,
                v_cache=v_out, out=out, lse=lse)
