"""Pins for one layer of the selective-recompute prefill in the oracle.

* Block-attention equivalence (Section 2 and Section 3.2: chunks with no
  cross-attention, final chunk attending to everything): per-chunk causal
  attention at local positions, then the position adjustment, then the
  query chunk over the whole cache, equals a brute-force masked softmax
  with the block-diagonal + all-attending-final-rows mask at global
  positions.  RoPE scores depend only on relative position, so the two
  agree up to rounding.
* Ratio 1.0 is plain causal attention over the recomputed K/V (Section 4,
  fully recomputed layer); ratio 0 leaves the reused cache as adjusted.
"""
import numpy as np

import oracle
from oracle import (inv_freq, rope_rotate, rope_shift, causal_attention,
                    sparse_query_attention, blend_prefill_layer, f64_to_bf16,
                    bf16_to_f64, key_deviation)


def test_block_attention_mask_equivalence():
    rng = np.random.default_rng(0)
    chunk_len, n_query = [5, 7, 4], 3
    hq, hkv, D, theta = 4, 2, 16, 500000.0
    n_r = sum(chunk_len); N = n_r + n_query
    G = hq // hkv
    f = inv_freq(D, theta)
    q_raw = rng.standard_normal((N, hq, D))
    k_raw = rng.standard_normal((N, hkv, D))
    v = rng.standard_normal((N, hkv, D))
    glob = np.arange(N)
    local = np.concatenate([np.arange(L) for L in chunk_len] + [np.arange(n_r, N)])
    chunk_id = np.concatenate([[c] * L for c, L in enumerate(chunk_len)] + [[-1] * n_query])

    # brute force at global positions with the block-attention mask
    qg, kg = rope_rotate(q_raw, glob, f), rope_rotate(k_raw, glob, f)
    s = np.einsum("ihd,jhd->hij", qg, np.repeat(kg, G, axis=1)) / np.sqrt(D)
    allowed = np.tril(np.ones((N, N), bool))
    same = (chunk_id[:, None] == chunk_id[None, :])
    allowed &= same | (chunk_id[:, None] == -1)
    s = np.where(allowed[None], s, -np.inf)
    p = np.exp(s - s.max(-1, keepdims=True)); p /= p.sum(-1, keepdims=True)
    brute = np.einsum("hij,jhd->ihd", p, np.repeat(v, G, axis=1))

    # oracle path: each chunk alone at local positions ...
    out = np.zeros((N, hq, D))
    r0 = 0
    for L in chunk_len:
        sl = slice(r0, r0 + L)
        ql, kl = rope_rotate(q_raw[sl], local[sl], f), rope_rotate(k_raw[sl], local[sl], f)
        out[sl] = causal_attention(ql, kl, v[sl], hq, hkv)[0]
        r0 += L
    # ... then the cached keys are moved and the query chunk attends to all
    k_cached = rope_rotate(k_raw[:n_r], local[:n_r], f)
    k_all = np.concatenate([rope_shift(k_cached, chunk_len, f), kg[n_r:]])
    out[n_r:] = sparse_query_attention(qg[n_r:], glob[n_r:], k_all, v, hq, hkv)[0]
    assert np.allclose(out, brute, rtol=0, atol=1e-10)


def _case(seed=0, chunk_len=(40, 33, 51), n_query=9, hq=8, hkv=2, D=32):
    rng = np.random.default_rng(seed)
    n_r = sum(chunk_len); N = n_r + n_query
    f = inv_freq(D, 500000.0)
    local = np.concatenate([np.arange(L) for L in chunk_len] + [np.zeros(n_query, int)])
    k_raw = rng.standard_normal((N, hkv, D))
    noise = 0.1 * rng.standard_normal((N, hkv, D))
    k_src = f64_to_bf16(rope_rotate(k_raw, local, f))
    k_fresh = f64_to_bf16(rope_rotate(k_raw + noise, np.arange(N), f))
    v = f64_to_bf16(rng.standard_normal((N, hkv, D)))
    v_fresh = f64_to_bf16(bf16_to_f64(v) + 0.1 * rng.standard_normal((N, hkv, D)))
    q = f64_to_bf16(rope_rotate(rng.standard_normal((N, hq, D)), np.arange(N), f))
    return dict(chunk_len=list(chunk_len), n_query=n_query, n_q_heads=hq, n_kv_heads=hkv,
                rope_theta=500000.0, k_src=k_src, v_cache=v, q_fresh=q, k_fresh=k_fresh,
                v_fresh=v_fresh)


def test_ratio_one_is_causal_attention_over_fresh_kv():
    c = _case(1)
    r = blend_prefill_layer(**c, is_check_layer=True, ratio=1.0)
    N = len(c["q_fresh"])
    assert list(r["sel"]) == list(range(N))
    ref, ref_lse = causal_attention(c["q_fresh"], c["k_fresh"], c["v_fresh"], 8, 2)
    assert np.array_equal(r["out"], ref) and np.array_equal(r["lse"], ref_lse)


def test_ratio_zero_keeps_reused_cache():
    c = _case(2)
    r = blend_prefill_layer(**c, is_check_layer=True, ratio=0.0)
    n_r = sum(c["chunk_len"]); N = n_r + c["n_query"]
    assert list(r["sel"]) == list(range(n_r, N))
    assert np.array_equal(r["v_cache"][:n_r], c["v_cache"][:n_r])
    assert np.array_equal(r["k_cache"][:n_r], r["k_shift"])
    assert r["out"].shape[0] == c["n_query"]


def test_check_layer_selects_largest_deviation_and_blends():
    c = _case(3)
    r = blend_prefill_layer(**c, is_check_layer=True, ratio=0.15)
    n_r = sum(c["chunk_len"]); N = n_r + c["n_query"]
    k = int(np.floor(0.15 * n_r))
    d = key_deviation(r["k_shift"], c["k_fresh"][:n_r])
    assert np.array_equal(d, r["dev"])
    top = r["sel"][:k]
    rest = np.setdiff1d(np.arange(n_r), top)
    assert d[top].min() >= d[rest].max()
    # recomputed rows carry fresh K/V; the others the adjusted cache
    assert np.array_equal(r["k_cache"][top], c["k_fresh"][top])
    assert np.array_equal(r["v_cache"][top], c["v_fresh"][top])
    assert np.array_equal(r["k_cache"][rest], r["k_shift"][rest])
    # the adjusted cache is the float64 shift rounded once to bfloat16
    f = inv_freq(32, 500000.0)
    assert np.array_equal(r["k_shift"], f64_to_bf16(rope_shift(c["k_src"][:n_r], c["chunk_len"], f)))


def test_reuse_layer_takes_compact_fresh_rows_in_selection_order():
    c = _case(4)
    chk = blend_prefill_layer(**c, is_check_layer=True, ratio=0.3)
    sel = chk["sel"]
    c2 = _case(5)        # another layer: different cache and fresh tensors
    comp = dict(c2)
    comp["q_fresh"] = c2["q_fresh"][sel]
    comp["k_fresh"] = c2["k_fresh"][sel]
    comp["v_fresh"] = c2["v_fresh"][sel]
    r = blend_prefill_layer(**comp, is_check_layer=False, ratio=0.3, sel=sel)
    full = blend_prefill_layer(**c2, is_check_layer=True, ratio=1.0)
    # attention over the blended cache, evaluated independently
    kc = np.array(r["k_cache"]); vc = np.array(r["v_cache"])
    ref, _ = sparse_query_attention(c2["q_fresh"][sel], sel, kc, vc, 8, 2)
    assert np.array_equal(r["out"], ref)
    assert np.array_equal(kc[sel], c2["k_fresh"][sel])
    assert not np.allclose(r["out"], full["out"][sel])   # non-selected rows differ


def test_separator_rows_are_selected_first():
    # zero cached K makes a separator row's deviation the squared norm of
    # its recomputed key, far above the noise-level deviation of document
    # rows, so at a 15 % ratio every separator row is recomputed (the large
    # separator deviations the paper reports, Section 3.2)
    import workloads as W
    from _inputs import build
    w = W.get("sep-tiny")
    x = build(w, seed=0)
    r = oracle.blend_prefill_layer(w.chunk_len, w.n_query, w.n_q_heads, w.n_kv_heads, w.rope_theta,
                                   x["k_src"], x["v_cache"], x["q"], x["k_fresh"], x["v_fresh"],
                                   True, w.ratio, attn_rows=np.arange(4))
    assert set(w.zero_rows.tolist()) <= set(r["sel"].tolist())
