"""GPU parity of the whole layer (kvc_blend_prefill_layer) against the oracle.

Selection indices and blended caches bit-exact; attention outputs within
2e-2 abs + 1e-2 rel; LSE within ln(1 + 2^-8) + 1e-4 (see LSE_ATOL).
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as W
from _blend import gpu_layer, oracle_layer, layout
from _gpu import within_tol, LSE_ATOL
from _inputs import build

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


def _vals(bits):
    return oracle.bf16_to_f64(bits)


def _compare(g, r, rows=None):
    assert np.array_equal(g["sel"], r["sel"])
    N = r["k_cache"].shape[0]
    assert np.array_equal(_vals(g["k_cache"][:N]), _vals(r["k_cache"]))
    assert np.array_equal(g["v_cache"][:N], r["v_cache"])
    go = _vals(g["out"]) if rows is None else _vals(g["out"][rows])
    ok, err = within_tol(go, r["out"])
    assert ok, f"max attention error {err}"
    gl = g["lse"] if rows is None else g["lse"][rows]
    assert np.allclose(gl, r["lse"], rtol=0, atol=LSE_ATOL)


def test_tiny_check_layer_matches_oracle_and_fixture(K):
    w = W.get("tiny")
    x = build(w, seed=0)
    g = gpu_layer(K, w, x, True, w.ratio)
    r = oracle_layer(w, x, True, w.ratio)
    _compare(g, r)
    with open(os.path.join(HERE, "golden", "tiny_seed0.json")) as fh:
        assert g["sel"].tolist() == json.load(fh)["sel"]


def test_tiny_reuse_layer_and_in_place(K):
    w = W.get("tiny")
    x0 = build(w, seed=0, layer=0)
    sel = oracle_layer(w, x0, True, w.ratio)["sel"]
    x1 = build(w, seed=0, layer=1)
    xc = dict(x1, q=x1["q"][sel], k_fresh=x1["k_fresh"][sel], v_fresh=x1["v_fresh"][sel])
    r = oracle_layer(w, xc, False, w.ratio, sel=sel)
    for in_place in (False, True):
        g = gpu_layer(K, w, xc, False, w.ratio, sel_in=sel, in_place=in_place)
        _compare(g, r)


@pytest.mark.parametrize("ratio", [0.0, 0.05, 0.3, 1.0])
def test_tiny_ratio_sweep(K, ratio):
    w = W.get("tiny")
    x = build(w, seed=1)
    g = gpu_layer(K, w, x, True, ratio)
    r = oracle_layer(w, x, True, ratio)
    _compare(g, r)
    n_r = w.n_reused
    if ratio == 0.0:
        assert np.array_equal(g["v_cache"][:n_r], x["v_cache"][:n_r])
    if ratio == 1.0:
        ref, _ = oracle.causal_attention(x["q"], x["k_fresh"], x["v_fresh"], w.n_q_heads, w.n_kv_heads)
        ok, err = within_tol(_vals(g["out"]), ref)
        assert ok, err


def test_structured_ragged_layout_with_old_positions(K):
    # attention-sink-like deviations on each chunk's first tokens, ragged
    # chunks, cached positions not starting at 0, G = 4 with 4 kv heads
    w = W.Workload("ragged", (300, 1, 77, 512, 129), 33, 16, 4, structured=True,
                   chunk_old_pos0=(0, 5, 1000, 0, 77))
    x = build(w, seed=2)
    g = gpu_layer(K, w, x, True, 0.15)
    r = oracle_layer(w, x, True, 0.15)
    _compare(g, r)


@pytest.mark.parametrize("seed", range(12))
def test_random_layouts(K, seed):
    # seeded random requests: 1-40 chunks of 0-300 rows, 0-100 query rows,
    # 1-8 kv heads, groups 1-4, cached positions from 0 or elsewhere, ratios
    # from 0 to 1; check layer, then a reuse layer on its selection
    rng = np.random.default_rng(500 + seed)
    n_chunks = int(rng.integers(1, 41))
    cl = tuple(int(c) for c in rng.integers(0, 301, n_chunks))
    hkv = int(rng.choice([1, 2, 4, 8]))
    old = tuple(int(o) for o in rng.integers(0, 5000, n_chunks)) if seed % 2 else None
    ratio = [0.0, 1.0][seed % 2] if seed % 5 == 0 else float(rng.uniform(0.01, 0.6))
    w = W.Workload(f"random{seed}", cl, int(rng.integers(0, 101)), hkv * int(rng.choice([1, 2, 4])), hkv,
                   ratio=ratio, structured=bool(seed % 3 == 0), chunk_old_pos0=old)
    if w.n_rows == 0:
        pytest.skip("empty request")
    x = build(w, seed=seed)
    g = gpu_layer(K, w, x, True, ratio)
    r = oracle_layer(w, x, True, ratio)
    _compare(g, r)
    sel = r["sel"]
    if len(sel):
        xc = dict(x, q=x["q"][sel], k_fresh=x["k_fresh"][sel], v_fresh=x["v_fresh"][sel])
        g2 = gpu_layer(K, w, xc, False, ratio, sel_in=sel)
        _compare(g2, oracle_layer(w, xc, False, ratio, sel=sel))


def test_4k_check_layer(K):
    w = W.get("4k")
    x = build(w, seed=0)
    g = gpu_layer(K, w, x, True, w.ratio)
    r = oracle_layer(w, x, True, w.ratio)
    _compare(g, r)


def test_layer_is_deterministic(K):
    w = W.get("4k")
    x = build(w, seed=3)
    a = gpu_layer(K, w, x, True, w.ratio)
    b = gpu_layer(K, w, x, True, w.ratio)
    for key in ("sel", "out", "lse", "k_cache", "v_cache"):
        assert np.array_equal(a[key], b[key]), key


@pytest.mark.parametrize("ratio", [0.05, 0.15, 0.3, 1.0])
def test_32k_check_layer_sampled_rows(K, ratio):
    w = W.get("32k")
    x = build(w, seed=0)
    g = gpu_layer(K, w, x, True, ratio)
    n_sel = len(g["sel"])
    rng = np.random.default_rng(int(ratio * 100))
    rows = np.unique(np.concatenate([[0, 1, n_sel - 1], np.arange(n_sel - 40, n_sel),
                                     rng.choice(n_sel, 40, replace=False)]))
    r = oracle_layer(w, x, True, ratio, attn_rows=rows)
    _compare(g, r, rows=rows)


@pytest.mark.parametrize("name", ["sep-tiny", "sep-4k"])
def test_document_layout_with_zero_separators(K, name):
    # documents of mixed length with two-token zero-K/V separator slots
    # (Section 3.1): many chunks, ragged shift tiles, zero rows in the cache
    w = W.get(name)
    x = build(w, seed=4)
    g = gpu_layer(K, w, x, True, w.ratio)
    r = oracle_layer(w, x, True, w.ratio)
    _compare(g, r)
    assert set(w.zero_rows.tolist()) <= set(g["sel"].tolist())
    # separators not selected would keep zero K/V; all are selected here, so
    # every separator row carries its recomputed K/V
    z = w.zero_rows
    assert np.array_equal(g["v_cache"][z], x["v_fresh"][z])


@pytest.mark.parametrize("ratio", [0.05, 0.15])
def test_qa_32k_document_layout_sampled_rows(K, ratio):
    # 179 documents, 359 chunks at 32k rows
    w = W.get("qa-32k")
    x = build(w, seed=0)
    g = gpu_layer(K, w, x, True, ratio)
    n_sel = len(g["sel"])
    rng = np.random.default_rng(int(ratio * 1000) + 1)
    rows = np.unique(np.concatenate([[0, 1, n_sel - 1], np.arange(n_sel - 40, n_sel),
                                     rng.choice(n_sel, 40, replace=False)]))
    r = oracle_layer(w, x, True, ratio, attn_rows=rows)
    _compare(g, r, rows=rows)


def test_32k_five_percent_layer_with_split_attention(K):
    # 1,856 selected rows fill only 232 workgroups: with the layer workspace
    # enlarged by the attention's share the key ranges are split
    import torch
    from _gpu import up, down_bf16, empty_bf16, bytes_buf
    w = W.get("32k")
    ratio = 0.05
    x = build(w, seed=0)
    L = layout(K, w)
    pb = K.kvc_plan_bytes(L)
    plan = bytes_buf(pb)
    plan = K.kvc_plan_upload(L, plan, pb)
    n_sel = K.kvc_recompute_count(ratio, w.n_reused) + w.n_query
    extra = K.kvc_attention_workspace(n_sel, w.n_q_heads, w.n_kv_heads, 128)
    assert extra > 0
    wb = K.kvc_blend_workspace(L) + extra
    ws = bytes_buf(wb)
    k_cache = empty_bf16(w.n_rows, w.n_kv_heads, 128)
    v_cache = up(x["v_cache"])
    sel = torch.full((n_sel,), -1, dtype=torch.int32, device="cuda:0")
    out = empty_bf16(n_sel, w.n_q_heads, 128)
    lse = torch.empty((n_sel, w.n_q_heads), dtype=torch.float32, device="cuda:0")
    K.kvc_blend_prefill_layer(L, plan, True, ratio, up(x["k_src"]), k_cache, v_cache, up(x["q"]), up(x["k_fresh"]),
                              up(x["v_fresh"]), sel, n_sel, out, lse, ws, wb)
    torch.cuda.synchronize()
    g = dict(sel=sel.cpu().numpy().astype(np.int64), out=down_bf16(out), lse=lse.cpu().numpy(),
             k_cache=down_bf16(k_cache), v_cache=down_bf16(v_cache))
    rng = np.random.default_rng(5)
    rows = np.unique(np.concatenate([[0, 1, n_sel - 1], np.arange(n_sel - 40, n_sel),
                                     rng.choice(n_sel, 40, replace=False)]))
    r = oracle_layer(w, x, True, ratio, attn_rows=rows)
    _compare(g, r, rows=rows)


def _layers(K, w, n_layers, check_at, seed=7):
    """Run a multi-layer prefill through the C ABI; layers before `check_at`
    are fully recomputed (ratio 1), `check_at` selects, later layers reuse."""
    import torch
    from _gpu import up, down_bf16, empty_bf16, bytes_buf
    from _blend import layout
    L = layout(K, w)
    pb = K.kvc_plan_bytes(L)
    plan = bytes_buf(pb)
    plan = K.kvc_plan_upload(L, plan, pb)
    wb = K.kvc_blend_workspace(L)
    ws = bytes_buf(wb)
    n_sel = K.kvc_recompute_count(w.ratio, w.n_reused) + w.n_query
    sel = torch.full((n_sel,), -1, dtype=torch.int32, device="cuda:0")
    outs, sels, inputs = [], [], []
    for layer in range(n_layers):
        x = build(w, seed=seed, layer=layer)
        if layer < check_at:
            ratio, is_check, ns = 1.0, True, w.n_rows
            sl = torch.empty(ns, dtype=torch.int32, device="cuda:0")
            q, kf, vf = x["q"], x["k_fresh"], x["v_fresh"]
        elif layer == check_at:
            ratio, is_check, ns, sl = w.ratio, True, n_sel, sel
            q, kf, vf = x["q"], x["k_fresh"], x["v_fresh"]
        else:
            ratio, is_check, ns, sl = w.ratio, False, n_sel, sel
            s_np = sels[check_at]
            q, kf, vf = x["q"][s_np], x["k_fresh"][s_np], x["v_fresh"][s_np]
            x = dict(x, q=q, k_fresh=kf, v_fresh=vf)
        k_src = up(x["k_src"])
        k_cache = empty_bf16(*x["k_src"].shape)
        v_cache = up(x["v_cache"])
        out = empty_bf16(ns, w.n_q_heads, w.head_dim)
        lse = torch.empty((ns, w.n_q_heads), dtype=torch.float32, device="cuda:0")
        K.kvc_blend_prefill_layer(L, plan, is_check, ratio, k_src, k_cache, v_cache, up(q), up(kf), up(vf),
                                  sl, ns, out, lse, ws, wb)
        torch.cuda.synchronize()
        sels.append(sl.cpu().numpy().astype(np.int64))
        outs.append(oracle.bf16_to_f64(down_bf16(out)))
        inputs.append((x, is_check, ratio))
    return outs, sels, inputs


@pytest.mark.parametrize("check_at", [0, 1])
def test_multi_layer_prefill_reuses_the_selection(K, check_at):
    # layer `check_at` selects; later layers reuse its selection (the
    # 32-layer configuration in miniature); with check_at = 1 the first layer
    # is fully recomputed (causal), as the paper does for its 0th layer
    w = W.get("tiny")
    outs, sels, inputs = _layers(K, w, 4, check_at)
    for layer, (x, is_check, ratio) in enumerate(inputs):
        sel = None if layer <= check_at else sels[check_at]
        r = oracle_layer(w, x, is_check, ratio, sel=sel)
        assert np.array_equal(sels[layer] if layer <= check_at else sels[check_at], r["sel"])
        ok, err = within_tol(outs[layer], r["out"])
        assert ok, (layer, err)
    for layer in range(check_at + 1, 4):
        assert np.array_equal(sels[layer], sels[check_at])   # selection untouched
