"""Parity at the full 124k-context size, in the launch configuration bench.py
times (one check layer through kvc_blend_prefill_layer), for the headline
16-chunk layout and for a 1,431-chunk document layout with separators.

The oracle computes the adjustment, the exact deviations and the selection
for all 124,000 reused rows (bit-exact comparison), and the attention of a
sample of selected rows one by one: the first rows, the last 16 (query
chunk, the longest), and 32 seeded random rows.  Queries are generated only
for the selected rows (the layer reads no other query row); the other rows
of the query tensor are zero.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from _blend import layout
from _gpu import up, down_bf16, empty_bf16, bytes_buf, within_tol
from _inputs import build, build_q

pytestmark = pytest.mark.gpu
LSE_ATOL = 2.0 ** -8 + 1e-4


@pytest.mark.timeout(400)
@pytest.mark.parametrize("name", ["124k", "qa-124k"])
def test_124k_check_layer(K, name):
    # 124k: 16 chunks of 7,750 rows; qa-124k: 715 documents with two-token
    # zero-K/V separators (1,431 chunks), the same 124,256 rows
    w = W.get(name)
    N, n_r = w.n_rows, w.n_reused
    x = build(w, seed=0, with_q=False)
    f = oracle.inv_freq(w.head_dim, w.rope_theta)
    k_shift = oracle.f64_to_bf16(oracle.rope_shift(x["k_src"][:n_r], w.chunk_len, f))
    dev = oracle.key_deviation(k_shift, x["k_fresh"][:n_r])
    k = oracle.recompute_count(w.ratio, n_r)
    sel = oracle.selection(dev, k, n_r, N)
    q_sel = build_q(w, sel, seed=0)

    L = layout(K, w)
    pb = K.kvc_plan_bytes(L)
    plan = bytes_buf(pb)
    K.kvc_plan_upload(L, plan, pb)
    q = torch.zeros((N, w.n_q_heads, w.head_dim), dtype=torch.int16, device="cuda:0")
    q[torch.from_numpy(sel).cuda()] = up(q_sel)
    k_src, v_cache = up(x["k_src"]), up(x["v_cache"])
    k_cache = empty_bf16(N, w.n_kv_heads, w.head_dim)
    n_sel = len(sel)
    g_sel = torch.full((n_sel,), -1, dtype=torch.int32, device="cuda:0")
    out = empty_bf16(n_sel, w.n_q_heads, w.head_dim)
    lse = torch.empty((n_sel, w.n_q_heads), dtype=torch.float32, device="cuda:0")
    wb = K.kvc_blend_workspace(L)
    ws = bytes_buf(wb)
    K.kvc_blend_prefill_layer(L, plan, True, w.ratio, k_src, k_cache, v_cache, q, up(x["k_fresh"]),
                              up(x["v_fresh"]), g_sel, n_sel, out, lse, ws, wb)
    torch.cuda.synchronize()

    got_sel = g_sel.cpu().numpy().astype(np.int64)
    assert np.array_equal(got_sel, sel)
    assert set(w.zero_rows.tolist()) <= set(got_sel.tolist())
    kc = down_bf16(k_cache)
    vc = down_bf16(v_cache)
    # blended cache: adjusted keys except selected rows, which carry fresh K/V
    want_k = np.array(x["k_src"], copy=True)
    want_k[:n_r] = k_shift
    want_v = np.array(x["v_cache"], copy=True)
    want_k[sel] = x["k_fresh"][sel]
    want_v[sel] = x["v_fresh"][sel]
    assert np.array_equal(oracle.bf16_to_f64(kc), oracle.bf16_to_f64(want_k))
    assert np.array_equal(vc, want_v)

    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([np.arange(4), np.arange(n_sel - 16, n_sel),
                                     rng.choice(n_sel, 32, replace=False)]))
    ref, ref_lse = oracle.sparse_query_attention(q_sel, sel, want_k, want_v, w.n_q_heads, w.n_kv_heads,
                                                 rows=rows)
    got = oracle.bf16_to_f64(down_bf16(out)[rows])
    ok, err = within_tol(got, ref)
    assert ok, f"max attention error {err}"
    assert np.allclose(lse[rows].cpu().numpy(), ref_lse, rtol=0, atol=LSE_ATOL)
