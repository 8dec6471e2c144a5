"""The library's compute entry points under HIP graph capture.

They only enqueue kernels on the caller's stream (no memset nodes, no
synchronisation, no allocation), so a caller can capture whole layers and
replay them.  Each graph is replayed several times with unrelated eager
work and synchronisations between replays, and every replay must equal the
eager result bit for bit (the kernels are deterministic).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from _blend import layout
from _gpu import up, down_bf16, empty_bf16, bytes_buf
from _inputs import build

pytestmark = pytest.mark.gpu


def _eager_noise(n=1 << 20):
    # unrelated eager work between replays (its own buffers)
    a = torch.randn(n, device="cuda:0")
    (a * 2 + 1).sum().item()


@pytest.mark.parametrize("name,split", [("4k", False), ("sep-4k", True)])
def test_check_layer_graph_replays(K, name, split):
    w = W.get(name)
    x = build(w, seed=3)
    L = layout(K, w)
    pb = K.kvc_plan_bytes(L)
    plan = bytes_buf(pb)
    plan = K.kvc_plan_upload(L, plan, pb)
    n_sel = K.kvc_recompute_count(w.ratio, w.n_reused) + w.n_query
    k_src, v0 = up(x["k_src"]), up(x["v_cache"])
    q, kf, vf = up(x["q"]), up(x["k_fresh"]), up(x["v_fresh"])
    k_cache, v_cache = empty_bf16(*x["k_src"].shape), torch.empty_like(v0)
    sel = torch.empty(n_sel, dtype=torch.int32, device="cuda:0")
    out = empty_bf16(n_sel, w.n_q_heads, w.head_dim)
    lse = torch.empty((n_sel, w.n_q_heads), dtype=torch.float32, device="cuda:0")
    wb = K.kvc_blend_workspace(L)
    if split:
        wb += K.kvc_attention_workspace(n_sel, w.n_q_heads, w.n_kv_heads, w.head_dim)
    ws = bytes_buf(wb)

    def layer():
        v_cache.copy_(v0)
        K.kvc_blend_prefill_layer(L, plan, 1, w.ratio, k_src, k_cache, v_cache, q, kf, vf, sel, n_sel,
                                  out, lse, ws, wb)

    layer()
    torch.cuda.synchronize()
    want = [t.clone() for t in (sel, out, lse, k_cache, v_cache)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        layer()                               # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        layer()
    for rep in range(4):
        for t in (sel, out, lse, k_cache, v_cache):
            t.fill_(-1) if t.dtype != torch.float32 else t.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        _eager_noise()
        torch.cuda.synchronize()
        for name_t, got, ref in zip(("sel", "out", "lse", "k_cache", "v_cache"),
                                    (sel, out, lse, k_cache, v_cache), want):
            assert torch.equal(got, ref), (rep, name_t)
    # and the eager result is the oracle's
    r = oracle.blend_prefill_layer(w.chunk_len, w.n_query, w.n_q_heads, w.n_kv_heads, w.rope_theta,
                                   x["k_src"], x["v_cache"], x["q"], x["k_fresh"], x["v_fresh"], True,
                                   w.ratio)
    assert np.array_equal(want[0].cpu().numpy(), r["sel"])


def test_layer_ops_graph_replays(K):
    # norm (gathering), Q/K/V split with RoPE, gated SiLU captured together
    rng = np.random.default_rng(5)
    N, hid, inter, n_sel = 900, 4096, 14336, 200
    h = up(oracle.f64_to_bf16(rng.standard_normal((N, hid))))
    g = up(oracle.f64_to_bf16(1 + 0.1 * rng.standard_normal(hid)))
    rows = up(np.sort(rng.choice(N, n_sel, replace=False)).astype(np.int32))
    y = up(oracle.f64_to_bf16(rng.standard_normal((n_sel, 48 * 128))))
    gu = up(oracle.f64_to_bf16(rng.standard_normal((n_sel, 2 * inter)) * 2))
    xs, hs = empty_bf16(n_sel, hid), empty_bf16(n_sel, hid)
    q, k, v = empty_bf16(n_sel, 32, 128), empty_bf16(n_sel, 8, 128), empty_bf16(n_sel, 8, 128)
    act = empty_bf16(n_sel, inter)
    outs = (xs, hs, q, k, v, act)

    def ops():
        K.kvc_rms_norm(h, N, rows, n_sel, hid, g, 1e-5, xs, hs)
        K.kvc_qkv_rope(y, n_sel, 32, 8, 8, 128, rows, 500000.0, q, k, v)
        K.kvc_swiglu(gu, n_sel, inter, act)

    ops()
    torch.cuda.synchronize()
    want = [t.clone() for t in outs]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ops()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        ops()
    for rep in range(4):
        for t in outs:
            t.fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        _eager_noise()
        torch.cuda.synchronize()
        for i, (got, ref) in enumerate(zip(outs, want)):
            assert torch.equal(got, ref), (rep, i)
