"""GPU checks of the layer-wise pipeline's transfer stage (kvc_stage_layer,
kvc_stage_layers) against the oracle: chunk caches from host (pinned) or
device memory are merged into the device cache, separator slots get zeros
and keys are adjusted in place, equal to the oracle's adjustment; a
two-stream pipeline (staging on a copy stream, each layer's computation
waiting for its own event) matches the oracle's layers, and, bit for bit,
the layer-by-layer path."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from _blend import gpu_layer, oracle_layer
from _gpu import up, down_bf16, empty_bf16, bytes_buf, within_tol, LSE_ATOL
from _inputs import build

pytestmark = pytest.mark.gpu


def _val(bits):
    # keys compare by value: rotating a zero key can give -0.0, the zeros
    # written for a separator slot are +0.0
    return oracle.bf16_to_f64(bits)


def _oracle_staged_k(w, k_src):
    """The oracle's adjusted keys of the reused rows, +0 in separator rows."""
    k = oracle.rope_shift(k_src[:w.n_reused], w.chunk_len, oracle.inv_freq(w.head_dim, w.rope_theta),
                          w.chunk_old_pos0)
    k = oracle.bf16_to_f64(oracle.f64_to_bf16(k))
    k[w.zero_rows] = 0.0
    return k


def _layout_plan(K, w, zero=True):
    L = K.Layout(w.chunk_len, w.n_query, w.n_q_heads, w.n_kv_heads, w.head_dim, w.rope_theta,
                 chunk_old_pos0=w.chunk_old_pos0, zero_kv=w.zero_kv_flags if zero else None)
    pb = K.kvc_plan_bytes(L)
    plan = bytes_buf(pb)
    plan = K.kvc_plan_upload(L, plan, pb)
    return L, plan


def _chunk_sources(w, arr, kind, keep):
    """Pointers to each chunk's rows of arr ([n_reused, Hkv, D] uint16): separate
    pinned tensors, views of one pinned buffer, or device tensors.  Zero-K/V
    chunks get None, except with "pinned_one_buffer_bridged", where they point
    into the buffer too (whose separator rows then hold junk, which staging
    must overwrite with zeros).  Tensors are appended to keep (alive until
    the copies ran)."""
    row0 = np.concatenate([[0], np.cumsum(w.chunk_len)[:-1]])
    zero = set(w.zero_kv_chunks)
    if kind.startswith("pinned_one_buffer"):
        host = np.ascontiguousarray(arr).copy()
        bridged = kind.endswith("bridged")
        if bridged:
            host[w.zero_rows] = 0x3F80          # 1.0: not what a separator holds
        buf = torch.from_numpy(host.view(np.int16)).pin_memory()
        keep.append(buf)
        rb = arr.shape[1] * arr.shape[2] * 2
        return [None if (i in zero and not bridged) else buf.data_ptr() + int(row0[i]) * rb
                for i in range(len(w.chunk_len))]
    out = []
    for i, n in enumerate(w.chunk_len):
        if i in zero:
            out.append(None)
            continue
        part = np.ascontiguousarray(arr[row0[i]:row0[i] + n]).view(np.int16)
        t = torch.from_numpy(part).pin_memory() if kind == "pinned_chunks" else torch.from_numpy(part).cuda()
        keep.append(t)
        out.append(t)
    return out


@pytest.mark.parametrize("kind", ["pinned_chunks", "pinned_one_buffer", "pinned_one_buffer_bridged", "device"])
def test_stage_layer_merges_zero_fills_and_adjusts(K, kind):
    w = W.get("sep-4k").with_(chunk_old_pos0=None)
    x = build(w, seed=5, with_q=False)
    L, plan = _layout_plan(K, w)
    N, n_r = w.n_rows, w.n_reused
    keep = []
    kp = _chunk_sources(w, x["k_src"][:n_r], kind, keep)
    vp = _chunk_sources(w, x["v_cache"][:n_r], kind, keep)
    sentinel = 0x1234
    kc = torch.full((N, w.n_kv_heads, w.head_dim), sentinel, dtype=torch.int16, device="cuda:0")
    vc = torch.full_like(kc, sentinel)
    K.kvc_stage_layer(L, plan, kp, vp, kc, vc)
    torch.cuda.synchronize()
    g_k, g_v = down_bf16(kc), down_bf16(vc)
    assert np.array_equal(_val(g_k[:n_r]), _oracle_staged_k(w, x["k_src"]))
    assert np.array_equal(g_v[:n_r], x["v_cache"][:n_r])
    z = w.zero_rows
    assert len(z) > 0 and not g_k[z].any() and not g_v[z].any()      # separators: exact zeros
    assert np.all(g_k[n_r:] == sentinel) and np.all(g_v[n_r:] == sentinel)  # query rows untouched


def test_stage_layer_without_zero_flags_copies_every_chunk(K):
    # the same layout with no zero_kv flags: separator rows are ordinary
    # (zero-valued) chunks and need their own sources
    w = W.get("sep-tiny")
    x = build(w, seed=6, with_q=False)
    L, plan = _layout_plan(K, w, zero=False)
    n_r = w.n_reused
    w_all = w.with_(zero_kv_chunks=())
    keep = []
    kp = _chunk_sources(w_all, x["k_src"][:n_r], "pinned_chunks", keep)
    vp = _chunk_sources(w_all, x["v_cache"][:n_r], "pinned_chunks", keep)
    kc, vc = empty_bf16(w.n_rows, w.n_kv_heads, 128), empty_bf16(w.n_rows, w.n_kv_heads, 128)
    K.kvc_stage_layer(L, plan, kp, vp, kc, vc)
    torch.cuda.synchronize()
    # the separator rows are rotated zeros here (+-0), equal to the oracle's
    assert np.array_equal(_val(down_bf16(kc)[:n_r]), _oracle_staged_k(w, x["k_src"]))
    assert np.array_equal(down_bf16(vc)[:n_r], x["v_cache"][:n_r])


@pytest.mark.parametrize("name", ["sep-4k", "4k"])
def test_two_stream_pipeline_matches_layer_by_layer(K, name):
    # layer 0 is the check layer, layers 1-2 reuse its selection; staging of
    # all layers runs ahead on a copy stream, each layer's computation waits
    # for its own event
    w = W.get(name)
    n_layers, ratio = 3, w.ratio
    xs = [build(w, seed=9, layer=l) for l in range(n_layers)]
    N, n_r = w.n_rows, w.n_reused
    ref = [gpu_layer(K, w, xs[0], True, ratio)]
    sel_np = ref[0]["sel"]
    compact = [dict(x, q=x["q"][sel_np], k_fresh=x["k_fresh"][sel_np], v_fresh=x["v_fresh"][sel_np])
               for x in xs]
    for l in range(1, n_layers):
        ref.append(gpu_layer(K, w, compact[l], False, ratio, sel_in=sel_np))

    L, plan = _layout_plan(K, w)
    keep = []
    kp, vp = [], []
    for l in range(n_layers):
        kp += _chunk_sources(w, xs[l]["k_src"][:n_r], "pinned_one_buffer", keep)
        vp += _chunk_sources(w, xs[l]["v_cache"][:n_r], "pinned_one_buffer", keep)
    kcs = [empty_bf16(N, w.n_kv_heads, 128) for _ in range(n_layers)]
    vcs = [empty_bf16(N, w.n_kv_heads, 128) for _ in range(n_layers)]
    copy = torch.cuda.Stream()
    events = [torch.cuda.Event() for _ in range(n_layers)]
    for e in events:
        e.record(copy)           # creates the underlying event
    n_sel = K.kvc_recompute_count(ratio, n_r) + w.n_query
    sel = torch.full((n_sel,), -1, dtype=torch.int32, device="cuda:0")
    outs = [empty_bf16(n_sel, w.n_q_heads, 128) for _ in range(n_layers)]
    lses = [torch.empty((n_sel, w.n_q_heads), dtype=torch.float32, device="cuda:0") for _ in range(n_layers)]
    wb = K.kvc_blend_workspace(L)
    ws = bytes_buf(wb)
    fresh = [(up(xs[0]["q"]), up(xs[0]["k_fresh"]), up(xs[0]["v_fresh"]))]
    torch.cuda.synchronize()
    K.kvc_stage_layers(L, plan, n_layers, kp, vp, kcs, vcs, events, stream=copy)
    comp = torch.cuda.current_stream()
    for l in range(n_layers):
        comp.wait_event(events[l])
        if l == 1:
            # the reuse layers' recomputed rows follow the check layer's selection
            idx = sel.long()
            fresh += [(up(xs[j]["q"])[idx].contiguous(), up(xs[j]["k_fresh"])[idx].contiguous(),
                       up(xs[j]["v_fresh"])[idx].contiguous()) for j in range(1, n_layers)]
        q, kf, vf = fresh[l]
        K.kvc_blend_prefill_layer(L, plan, l == 0, ratio, None, kcs[l], vcs[l], q, kf, vf, sel, n_sel,
                                  outs[l], lses[l], ws, wb)
    torch.cuda.synchronize()
    got_sel = sel.cpu().numpy().astype(np.int64)
    # the oracle's layers: the check layer selects from its own adjustment
    # and deviations, the reuse layers take that selection; attention on
    # seeded sample rows (the first, the query chunk's, random ones)
    rng = np.random.default_rng(90)
    rows = np.unique(np.concatenate([[0, n_sel - 1], np.arange(n_sel - w.n_query, n_sel),
                                     rng.choice(n_sel, 96, replace=False)]))
    want = [oracle_layer(w, xs[0], True, ratio, attn_rows=rows)]
    assert np.array_equal(got_sel, want[0]["sel"])
    for l in range(1, n_layers):
        want.append(oracle_layer(w, compact[l], False, ratio, sel=want[0]["sel"], attn_rows=rows))
    for l in range(n_layers):
        assert np.array_equal(_val(down_bf16(kcs[l])), _val(want[l]["k_cache"])), l
        assert np.array_equal(down_bf16(vcs[l]), want[l]["v_cache"]), l
        ok, err = within_tol(_val(down_bf16(outs[l])[rows]), want[l]["out"])
        assert ok, (l, err)
        assert np.allclose(lses[l].cpu().numpy()[rows], want[l]["lse"], rtol=0, atol=LSE_ATOL), l
    # and bit for bit the layer-by-layer path of the library
    assert np.array_equal(got_sel, sel_np)
    for l in range(n_layers):
        assert np.array_equal(down_bf16(outs[l]), ref[l]["out"]), l
        assert np.array_equal(lses[l].cpu().numpy(), ref[l]["lse"]), l
        assert np.array_equal(_val(down_bf16(kcs[l])), _val(ref[l]["k_cache"])), l
        assert np.array_equal(down_bf16(vcs[l]), ref[l]["v_cache"]), l
