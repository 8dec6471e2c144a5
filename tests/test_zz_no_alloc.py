"""The entry point that allocates nothing (kvc_blend_prefill_layer_noalloc),
through the C ABI: two calls in a row on one GPU, the second on a smaller
request, each equal bit for bit to kvc_blend_prefill_layer given the same
amount of workspace, and the selection equal to the oracle's; a reuse layer
after them; a check layer too large for the static scratch is refused."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from _blend import layout, oracle_layer
from _gpu import up, down_bf16, empty_bf16, bytes_buf, within_tol, LSE_ATOL
from _inputs import build

pytestmark = pytest.mark.gpu


def _run(K, w, x, is_check, ratio, noalloc, sel_in=None):
    L = layout(K, w)
    pb = K.kvc_plan_bytes(L)
    plan = K.kvc_plan_upload(L, bytes_buf(pb), pb)
    n_sel = K.kvc_recompute_count(ratio, w.n_reused) + w.n_query
    k_src, v_cache = up(x["k_src"]), up(x["v_cache"])
    k_cache = empty_bf16(*x["k_src"].shape)
    q, kf, vf = up(x["q"]), up(x["k_fresh"]), up(x["v_fresh"])
    sel = up(np.asarray(sel_in, dtype=np.int32)) if sel_in is not None else \
        torch.full((n_sel,), -1, dtype=torch.int32, device="cuda:0")
    out = empty_bf16(n_sel, w.n_q_heads, w.head_dim)
    lse = torch.empty((n_sel, w.n_q_heads), dtype=torch.float32, device="cuda:0")
    if noalloc:
        K.kvc_blend_prefill_layer_noalloc(L, plan, is_check, ratio, k_src, k_cache, v_cache, q, kf, vf, sel, n_sel,
                                          out, lse)
    else:
        # the workspace the static variant uses: the layer's part, plus the
        # attention's split partials when both fit in the static scratch
        wb = K.kvc_blend_workspace(L)
        aw = K.kvc_attention_workspace(n_sel, w.n_q_heads, w.n_kv_heads, w.head_dim)
        wb = wb + aw if wb + aw <= K.STATIC_SCRATCH_BYTES else wb
        ws = bytes_buf(wb)
        K.kvc_blend_prefill_layer(L, plan, is_check, ratio, k_src, k_cache, v_cache, q, kf, vf, sel, n_sel,
                                  out, lse, ws, wb)
    torch.cuda.synchronize()
    return dict(sel=sel.cpu().numpy().astype(np.int64), out=down_bf16(out), lse=lse.cpu().numpy(),
                k_cache=down_bf16(k_cache), v_cache=down_bf16(v_cache))


def _same(a, b):
    for key in ("sel", "out", "lse", "k_cache", "v_cache"):
        assert np.array_equal(a[key], b[key]), key


def test_noalloc_matches_workspace_entry_point(K):
    # first call: the 4.1k check layer (its split partials do not fit beside
    # the selection state: unsplit); second call: the smaller Tiny layer
    # (split partials fit), reusing the scratch the first call left behind
    for name in ("4k", "tiny"):
        w = W.get(name)
        x = build(w, seed=7)
        print(f"noalloc check layer {name}", flush=True)
        got = _run(K, w, x, True, w.ratio, True)
        want = _run(K, w, x, True, w.ratio, False)
        _same(got, want)
        r = oracle_layer(w, x, True, w.ratio)
        assert np.array_equal(got["sel"], r["sel"])
        ok, err = within_tol(oracle.bf16_to_f64(got["out"]), r["out"])
        assert ok, err
        assert np.allclose(got["lse"], r["lse"], rtol=0, atol=LSE_ATOL)
    # a reuse layer on Tiny's selection
    w = W.get("tiny")
    x1 = build(w, seed=8, layer=1)
    sel = got["sel"]
    xc = dict(x1, q=x1["q"][sel], k_fresh=x1["k_fresh"][sel], v_fresh=x1["v_fresh"][sel])
    _same(_run(K, w, xc, False, w.ratio, True, sel_in=sel), _run(K, w, xc, False, w.ratio, False, sel_in=sel))


def test_noalloc_refuses_a_check_layer_beyond_its_scratch(K):
    # 3 million reused rows need more than the 16 MiB static scratch; the
    # refusal comes before anything is enqueued (fake addresses are fine)
    L = K.Layout([1_500_000, 1_500_000], 64, 32, 8, 128, 500000.0)
    assert K.kvc_blend_workspace(L) > K.STATIC_SCRATCH_BYTES
    plan = K.Plan(1 << 44, K.kvc_plan_bytes(L), K.kvc_layout_id(L))
    A = 1 << 40
    n_sel = K.kvc_recompute_count(0.15, L.n_reused) + 64
    with pytest.raises(K.KvcError) as e:
        K.kvc_blend_prefill_layer_noalloc(L, plan, 1, 0.15, A, A, A + (1 << 38), A + (2 << 38), A + (3 << 38),
                                          A + (4 << 38), A + (5 << 38), n_sel, A + (6 << 38), None)
    assert e.value.status == K.KVC_ERR_WORKSPACE and "static scratch" in str(e.value)
