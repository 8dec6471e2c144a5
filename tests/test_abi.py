"""C ABI checks that need no GPU: exports, host logic, argument validation.

Every invalid argument must be rejected on the host before any HIP call,
and with no GPU present a valid call must report KVC_ERR_DEVICE.  The
"device" addresses here are fake: a call that passes validation is made
only when no GPU is present (or when it has nothing to do), since on a GPU
it would launch kernels on those addresses.
"""
import ctypes
import math
import os
import re

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "kvc.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(kvc_[a-z_0-9]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(K):
    names = _declared()
    assert len(names) >= 14
    lib = ctypes.CDLL(K.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    # the binding exposes the same names
    for n in names:
        assert callable(getattr(K, n)), n


def test_abi_version_matches_header(K):
    src = open(os.path.join(ROOT, "include", "kvc.h")).read()
    v = int(re.search(r"#define KVC_ABI_VERSION (\d+)", src).group(1))
    assert K.kvc_abi_version() == v


def test_recompute_count_matches_oracle(K):
    for ratio in (0.0, 0.05, 0.15, 0.29, 0.3, 0.5, 0.999, 1.0):
        for n in (0, 1, 7, 100, 1024, 4000, 32000, 124000, 126976, 2**31 - 1):
            assert K.kvc_recompute_count(ratio, n) == oracle.recompute_count(ratio, n), (ratio, n)
    assert K.kvc_recompute_count(float("nan"), 10) == -1
    assert K.kvc_recompute_count(1.0000001, 10) == -1
    assert K.kvc_recompute_count(-0.0, 10) == 0
    assert K.kvc_recompute_count(0.5, -1) == -1


def _layout(K, **kw):
    a = dict(chunk_len=[256] * 4, n_query=64, n_q_heads=8, n_kv_heads=2, head_dim=128, rope_theta=5e5)
    a.update(kw)
    return K.Layout(**a)


def _fplan(K, L, addr=1 << 44):
    """A plan descriptor for layout L at a fake device address, as
    kvc_plan_upload would fill it (the address is never dereferenced)."""
    return K.Plan(addr, K.kvc_plan_bytes(L), K.kvc_layout_id(L))


def _status(fn, *a, **kw):
    import paper_2609_09768_amd as K
    try:
        fn(*a, **kw)
    except K.KvcError as e:
        return e.status, str(e)
    return 0, ""


def test_layout_validation(K):
    st, _ = _status(K.kvc_plan_bytes, None)
    assert st == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_plan_bytes, _layout(K, n_q_heads=6, n_kv_heads=4))[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_plan_bytes, _layout(K, head_dim=64))[0] == K.KVC_ERR_UNSUPPORTED
    assert _status(K.kvc_plan_bytes, _layout(K, chunk_len=[3, -1]))[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_plan_bytes, _layout(K, n_query=-1))[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_plan_bytes, _layout(K, rope_theta=0.0))[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_plan_bytes, _layout(K, rope_theta=float("nan")))[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_plan_bytes, _layout(K, chunk_len=[2**30, 2**30]))[0] == K.KVC_ERR_INVALID_ARG
    bad_inv = [1.0] * 63 + [float("inf")]
    assert _status(K.kvc_plan_bytes, _layout(K, rope_theta=0.0, inv_freq=bad_inv))[0] == K.KVC_ERR_INVALID_ARG
    # an explicit table makes theta irrelevant
    assert K.kvc_plan_bytes(_layout(K, rope_theta=0.0, inv_freq=[1.0] * 64)) > 0
    # empty request is valid
    assert K.kvc_plan_bytes(_layout(K, chunk_len=[], n_query=0)) > 0


def test_plan_and_workspace_sizes(K):
    L = _layout(K)
    pb = K.kvc_plan_bytes(L)
    # header + 4 chunks x 64 (cos, sin) float64 + the row tiles
    assert pb >= 4 * 64 * 16 + 16 * 16
    assert K.kvc_select_topk_workspace(0) > 0
    assert K.kvc_select_topk_workspace(124000) >= 2 * 4 * (124000 // 2048)
    assert K.kvc_blend_workspace(L) >= 8 * 1024
    # optional split workspace: partials (D + 1 floats per query head) for a
    # selection too small to fill the GPU, none for the 124k selection
    small = K.kvc_attention_workspace(217, 8, 2, 128)
    assert small > 0 and small % (217 * 8 * 129 * 4) == 0
    assert K.kvc_attention_workspace(18856, 32, 8, 128) == 0
    # one to two workgroups per CU (one GPU's share of an 8-way kv-head
    # split: 295 workgroups): two splits
    assert K.kvc_attention_workspace(18856, 4, 1, 128) == 2 * 18856 * 4 * 129 * 4
    assert K.kvc_attention_workspace(2 * 256 * 64, 4, 1, 128) == 0
    assert K.kvc_attention_workspace(0, 32, 8, 128) == 0
    assert _status(K.kvc_select_topk_workspace, -1)[0] == K.KVC_ERR_INVALID_ARG


def test_argument_errors_precede_device_calls(K):
    L = _layout(K)
    A = 1 << 20          # fake, aligned "device" addresses: never dereferenced
    # plan buffer too small
    assert _status(K.kvc_plan_upload, L, A, 16)[0] == K.KVC_ERR_WORKSPACE
    # misaligned pointers
    P = _fplan(K, L)
    assert _status(K.kvc_rope_shift, L, P, A + 2, A + 2)[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_kv_deviation, 10, 2, 128, A + 8, A, A)[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_kv_deviation, 10, 2, 128, A, A, A + 4)[0] == K.KVC_ERR_INVALID_ARG
    # partial overlap of src and dst
    assert _status(K.kvc_rope_shift, L, P, A, A + 4096)[0] == K.KVC_ERR_INVALID_ARG
    # top-k: k > n, small workspace
    assert _status(K.kvc_select_topk, A, 10, 11, A, A, 1 << 20)[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_select_topk, A, 100, 10, A, A, 8)[0] == K.KVC_ERR_WORKSPACE
    # attention: bad scale, heads, compact queries shorter than n_sel
    args = dict(q=A, n_q_rows=10, q_rows=None, q_pos=A, n_sel=10, k=A, v=A, n_kv=10,
                n_q_heads=8, n_kv_heads=2, head_dim=128, softmax_scale=0.0, out=A, lse=None)
    assert _status(K.kvc_sparse_query_attention, **{**args, "softmax_scale": -1.0})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_sparse_query_attention, **{**args, "softmax_scale": float("nan")})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_sparse_query_attention, **{**args, "n_q_heads": 7})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_sparse_query_attention, **{**args, "head_dim": 64})[0] == K.KVC_ERR_UNSUPPORTED
    assert _status(K.kvc_sparse_query_attention, **{**args, "n_q_rows": 5})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_sparse_query_attention, **{**args, "out": A + 2})[0] == K.KVC_ERR_INVALID_ARG
    # blend layer: ratio and n_sel consistency
    n_r = 1024
    k = K.kvc_recompute_count(0.15, n_r)
    bl = dict(layout=L, plan=P, is_check_layer=1, ratio=0.15, k_src=A, k_cache=A, v_cache=A,
              q_fresh=A, k_fresh=A, v_fresh=A, sel=A, n_sel=k + 64, out=A, lse=None, ws=A,
              ws_bytes=K.kvc_blend_workspace(L))
    assert _status(K.kvc_blend_prefill_layer, **{**bl, "ratio": 1.5})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_blend_prefill_layer, **{**bl, "ratio": float("nan")})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_blend_prefill_layer, **{**bl, "n_sel": k + 63})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_blend_prefill_layer, **{**bl, "ws_bytes": 64})[0] == K.KVC_ERR_WORKSPACE
    assert _status(K.kvc_blend_prefill_layer, **{**bl, "k_cache": A + 4096})[0] == K.KVC_ERR_INVALID_ARG
    # error messages are kept per thread and name the entry point
    st, msg = _status(K.kvc_blend_prefill_layer, **{**bl, "n_sel": 1})
    assert "kvc_blend_prefill_layer" in msg and "n_sel" in msg


def test_row_count_limit(K):
    # row counts stop at 2^31 - 128 (int32 row indices, 64-row key tiles)
    M = 2**31 - 128
    A, B, C = 1 << 20, 1 << 40, 1 << 41      # fake aligned addresses, never dereferenced
    assert K.kvc_select_topk_workspace(M) > 0
    assert _status(K.kvc_select_topk_workspace, M + 1)[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_kv_deviation, M + 1, 8, 128, A, B, C)[0] == K.KVC_ERR_INVALID_ARG
    assert K.kvc_plan_bytes(_layout(K, chunk_len=[2**30, 2**30 - 256], n_query=128)) > 0
    assert _status(K.kvc_plan_bytes, _layout(K, chunk_len=[2**30, 2**30 - 256], n_query=129))[0] \
        == K.KVC_ERR_INVALID_ARG
    args = dict(q=A, n_q_rows=10, q_rows=None, q_pos=A, n_sel=10, k=B, v=C, n_kv=10,
                n_q_heads=8, n_kv_heads=2, head_dim=128, softmax_scale=0.0, out=A, lse=None)
    assert _status(K.kvc_sparse_query_attention, **{**args, "n_kv": M + 1})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_sparse_query_attention, **{**args, "n_sel": M + 1,
                                                     "n_q_rows": M + 1})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_attention_workspace, M + 1, 8, 2, 128)[0] == K.KVC_ERR_INVALID_ARG


def test_outputs_must_not_overlap_other_buffers(K):
    # every check below fails on the host before any device call
    A, MB = 1 << 32, 1 << 20
    inv = K.KVC_ERR_INVALID_ARG

    def msg_has(st_msg, *words):
        st, msg = st_msg
        return st == inv and all(w in msg for w in words)

    # deviation: dev_out inside k_fresh
    assert msg_has(_status(K.kvc_kv_deviation, 100, 2, 128, A, A + 64 * MB, A + 64 * MB + 4096),
                   "dev_out", "k_fresh")
    # top-k: idx_out or the workspace on top of dev
    assert msg_has(_status(K.kvc_select_topk, A, 1000, 10, A + 4000, A + 64 * MB, 1 << 20), "idx_out", "dev")
    assert msg_has(_status(K.kvc_select_topk, A, 1000, 10, A + 64 * MB, A + 4096, 1 << 20), "ws", "dev")
    # scatter: the two caches, or a fresh tensor and a cache
    sc = dict(sel=A, n_sel=10, fresh_is_compact=1, k_fresh=A + MB, v_fresh=A + 2 * MB, n_fresh_rows=10,
              k_cache=A + 4 * MB, v_cache=A + 8 * MB, n_rows=100, n_kv_heads=2, head_dim=128)
    assert msg_has(_status(K.kvc_scatter_rows, **{**sc, "v_cache": A + 4 * MB + 512}), "k_cache", "v_cache")
    assert msg_has(_status(K.kvc_scatter_rows, **{**sc, "k_fresh": A + 8 * MB + 1024}), "v_cache", "k_fresh")
    # attention: out over q / k, lse over v, ws over out, out over q_pos
    at = dict(q=A, n_q_rows=10, q_rows=None, q_pos=A + MB, n_sel=10, k=A + 2 * MB, v=A + 3 * MB, n_kv=10,
              n_q_heads=8, n_kv_heads=2, head_dim=128, softmax_scale=0.0, out=A + 4 * MB, lse=A + 5 * MB,
              ws=A + 6 * MB, ws_bytes=4096)
    assert msg_has(_status(K.kvc_sparse_query_attention, **{**at, "out": A + 256}), "out", "q")
    assert msg_has(_status(K.kvc_sparse_query_attention, **{**at, "out": A + 2 * MB}), "out", "k")
    assert msg_has(_status(K.kvc_sparse_query_attention, **{**at, "lse": A + 3 * MB + 16}), "lse", "v")
    assert msg_has(_status(K.kvc_sparse_query_attention, **{**at, "ws": A + 4 * MB + 1024}), "out", "ws")
    assert msg_has(_status(K.kvc_sparse_query_attention, **{**at, "q_pos": A + 4 * MB}), "out", "q_pos")
    # blend layer and selection
    L = _layout(K)
    k = K.kvc_recompute_count(0.15, 1024)
    wb = K.kvc_blend_workspace(L)
    bl = dict(layout=L, plan=_fplan(K, L), is_check_layer=1, ratio=0.15, k_src=A + MB, k_cache=A + 4 * MB,
              v_cache=A + 8 * MB, q_fresh=A + 12 * MB, k_fresh=A + 16 * MB, v_fresh=A + 20 * MB, sel=A + 24 * MB,
              n_sel=k + 64, out=A + 28 * MB, lse=A + 32 * MB, ws=A + 36 * MB, ws_bytes=wb)
    assert msg_has(_status(K.kvc_blend_prefill_layer, **{**bl, "out": A + 4 * MB + 4096}), "k_cache", "out")
    assert msg_has(_status(K.kvc_blend_prefill_layer, **{**bl, "sel": A + 28 * MB + 64}), "sel", "out")
    assert msg_has(_status(K.kvc_blend_prefill_layer, **{**bl, "ws": A + 8 * MB + 4096}), "v_cache", "ws")
    assert msg_has(_status(K.kvc_blend_prefill_layer, **{**bl, "k_fresh": A + 4 * MB + 4096}), "k_cache",
                   "k_fresh")
    assert msg_has(_status(K.kvc_blend_prefill_layer, **{**bl, "q_fresh": A + 32 * MB}), "lse", "q_fresh")
    st_ = dict(layout=L, plan=_fplan(K, L), ratio=0.15, k_src=A + MB, k_cache=A + 4 * MB, k_fresh=A + 8 * MB,
               sel=A + 12 * MB, n_sel=k + 64, ws=A + 16 * MB, ws_bytes=wb)
    assert msg_has(_status(K.kvc_select_tokens, **{**st_, "sel": A + 16 * MB + 64}), "sel", "ws")
    assert msg_has(_status(K.kvc_select_tokens, **{**st_, "k_fresh": A + 4 * MB + 4096}), "k_cache", "k_fresh")


def test_empty_work_is_ok_without_device(K):
    # nothing to do -> OK before any device query
    K.kvc_kv_deviation(0, 8, 128, None, None, None)
    K.kvc_select_topk(None, 0, 0, None, None, 0)
    K.kvc_scatter_rows(None, 0, 1, None, None, 0, None, None, 0, 8, 128)
    K.kvc_sparse_query_attention(None, 0, None, None, 0, None, None, 0, 8, 2, 128, 0.0, None, None)


def test_valid_call_without_gpu_reports_device_error(K):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    L = _layout(K)
    A = 1 << 20
    st, msg = _status(K.kvc_rope_shift, L, _fplan(K, L), A, A, stream=0)
    assert st == K.KVC_ERR_DEVICE, msg
    st, msg = _status(K.kvc_plan_upload, L, A, K.kvc_plan_bytes(L), stream=0)
    assert st == K.KVC_ERR_DEVICE, msg
    # with host staging the image is built there, then the device check
    import numpy as np
    staging = np.zeros(K.kvc_plan_bytes(L), np.uint8)
    st, msg = _status(K.kvc_plan_upload, L, A, K.kvc_plan_bytes(L), stream=0, staging=staging.ctypes.data)
    assert st == K.KVC_ERR_DEVICE, msg


def test_stage_and_pipeline_argument_errors(K):
    A = 1 << 20
    # chunks 0 and 2 are zero-K/V separator slots: their pointers may be NULL
    L = _layout(K, chunk_len=[2, 256, 2], zero_kv=[1, 0, 1])
    assert _status(K.kvc_stage_layer, L, None, [None, A, None], [None, A, None], A, A)[0] == K.KVC_ERR_INVALID_ARG
    P = _fplan(K, L)
    assert _status(K.kvc_stage_layer, L, P, [None, None, None], [None, A, None], A, A)[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_stage_layer, L, P, None, None, A, A)[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_stage_layer, L, P, [None, A, None], [None, A, None], A + 8, A)[0] == K.KVC_ERR_INVALID_ARG
    with pytest.raises(ValueError):
        _layout(K, chunk_len=[2, 256], zero_kv=[1])
    sl = dict(layout=L, plan=P, n_layers=2, k_chunks=[None, A, None] * 2, v_chunks=[None, A, None] * 2,
              k_cache=[A, A], v_cache=[A, A], events=None)
    assert _status(K.kvc_stage_layers, **{**sl, "n_layers": -1})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_stage_layers, **{**sl, "k_cache": [A, A + 8]})[0] == K.KVC_ERR_INVALID_ARG
    st, msg = _status(K.kvc_stage_layers, **{**sl, "k_chunks": [None, A, None, None, None, None]})
    assert st == K.KVC_ERR_INVALID_ARG and "layer 1" in msg, msg
    K.kvc_stage_layers(**{**sl, "n_layers": 0})            # nothing to do
    # the layers' caches share no byte with each other or with a chunk source
    C1, C2, C3, C4, S = A + (1 << 24), A + (2 << 24), A + (3 << 24), A + (4 << 24), A + (5 << 24)
    ok = dict(sl, k_chunks=[None, S, None] * 2, v_chunks=[None, S, None] * 2, k_cache=[C1, C2], v_cache=[C3, C4])
    st, msg = _status(K.kvc_stage_layers, **{**ok, "k_cache": [C1, C1]})
    assert st == K.KVC_ERR_INVALID_ARG and "overlaps" in msg, msg
    st, msg = _status(K.kvc_stage_layers, **{**ok, "v_chunks": [None, S, None, None, C4 + 4096, None]})
    assert st == K.KVC_ERR_INVALID_ARG and "chunk source" in msg and "v_cache" in msg, msg
    import torch
    if not torch.cuda.is_available():
        assert _status(K.kvc_stage_layer, L, P, [None, S, None], [None, S, None], C1, C3, stream=0)[0] == K.KVC_ERR_DEVICE
        assert _status(K.kvc_stage_layers, **ok, stream=0)[0] == K.KVC_ERR_DEVICE


def test_layer_op_argument_errors(K):
    A = 1 << 20
    # RMS normalisation
    rn = dict(x=A, n_x_rows=10, rows=None, n=10, hidden=4096, gamma=A + (1 << 20), eps=1e-5, out=A + (1 << 21))
    assert _status(K.kvc_rms_norm, **{**rn, "hidden": 4100})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_rms_norm, **{**rn, "hidden": 16392})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_rms_norm, **{**rn, "eps": -1.0})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_rms_norm, **{**rn, "eps": float("nan")})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_rms_norm, **{**rn, "n": 11})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_rms_norm, **{**rn, "x": A + 2})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_rms_norm, **{**rn, "rows": A + 2, "n": 20})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_rms_norm, **{**rn, "res_out": A + 8})[0] == K.KVC_ERR_INVALID_ARG
    # Q/K/V split with RoPE
    qr = dict(y=A, n=5, n_q_heads=32, n_k_heads=8, n_v_heads=8, head_dim=128, pos=None,
              rope_theta=5e5, q=A + (1 << 20), k=A + (1 << 21), v=A + (1 << 22))
    assert _status(K.kvc_qkv_rope, **{**qr, "head_dim": 64})[0] == K.KVC_ERR_UNSUPPORTED
    assert _status(K.kvc_qkv_rope, **{**qr, "n_q_heads": 0, "n_k_heads": 0, "n_v_heads": 0})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_qkv_rope, **{**qr, "n_k_heads": -1})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_qkv_rope, **{**qr, "rope_theta": 0.0})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_qkv_rope, **{**qr, "inv_freq": [1.0] * 63 + [float("inf")]})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_qkv_rope, **{**qr, "q": None})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_qkv_rope, **{**qr, "pos": A + 1})[0] == K.KVC_ERR_INVALID_ARG
    # a part with no heads may be NULL; theta is irrelevant with a table.
    # The call is valid and its addresses are fake, so it is made only
    # where no GPU could run it (it then stops at the device check).
    import torch
    if not torch.cuda.is_available():
        st, msg = _status(K.kvc_qkv_rope, **{**qr, "n_q_heads": 0, "n_v_heads": 0, "q": None, "v": None,
                                              "rope_theta": 0.0, "inv_freq": [1.0] * 64})
        assert st == K.KVC_ERR_DEVICE, msg
    # gated SiLU
    assert _status(K.kvc_swiglu, A, 4, 12, A)[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_swiglu, A, 4, 0, A)[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_swiglu, A, 4, 14336, A + 4)[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_swiglu, A, -1, 14336, A)[0] == K.KVC_ERR_INVALID_ARG
    # outputs overlapping inputs
    B = A + (1 << 28)
    assert _status(K.kvc_rms_norm, **{**rn, "out": A + 4096 * 2 * 3})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_rms_norm, **{**rn, "out": B, "res_out": B + 16})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_qkv_rope, **{**qr, "q": B, "k": B + 4096, "v": B + (1 << 24)})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_qkv_rope, **{**qr, "q": B, "k": B + (1 << 24), "v": A + 16})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_swiglu, A, 4, 14336, A + 4 * 14336 * 4 - 16)[0] == K.KVC_ERR_INVALID_ARG
    # index arrays are inputs too
    st, msg = _status(K.kvc_rms_norm, **{**rn, "out": B, "rows": B + 64, "n": 10})
    assert st == K.KVC_ERR_INVALID_ARG and "rows" in msg, msg
    st, msg = _status(K.kvc_qkv_rope, **{**qr, "q": B, "k": B + (1 << 24), "v": B + (2 << 24), "pos": B + 128})
    assert st == K.KVC_ERR_INVALID_ARG and "pos" in msg, msg
    # nothing to do -> OK before any device query
    K.kvc_rms_norm(None, 0, None, 0, 4096, None, 1e-5, None)
    K.kvc_qkv_rope(None, 0, 32, 8, 8, 128, None, 5e5, None, None, None)
    K.kvc_swiglu(None, 0, 14336, None)


def test_projection_argument_errors(K):
    A = 1 << 20
    W = A + (1 << 30)
    C = A + (2 << 30)
    R = A + (3 << 30)
    m, n, k = 300, 1024, 4096
    pj = dict(m=m, n=n, k=k, a=A, n_a_rows=m, a_rows=None, w=W, residual=None, c=C)
    # shapes the kernel does not take
    assert _status(K.kvc_projection, **{**pj, "k": 4100})[0] == K.KVC_ERR_UNSUPPORTED
    assert _status(K.kvc_projection, **{**pj, "k": 0})[0] == K.KVC_ERR_UNSUPPORTED
    assert _status(K.kvc_projection, **{**pj, "k": (1 << 24) + 64})[0] == K.KVC_ERR_UNSUPPORTED
    assert _status(K.kvc_projection, **{**pj, "n": 1020})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_projection, **{**pj, "n": (1 << 24) + 8})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_projection, **{**pj, "m": -1})[0] == K.KVC_ERR_INVALID_ARG
    # without a gather list c's rows are a's first m rows
    assert _status(K.kvc_projection, **{**pj, "n_a_rows": m - 1})[0] == K.KVC_ERR_INVALID_ARG
    # with one, a may hold any number of rows, but some
    assert _status(K.kvc_projection, **{**pj, "a_rows": A - 4096, "n_a_rows": 0})[0] == K.KVC_ERR_INVALID_ARG
    # NULL or misaligned pointers
    for key, val in (("a", None), ("w", None), ("c", None), ("a", A + 8), ("w", W + 2), ("c", C + 4),
                     ("residual", R + 8), ("a_rows", A - 4094)):
        assert _status(K.kvc_projection, **{**pj, key: val})[0] == K.KVC_ERR_INVALID_ARG, key
    # c overlapping an input (the residual itself is allowed: added in place)
    assert _status(K.kvc_projection, **{**pj, "c": A + 4096})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_projection, **{**pj, "c": W + 16})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_projection, **{**pj, "residual": C + 64})[0] == K.KVC_ERR_INVALID_ARG
    st, msg = _status(K.kvc_projection, **{**pj, "a_rows": C + 1024})
    assert st == K.KVC_ERR_INVALID_ARG and "a_rows" in msg, msg
    # nothing to do -> OK before any device query
    K.kvc_projection(0, n, k, None, 0, None, None, None, None)
    K.kvc_projection(m, 0, k, None, m, None, None, None, None)
    # valid calls (fake addresses) only where no GPU could run them
    import torch
    if not torch.cuda.is_available():
        assert _status(K.kvc_projection, **{**pj, "residual": C})[0] == K.KVC_ERR_DEVICE
        assert _status(K.kvc_projection, **{**pj, "a_rows": A - 4096, "n_a_rows": 7})[0] == K.KVC_ERR_DEVICE


def test_select_tokens_argument_errors(K):
    A = 1 << 20
    L = _layout(K)
    k = K.kvc_recompute_count(0.15, 1024)
    wb = K.kvc_blend_workspace(L)
    st_ = dict(layout=L, plan=_fplan(K, L), ratio=0.15, k_src=A, k_cache=A + (1 << 24), k_fresh=A, sel=A,
               n_sel=k + 64, ws=A, ws_bytes=wb)
    assert _status(K.kvc_select_tokens, **{**st_, "ratio": 1.5})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_select_tokens, **{**st_, "n_sel": k})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_select_tokens, **{**st_, "ws_bytes": wb - 1})[0] == K.KVC_ERR_WORKSPACE
    assert _status(K.kvc_select_tokens, **{**st_, "k_fresh": None})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_select_tokens, **{**st_, "sel": None})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_select_tokens, **{**st_, "plan": None})[0] == K.KVC_ERR_INVALID_ARG
    assert _status(K.kvc_select_tokens, **{**st_, "k_cache": A + 4096})[0] == K.KVC_ERR_INVALID_ARG
    st, msg = _status(K.kvc_select_tokens, **{**st_, "n_sel": 1})
    assert "kvc_select_tokens" in msg and "n_sel" in msg
    # ratio 0 with no query rows: nothing selected and no keys to adjust
    L0 = _layout(K, n_query=0)
    K.kvc_select_tokens(L0, None, 0.0, None, None, None, None, 0, None, 0)


def test_empty_selection_still_adjusts_keys(K):
    # n_sel == 0 (ratio 0, no query rows) still runs step a1, so on a host
    # without a GPU the call reaches the device check
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    A = 1 << 20
    L = _layout(K, n_query=0)
    st, msg = _status(K.kvc_blend_prefill_layer, L, _fplan(K, L), 1, 0.0, A, A + (1 << 24), A, None, None, None,
                      None, 0, None, None, None, 0)
    assert st == K.KVC_ERR_DEVICE, msg
    # without keys to adjust there is nothing to do
    K.kvc_blend_prefill_layer(L, None, 1, 0.0, None, None, None, None, None, None, None, 0, None, None, None, 0)


def test_plan_of_another_layout_is_refused(K):
    # a plan carries the id of the layout it was built for; every entry point
    # that adjusts keys compares it with its own layout before any launch
    A = 1 << 20
    L = _layout(K)
    P = _fplan(K, L)
    others = [_layout(K, chunk_len=[256, 256, 256, 255]), _layout(K, chunk_old_pos0=[0, 1, 0, 0]),
              _layout(K, rope_theta=1e4), _layout(K, zero_kv=[0, 0, 1, 0]), _layout(K, n_kv_heads=1, n_q_heads=8)]
    for L2 in others:
        assert K.kvc_layout_id(L2) != P.layout_id
        st, msg = _status(K.kvc_rope_shift, L2, P, A, A)
        assert st == K.KVC_ERR_INVALID_ARG and "another layout" in msg, msg
        k2 = K.kvc_recompute_count(0.15, L2.n_reused)
        st, _ = _status(K.kvc_blend_prefill_layer, L2, P, 1, 0.15, A, A, A + (1 << 30), A, A, A, A + (2 << 30),
                        k2 + 64, A + (3 << 30), None, A + (4 << 30), K.kvc_blend_workspace(L2))
        assert st == K.KVC_ERR_INVALID_ARG
        st, _ = _status(K.kvc_select_tokens, L2, P, 0.15, A, A, A + (1 << 30), A + (2 << 30), k2 + 64,
                        A + (4 << 30), K.kvc_blend_workspace(L2))
        assert st == K.KVC_ERR_INVALID_ARG
        st, _ = _status(K.kvc_stage_layer, L2, P, [A] * len(L2.chunk_len), [A] * len(L2.chunk_len),
                        A + (1 << 30), A + (2 << 30))
        assert st == K.KVC_ERR_INVALID_ARG
    # a NULL plan is refused where keys are adjusted, and a short buffer too
    assert _status(K.kvc_rope_shift, L, None, A, A)[0] == K.KVC_ERR_INVALID_ARG
    short = K.Plan(1 << 44, K.kvc_plan_bytes(L) - 16, P.layout_id)
    assert _status(K.kvc_rope_shift, L, short, A, A)[0] == K.KVC_ERR_WORKSPACE
    # an output over the plan buffer is refused
    st, msg = _status(K.kvc_rope_shift, L, K.Plan(A + 4096, K.kvc_plan_bytes(L), P.layout_id), A, A)
    assert st == K.KVC_ERR_INVALID_ARG and "plan" in msg, msg


def test_layout_id_compares_values_not_representations(K):
    base = K.kvc_layout_id(_layout(K))
    assert base != 0
    assert K.kvc_layout_id(_layout(K, zero_kv=[0, 0, 0, 0])) == base
    assert K.kvc_layout_id(_layout(K, chunk_old_pos0=[0, 0, 0, 0])) == base
    # with a table, theta is not used
    T = list(oracle.inv_freq(128, 1e4))
    assert K.kvc_layout_id(_layout(K, inv_freq=T, rope_theta=1.0)) == K.kvc_layout_id(_layout(K, inv_freq=T))
    # the query rows and the number of query heads do not enter the plan
    assert K.kvc_layout_id(_layout(K, n_query=3, n_q_heads=2)) == base
    assert K.kvc_layout_id(_layout(K, zero_kv=[1, 0, 0, 0])) != base
    assert _status(K.kvc_layout_id, None)[0] == K.KVC_ERR_INVALID_ARG
