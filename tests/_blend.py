"""Runs one blend layer through the C ABI and through the oracle (tests only)."""
import numpy as np
import torch

import oracle
from _gpu import up, down_bf16, empty_bf16, bytes_buf


def layout(K, w):
    return K.Layout(w.chunk_len, w.n_query, w.n_q_heads, w.n_kv_heads, w.head_dim, w.rope_theta,
                    chunk_old_pos0=w.chunk_old_pos0)


def gpu_layer(K, w, x, is_check, ratio, sel_in=None, in_place=False, plan=None, L=None):
    """x: dict of bf16 bit arrays (k_src, v_cache, q, k_fresh, v_fresh).  Returns numpy results."""
    L = L or layout(K, w)
    if plan is None:
        pb = K.kvc_plan_bytes(L)
        plan = bytes_buf(pb)
        plan = K.kvc_plan_upload(L, plan, pb)
    n_sel = K.kvc_recompute_count(ratio, w.n_reused) + w.n_query
    k_src = up(x["k_src"])
    k_cache = k_src if in_place else empty_bf16(*x["k_src"].shape)
    v_cache = up(x["v_cache"])
    q, kf, vf = up(x["q"]), up(x["k_fresh"]), up(x["v_fresh"])
    sel = up(np.asarray(sel_in, dtype=np.int32)) if sel_in is not None else \
        torch.full((max(n_sel, 1),), -1, dtype=torch.int32, device="cuda:0")
    out = empty_bf16(max(n_sel, 1), w.n_q_heads, w.head_dim)
    lse = torch.empty((max(n_sel, 1), w.n_q_heads), dtype=torch.float32, device="cuda:0")
    wb = K.kvc_blend_workspace(L)
    ws = bytes_buf(wb)
    K.kvc_blend_prefill_layer(L, plan, is_check, ratio, k_src, k_cache, v_cache, q, kf, vf, sel, n_sel,
                              out, lse, ws, wb)
    torch.cuda.synchronize()
    return dict(sel=sel[:n_sel].cpu().numpy().astype(np.int64), out=down_bf16(out)[:n_sel],
                lse=lse[:n_sel].cpu().numpy(), k_cache=down_bf16(k_cache), v_cache=down_bf16(v_cache))


def oracle_layer(w, x, is_check, ratio, sel=None, attn_rows=None):
    return oracle.blend_prefill_layer(w.chunk_len, w.n_query, w.n_q_heads, w.n_kv_heads, w.rope_theta,
                                      x["k_src"], x["v_cache"], x["q"], x["k_fresh"], x["v_fresh"],
                                      is_check, ratio, sel=sel, old_pos0=w.chunk_old_pos0,
                                      attn_rows=attn_rows)
