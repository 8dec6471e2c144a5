"""GPU parity of the whole layer (kvc_blend_prefill_layer) against the oracle.

Selection indices and blended caches bit-exact; attention outputs within
2e-2 abs + 1e-2 rel; LSE within 1e-4.
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as W
from _blend import gpu_layer, oracle_layer, layout
from _gpu import within_tol
from _inputs import build

pytestmark = pytest.mark.gpu
# The kernel normalises by the sum of the bfloat16-rounded softmax weights it
# multiplies V with (so O is an exact weighted average); each weight carries a
# relative rounding error of at most 2^-8, hence |LSE error| <= ln(1 + 2^-8)
# plus float32 noise.
LSE_ATOL = 2.0 ** -8 + 1e-4
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
