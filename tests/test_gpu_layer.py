"""GPU parity of the decoder-layer steps around the attention.

Each kernel is compared element by element with the oracle on the same
bfloat16 inputs:
* RMS normalisation and the gated SiLU compute in float32 and round once,
  so every output lies within one bfloat16 rounding (half an ulp, 2^-8
  relative) of the exact value, plus the float32 error of the sums,
  reciprocal and exponential (a few 1e-6 relative);
* the Q/K/V split with RoPE reduces the angle in float64, rotates in
  float32 and rounds once: within one bfloat16 rounding of the exact value
  plus 2^-20 of the rotated pair's norm (the float32 sine, cosine and
  products are each good to about 2^-23 of it); value heads are copied bit
  for bit.
The composed check and reuse layers run the projections as bfloat16 GEMMs
in torch (a GEMM library) between the library's steps.  Every library step
in them is compared with the oracle on the GPU's own inputs to that step's
bar (the attention to 2e-2 absolute + 1e-2 relative), the selection bit
for bit, and the whole layer with the exact one to a bound derived from
the number of bfloat16 roundings on the path (``_check_end_to_end``).
"""
import numpy as np
import pytest
import torch

import oracle
from _gpu import up, down_bf16, empty_bf16, bytes_buf, within_tol, device_normal_bf16
from _rope_tables import llama31_inv_freq, yarn_inv_freq
from _proj import projection_close

pytestmark = pytest.mark.gpu


def _one_rounding(got_bits, exact, rel_extra, abs_floor=1e-37):
    """|got - exact| <= (2^-8 + rel_extra) |exact| + abs_floor everywhere."""
    got = oracle.bf16_to_f64(got_bits)
    err = np.abs(got - exact)
    bound = (2.0 ** -8 + rel_extra) * np.abs(exact) + abs_floor
    return bool(np.all(err <= bound)), float(np.max(err / (np.abs(exact) + abs_floor))) if err.size else 0.0


def _rope_close(got_bits, want):
    """Rotated heads: |got - exact| <= 2^-8 |exact| + 2^-20 * (pair norm)."""
    got = oracle.bf16_to_f64(got_bits)
    pn = np.sqrt(want[..., :64] ** 2 + want[..., 64:] ** 2)
    pn = np.concatenate([pn, pn], axis=-1)
    err = np.abs(got - want)
    ok = bool(np.all(err <= 2.0 ** -8 * np.abs(want) + 2.0 ** -20 * pn))
    return ok, float(np.max(err / (np.abs(want) + pn + 1e-300))) if err.size else 0.0


def _bf16(rng, shape, scale=1.0):
    return oracle.f64_to_bf16(rng.standard_normal(shape) * scale)


# ---------------------------------------------------------------- RMS norm
@pytest.mark.parametrize("hidden,n", [(4096, 37), (3584, 5), (8, 3), (520, 70), (16384, 4), (1024, 1)])
def test_rms_norm(K, hidden, n):
    rng = np.random.default_rng(hidden + n)
    x = oracle.f64_to_bf16(rng.standard_normal((n, hidden)) * rng.lognormal(0, 1.5, (n, 1)))
    g = oracle.f64_to_bf16(1 + 0.2 * rng.standard_normal(hidden))
    out = empty_bf16(n, hidden)
    K.kvc_rms_norm(up(x), n, None, n, hidden, up(g), 1e-5, out)
    torch.cuda.synchronize()
    ok, err = _one_rounding(down_bf16(out), oracle.rms_norm(x, g, 1e-5), 3e-5)
    assert ok, err


def test_rms_norm_gather_and_residual_rows(K):
    rng = np.random.default_rng(11)
    n_x, hidden = 300, 4096
    x = _bf16(rng, (n_x, hidden))
    g = oracle.f64_to_bf16(1 + 0.2 * rng.standard_normal(hidden))
    rows = np.sort(rng.choice(n_x, 45, replace=False)).astype(np.int32)
    rows[7] = -1          # out of range: zero rows
    rows[20] = n_x
    out, res = empty_bf16(45, hidden), empty_bf16(45, hidden)
    K.kvc_rms_norm(up(x), n_x, up(rows), 45, hidden, up(g), 1e-5, out, res)
    torch.cuda.synchronize()
    ok_rows = (rows >= 0) & (rows < n_x)
    want = np.zeros((45, hidden))
    want[ok_rows] = oracle.rms_norm(x[rows[ok_rows]], g, 1e-5)
    got = down_bf16(out)
    ok, err = _one_rounding(got[ok_rows], want[ok_rows], 3e-5)
    assert ok, err
    assert not np.any(oracle.bf16_to_f64(got[~ok_rows]))
    r = down_bf16(res)
    assert np.array_equal(r[ok_rows], x[rows[ok_rows]])
    assert not np.any(oracle.bf16_to_f64(r[~ok_rows]))


def test_rms_norm_zero_row_and_eps(K):
    # an all-zero row with eps > 0 gives zeros; constant rows are exact
    hidden = 256
    x = np.zeros((3, hidden))
    x[1] = 2.0
    x[2] = -0.0078125
    xb = oracle.f64_to_bf16(x)
    g = oracle.f64_to_bf16(np.ones(hidden))
    out = empty_bf16(3, hidden)
    K.kvc_rms_norm(up(xb), 3, None, 3, hidden, up(g), 1e-5, out)
    torch.cuda.synchronize()
    ok, err = _one_rounding(down_bf16(out), oracle.rms_norm(xb, g, 1e-5), 3e-5)
    assert ok, err
    assert not np.any(oracle.bf16_to_f64(down_bf16(out)[0]))


# ---------------------------------------------------------------- Q/K/V + RoPE
@pytest.mark.parametrize("hq,hk,hv,with_pos", [(32, 8, 8, True), (0, 8, 0, False), (32, 0, 8, True),
                                               (1, 0, 0, True), (4, 2, 2, False), (0, 0, 3, True),
                                               (64, 64, 64, True)])
def test_qkv_rope(K, hq, hk, hv, with_pos):
    rng = np.random.default_rng(hq * 7 + hk * 3 + hv)
    n = 37
    y = _bf16(rng, (n, (hq + hk + hv) * 128), 2.0)
    pos = np.sort(rng.choice(130000, n, replace=False)).astype(np.int32) if with_pos else None
    f = oracle.inv_freq(128, 500000.0)
    q, k, v = empty_bf16(n, max(hq, 1), 128), empty_bf16(n, max(hk, 1), 128), empty_bf16(n, max(hv, 1), 128)
    K.kvc_qkv_rope(up(y), n, hq, hk, hv, 128, None if pos is None else up(pos), 500000.0,
                   q if hq else None, k if hk else None, v if hv else None)
    torch.cuda.synchronize()
    wq, wk, wv = oracle.qkv_rope(y, np.arange(n) if pos is None else pos, hq, hk, hv, f)
    for got, want, h in ((q, wq, hq), (k, wk, hk)):
        if h:
            ok, err = _rope_close(down_bf16(got), want)
            assert ok, err
    if hv:
        assert np.array_equal(down_bf16(v), oracle.f64_to_bf16(wv))


def test_qkv_rope_scaled_frequencies(K):
    # Llama-3.1's rescaled frequency table, positions up to 2^17
    rng = np.random.default_rng(12)
    n = 64
    y = _bf16(rng, (n, 48 * 128))
    pos = np.sort(rng.choice(1 << 17, n, replace=False)).astype(np.int32)
    f = llama31_inv_freq()
    q, k, v = empty_bf16(n, 32, 128), empty_bf16(n, 8, 128), empty_bf16(n, 8, 128)
    K.kvc_qkv_rope(up(y), n, 32, 8, 8, 128, up(pos), 0.0, q, k, v, inv_freq=list(f))
    torch.cuda.synchronize()
    wq, wk, wv = oracle.qkv_rope(y, pos, 32, 8, 8, f)
    for got, want in ((q, wq), (k, wk)):
        ok, err = _rope_close(down_bf16(got), want)
        assert ok, err
    assert np.array_equal(down_bf16(v), oracle.f64_to_bf16(wv))


def test_qkv_rope_yarn_frequencies(K):
    # Qwen2.5's YaRN table, Qwen2.5-7B's head mix (28 query, 4 key/value
    # heads), positions up to 2^17
    rng = np.random.default_rng(13)
    n = 64
    y = _bf16(rng, (n, 36 * 128))
    pos = np.sort(rng.choice(1 << 17, n, replace=False)).astype(np.int32)
    f = yarn_inv_freq()
    q, k, v = empty_bf16(n, 28, 128), empty_bf16(n, 4, 128), empty_bf16(n, 4, 128)
    K.kvc_qkv_rope(up(y), n, 28, 4, 4, 128, up(pos), 0.0, q, k, v, inv_freq=list(f))
    torch.cuda.synchronize()
    wq, wk, wv = oracle.qkv_rope(y, pos, 28, 4, 4, f)
    for got, want in ((q, wq), (k, wk)):
        ok, err = _rope_close(down_bf16(got), want)
        assert ok, err
    assert np.array_equal(down_bf16(v), oracle.f64_to_bf16(wv))


def test_qkv_rope_position_zero_and_largest(K):
    # position 0 is a plain split (cos 1, sin 0: exact); the largest int32
    # position still reduces its angle exactly enough
    rng = np.random.default_rng(15)
    y = _bf16(rng, (3, 3 * 128))
    pos = np.array([0, 2**31 - 1, 123456789], dtype=np.int32)
    q, k, v = empty_bf16(3, 1, 128), empty_bf16(3, 1, 128), empty_bf16(3, 1, 128)
    K.kvc_qkv_rope(up(y), 3, 1, 1, 1, 128, up(pos), 500000.0, q, k, v)
    torch.cuda.synchronize()
    wq, wk, wv = oracle.qkv_rope(y, pos, 1, 1, 1, oracle.inv_freq(128, 500000.0))
    assert np.array_equal(oracle.bf16_to_f64(down_bf16(q)[0]), oracle.bf16_to_f64(y[0, :128]).reshape(1, 128))
    for got, want in ((q, wq), (k, wk)):
        ok, err = _rope_close(down_bf16(got), want)
        assert ok, err


# ---------------------------------------------------------------- gated SiLU
@pytest.mark.parametrize("inter,n", [(14336, 19), (8, 5), (2056, 3), (18944, 2)])
def test_swiglu(K, inter, n):
    rng = np.random.default_rng(inter + n)
    gu = rng.standard_normal((n, 2 * inter)) * 3
    gu[0, :6] = [0.0, -100.0, 100.0, -20.0, 20.0, -1e-30]
    gub = oracle.f64_to_bf16(gu)
    out = empty_bf16(n, inter)
    K.kvc_swiglu(up(gub), n, inter, out)
    torch.cuda.synchronize()
    ok, err = _one_rounding(down_bf16(out), oracle.swiglu(gub, inter), 1e-5)
    assert ok, err


# ---------------------------------------------------------------- tensors past 2^31 elements
@pytest.mark.timeout(300)
def test_layer_ops_beyond_2g_elements(K):
    # each input holds more than 2^31 elements (4.3-4.9 GB); sampled rows on
    # both sides of the boundary against the oracle
    rng = np.random.default_rng(31)

    def sample(n, boundary_row):
        return np.unique(np.concatenate([[0, 1, n - 1], rng.integers(0, n, 16),
                                         rng.integers(boundary_row, n, 16)]))

    # RMS norm: 600,000 x 4,096, and a gather of rows past the boundary
    n, hid = 600_000, 4096
    print(f"layer ops past 2^31 elements: rms_norm {n}x{hid}", flush=True)
    x = device_normal_bf16((n, hid), 41, 2.0)
    g = oracle.f64_to_bf16(1 + 0.2 * rng.standard_normal(hid))
    out = empty_bf16(n, hid)
    K.kvc_rms_norm(x, n, None, n, hid, up(g), 1e-5, out)
    rows = sample(n, 2**31 // hid)
    gat = np.sort(rng.integers(2**31 // hid, n, 40)).astype(np.int32)
    gout, gres = empty_bf16(40, hid), empty_bf16(40, hid)
    K.kvc_rms_norm(x, n, up(gat), 40, hid, up(g), 1e-5, gout, gres)
    torch.cuda.synchronize()
    idx = torch.from_numpy(rows).cuda()
    xr = down_bf16(x[idx])
    ok, err = _one_rounding(down_bf16(out[idx]), oracle.rms_norm(xr, g, 1e-5), 3e-5)
    assert ok, err
    xg = down_bf16(x[torch.from_numpy(gat.astype(np.int64)).cuda()])
    ok, err = _one_rounding(down_bf16(gout), oracle.rms_norm(xg, g, 1e-5), 3e-5)
    assert ok, err
    assert np.array_equal(down_bf16(gres), xg)
    del x, out

    # Q/K/V split with RoPE: 360,000 rows of 48 heads
    n, hq, hk, hv = 360_000, 32, 8, 8
    print(f"layer ops past 2^31 elements: qkv_rope {n}x{(hq + hk + hv) * 128}", flush=True)
    y = device_normal_bf16((n, (hq + hk + hv) * 128), 42, 2.0)
    pos = (np.arange(n, dtype=np.int64) * 3 + 7).astype(np.int32)
    q, k, v = empty_bf16(n, hq, 128), empty_bf16(n, hk, 128), empty_bf16(n, hv, 128)
    K.kvc_qkv_rope(y, n, hq, hk, hv, 128, up(pos), 500000.0, q, k, v)
    torch.cuda.synchronize()
    rows = sample(n, 2**31 // ((hq + hk + hv) * 128))
    idx = torch.from_numpy(rows).cuda()
    wq, wk, wv = oracle.qkv_rope(down_bf16(y[idx]), pos[rows], hq, hk, hv, oracle.inv_freq(128, 500000.0))
    for got, want in ((q, wq), (k, wk)):
        ok, err = _rope_close(down_bf16(got[idx]), want)
        assert ok, err
    assert np.array_equal(down_bf16(v[idx]), oracle.f64_to_bf16(wv))
    del y, q, k, v

    # gated SiLU: 80,000 rows of 2 x 14,336
    n, inter = 80_000, 14336
    print(f"layer ops past 2^31 elements: swiglu {n}x{2 * inter}", flush=True)
    gu = device_normal_bf16((n, 2 * inter), 43, 3.0)
    act = empty_bf16(n, inter)
    K.kvc_swiglu(gu, n, inter, act)
    torch.cuda.synchronize()
    rows = sample(n, 2**31 // (2 * inter))
    idx = torch.from_numpy(rows).cuda()
    ok, err = _one_rounding(down_bf16(act[idx]), oracle.swiglu(down_bf16(gu[idx]), inter), 1e-5)
    assert ok, err


# ---------------------------------------------------------------- composed layers
D = 128
SMALL = dict(hq=4, hkv=2, hid=512, inter=1024)
LLAMA = dict(hq=32, hkv=8, hid=4096, inter=14336)   # Llama-3.1-8B's layer


def _bf16_of_f32(a):
    """float32 -> bf16 bits, nearest even (torch's conversion; its agreement
    with the oracle's rounding is pinned in test_oracle_bf16): fast for the
    layer-sized weight matrices."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16) \
        .view(torch.int16).numpy().view(np.uint16)


def _weights(rng, hq, hkv, hid, inter):
    b = lambda shape, s: _bf16_of_f32(rng.standard_normal(shape, dtype=np.float32) * np.float32(s))
    sc = 1.0 / np.sqrt(hid)
    return dict(norm1=oracle.f64_to_bf16(1 + 0.1 * rng.standard_normal(hid)),
                norm2=oracle.f64_to_bf16(1 + 0.1 * rng.standard_normal(hid)),
                qkv=b((hid, (hq + 2 * hkv) * D), sc), o=b((hq * D, hid), sc),
                gate_up=b((hid, 2 * inter), sc), down=b((inter, hid), 1.0 / np.sqrt(inter)))


def _proj(K, a, n, w_in_out, res=None, out=None):
    """a [n, in] times a weight given in the oracle's [in, out] layout, on the
    GPU through kvc_projection (which takes the [out, in] layout); res is
    added, out may be res (in place)."""
    wt = up(np.ascontiguousarray(w_in_out.T))
    n_out, k = wt.shape
    if out is None:
        out = empty_bf16(n, n_out)
    K.kvc_projection(n, n_out, k, a, n, None, wt, res, out)
    return out


def _gpu_rest(K, h_sel, attn, w, n_sel, hq, hkv, hid, inter):
    """Residual addition, second norm, feed-forward: library steps only."""
    h = h_sel.clone()
    h_res = h.clone()
    _proj(K, attn.reshape(n_sel, hq * D), n_sel, w["o"], res=h, out=h)
    x2 = empty_bf16(n_sel, hid)
    K.kvc_rms_norm(h, n_sel, None, n_sel, hid, up(w["norm2"]), 1e-5, x2)
    gu = _proj(K, x2, n_sel, w["gate_up"])
    act = empty_bf16(n_sel, inter)
    K.kvc_swiglu(gu, n_sel, inter, act)
    h_mid = h.clone()
    _proj(K, act, n_sel, w["down"], res=h, out=h)
    return {n: down_bf16(t) for n, t in
            (("h_in", h_res), ("h_mid", h_mid), ("x2", x2), ("gu", gu), ("act", act), ("out", h))}


def _check_steps(got, w, sel, kc, vc, hq, hkv, hid, inter):
    """Each library step against the oracle on the GPU's own inputs."""
    f64 = oracle.bf16_to_f64
    ok, err = _one_rounding(got["x"], oracle.rms_norm(got["h"], w["norm1"], 1e-5), 3e-5)
    assert ok, ("x", err)
    q, k, v = oracle.qkv_rope(got["y"], sel, hq, hkv, hkv, oracle.inv_freq(D, 500000.0))
    for name, want in (("q", q), ("k", k)):
        ok, err = _rope_close(got[name], want)
        assert ok, (name, err)
    assert np.array_equal(got["v"], oracle.f64_to_bf16(v))
    attn, _ = oracle.sparse_query_attention(got["q"], sel, kc, vc, hq, hkv)
    ok, err = within_tol(f64(got["attn"]), attn)
    assert ok, ("attn", err)
    ok, err = _one_rounding(got["x2"], oracle.rms_norm(got["h_mid"], w["norm2"], 1e-5), 3e-5)
    assert ok, ("x2", err)
    ok, err = _one_rounding(got["act"], oracle.swiglu(got["gu"], inter), 1e-5)
    assert ok, ("act", err)
    # the four projections, each on the GPU's own inputs
    n = len(sel)
    for name, a, wk, res in (("y", got["x"], "qkv", None), ("h_mid", got["attn"].reshape(n, hq * D), "o", got["h_in"]),
                             ("gu", got["x2"], "gate_up", None), ("out", got["act"], "down", got["h_mid"])):
        ok, excess = projection_close(got[name], a, np.ascontiguousarray(w[wk].T), residual=res)
        assert ok, (name, excess)


def _check_end_to_end(out_bits, exact):
    """The whole bf16 layer against the exact one.  The path rounds nine
    stored tensors to bfloat16 (norm, projection, Q/K/V, attention, residual,
    norm, gate/up, activation, residual); each rounding adds a relative error
    of at most 2^-9 (about 2^-9/sqrt(3) in norm), and the errors add up at
    random: a few times 2^-9 in norm.  Bounds: 2^-6 in Frobenius norm and
    2^-4 times the output's RMS for any element; a wiring mistake (a head,
    a residual, gate and up swapped) is off by order one."""
    got = oracle.bf16_to_f64(out_bits)
    rms = np.sqrt(np.mean(exact ** 2))
    rel = np.linalg.norm(got - exact) / np.linalg.norm(exact)
    assert rel <= 2.0 ** -6, rel
    assert np.max(np.abs(got - exact)) <= 2.0 ** -4 * rms, np.max(np.abs(got - exact)) / rms


def _reuse_layer(K, shape, seed, chunk_len, n_query, n_pick):
    """A reuse layer: the selected rows' hidden states at positions sel and
    the blended cache of the other rows; projections as bf16 GEMMs in torch."""
    hq, hkv, hid, inter = shape["hq"], shape["hkv"], shape["hid"], shape["inter"]
    rng = np.random.default_rng(seed)
    n_r = sum(chunk_len)
    N = n_r + n_query
    sel = np.concatenate([np.sort(rng.choice(n_r, n_pick, replace=False)), np.arange(n_r, N)])
    n_sel = len(sel)
    ratio = n_pick / n_r
    assert K.kvc_recompute_count(ratio, n_r) == n_pick
    w = _weights(rng, hq, hkv, hid, inter)
    h = _bf16(rng, (n_sel, hid))
    k_cache, v_cache = _bf16(rng, (N, hkv, D)), _bf16(rng, (N, hkv, D))
    f = oracle.inv_freq(D, 500000.0)

    L = K.Layout(chunk_len, n_query, hq, hkv, D, 500000.0)
    sel_d = up(sel.astype(np.int32))
    x = empty_bf16(n_sel, hid)
    K.kvc_rms_norm(up(h), n_sel, None, n_sel, hid, up(w["norm1"]), 1e-5, x)
    y = _proj(K, x, n_sel, w["qkv"])
    q, k, v = empty_bf16(n_sel, hq, D), empty_bf16(n_sel, hkv, D), empty_bf16(n_sel, hkv, D)
    K.kvc_qkv_rope(y, n_sel, hq, hkv, hkv, D, sel_d, 500000.0, q, k, v)
    kc, vc = up(k_cache), up(v_cache)
    attn = empty_bf16(n_sel, hq, D)
    K.kvc_blend_prefill_layer(L, None, 0, ratio, None, kc, vc, q, k, v, sel_d, n_sel, attn, None, None, 0)
    got = _gpu_rest(K, up(h), attn, w, n_sel, hq, hkv, hid, inter)
    torch.cuda.synchronize()
    got.update(h=h, x=down_bf16(x), y=down_bf16(y), q=down_bf16(q), k=down_bf16(k),
               v=down_bf16(v), attn=down_bf16(attn))

    # the blended cache: selected rows hold the fresh K/V, the rest is untouched
    kcg, vcg = down_bf16(kc), down_bf16(vc)
    rest = np.setdiff1d(np.arange(N), sel)
    assert np.array_equal(kcg[rest], k_cache[rest]) and np.array_equal(vcg[rest], v_cache[rest])
    assert np.array_equal(kcg[sel], got["k"]) and np.array_equal(vcg[sel], got["v"])
    _check_steps(got, w, sel, kcg, vcg, hq, hkv, hid, inter)
    exact = oracle.decoder_layer(h, sel, k_cache, v_cache, w, hq, hkv, f, 1e-5, round_bf16=False)
    _check_end_to_end(got["out"], exact["out"])


def test_reuse_layer_composed(K):
    _reuse_layer(K, SMALL, 13, [90, 60, 110, 40], 23, 45)


@pytest.mark.timeout(300)
def test_reuse_layer_llama_shape(K):
    # the real layer widths: hidden 4096, 32 q / 8 kv heads, MLP 14336
    _reuse_layer(K, LLAMA, 16, [200, 150, 250], 100, 90)


def test_check_layer_composed(K):
    # a check layer: keys projected for every row, the selection, then Q/V
    # for the selected rows only and the rest of the layer on them
    rng = np.random.default_rng(14)
    chunk_len, n_query = [70, 130, 100], 17
    n_r = sum(chunk_len)
    N = n_r + n_query
    ratio = 0.15
    k_sel = K.kvc_recompute_count(ratio, n_r)
    n_sel = k_sel + n_query
    hq, hkv, hid, inter = SMALL["hq"], SMALL["hkv"], SMALL["hid"], SMALL["inter"]
    w = _weights(rng, hq, hkv, hid, inter)
    h_all = _bf16(rng, (N, hid))
    f = oracle.inv_freq(D, 500000.0)
    # cached keys at chunk-local positions, values as cached
    k_src, v_src = _bf16(rng, (N, hkv, D)), _bf16(rng, (N, hkv, D))

    L = K.Layout(chunk_len, n_query, hq, hkv, D, 500000.0)
    pb = K.kvc_plan_bytes(L)
    plan = bytes_buf(pb)
    plan = K.kvc_plan_upload(L, plan, pb)
    x_all = empty_bf16(N, hid)
    K.kvc_rms_norm(up(h_all), N, None, N, hid, up(w["norm1"]), 1e-5, x_all)
    y_k = _proj(K, x_all, N, np.ascontiguousarray(w["qkv"][:, hq * D:(hq + hkv) * D]))
    k_all = empty_bf16(N, hkv, D)
    K.kvc_qkv_rope(y_k, N, 0, hkv, 0, D, None, 500000.0, None, k_all, None)
    k_cache, v_cache = empty_bf16(N, hkv, D), up(v_src)
    sel = torch.full((n_sel,), -1, dtype=torch.int32, device="cuda:0")
    wb = K.kvc_blend_workspace(L)
    ws = bytes_buf(wb)
    K.kvc_select_tokens(L, plan, ratio, up(k_src), k_cache, k_all, sel, n_sel, ws, wb)
    x_sel, h_sel = empty_bf16(n_sel, hid), empty_bf16(n_sel, hid)
    K.kvc_rms_norm(up(h_all), N, sel, n_sel, hid, up(w["norm1"]), 1e-5, x_sel, h_sel)
    y = _proj(K, x_sel, n_sel, w["qkv"])
    q, k, v = empty_bf16(n_sel, hq, D), empty_bf16(n_sel, hkv, D), empty_bf16(n_sel, hkv, D)
    K.kvc_qkv_rope(y, n_sel, hq, hkv, hkv, D, sel, 500000.0, q, k, v)
    attn = empty_bf16(n_sel, hq, D)
    K.kvc_blend_prefill_layer(L, None, 0, ratio, None, k_cache, v_cache, q, k, v, sel, n_sel, attn, None,
                              None, 0)
    got = _gpu_rest(K, h_sel, attn, w, n_sel, hq, hkv, hid, inter)
    torch.cuda.synchronize()

    # the keys of every row, one step each on the GPU's inputs
    xa = down_bf16(x_all)
    ok, err = _one_rounding(xa, oracle.rms_norm(h_all, w["norm1"], 1e-5), 3e-5)
    assert ok, ("x_all", err)
    _, kf_want, _ = oracle.qkv_rope(down_bf16(y_k), np.arange(N), 0, hkv, 0, f)
    kf = down_bf16(k_all)
    ok, err = _rope_close(kf, kf_want)
    assert ok, ("k_fresh", err)
    # the selection, bit-exact given the same fresh keys
    k_shift = oracle.f64_to_bf16(oracle.rope_shift(k_src[:n_r], chunk_len, f))
    want_sel = oracle.selection(oracle.key_deviation(k_shift, kf[:n_r]), k_sel, n_r, N)
    got_sel = sel.cpu().numpy().astype(np.int64)
    assert np.array_equal(got_sel, want_sel)
    # gathered residual rows and the rest of the layer on the selected rows
    assert np.array_equal(down_bf16(h_sel), h_all[want_sel])
    got.update(h=h_all[want_sel], x=down_bf16(x_sel), y=down_bf16(y), q=down_bf16(q),
               k=down_bf16(k), v=down_bf16(v), attn=down_bf16(attn))
    kcg, vcg = down_bf16(k_cache), down_bf16(v_cache)
    kc0 = np.array(k_src, copy=True)
    kc0[:n_r] = k_shift
    rest = np.setdiff1d(np.arange(N), want_sel)
    assert np.array_equal(oracle.bf16_to_f64(kcg[rest]), oracle.bf16_to_f64(kc0[rest]))
    assert np.array_equal(vcg[rest], v_src[rest])
    assert np.array_equal(kcg[want_sel], got["k"]) and np.array_equal(vcg[want_sel], got["v"])
    _check_steps(got, w, want_sel, kcg, vcg, hq, hkv, hid, inter)
    exact = oracle.decoder_layer(h_all[want_sel], want_sel, kc0, v_src, w, hq, hkv, f, 1e-5,
                                 round_bf16=False)
    _check_end_to_end(got["out"], exact["out"])
