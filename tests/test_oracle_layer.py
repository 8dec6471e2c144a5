"""Pins for the oracle's decoder-layer steps around the attention.

The models the paper evaluates (Section 4.1) are Llama-style pre-norm
decoder layers.  Each step is checked against a hand-worked value, closed
forms and independent library routines (torch's RMSNorm and SiLU, scipy's
logistic function, Hugging Face's RoPE); the composed layer is checked
against Hugging Face's own Llama decoder layer in float64, which fixes the
wiring (order of Q/K/V heads and of gate/up, where the norms and residual
additions sit, which kv head a query head reads).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import rms_norm, qkv_rope, swiglu, projection, decoder_layer, inv_freq


def test_rms_norm_hand_worked():
    # x = [3, 4]: mean square 12.5
    out = rms_norm(np.array([[3.0, 4.0]]), np.array([1.0, 2.0]), 0.0)[0]
    r = math.sqrt(12.5)
    assert np.allclose(out, [3.0 / r, 8.0 / r], rtol=1e-15, atol=0)


def test_rms_norm_constant_row_and_eps():
    # a constant row c: c / sqrt(c^2 + eps) * gamma
    c, eps = -0.75, 1e-5
    g = np.linspace(0.5, 1.5, 64)
    out = rms_norm(np.full((1, 64), c), g, eps)[0]
    assert np.allclose(out, c / math.sqrt(c * c + eps) * g, rtol=1e-14, atol=0)


def test_rms_norm_scale_invariant_without_eps():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 96))
    g = rng.standard_normal(96)
    assert np.array_equal(rms_norm(x * 2.0 ** 9, g, 0.0), rms_norm(x, g, 0.0))


def test_rms_norm_matches_torch():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((7, 4096)) * rng.lognormal(0, 1, (7, 1))
    g = rng.standard_normal(4096)
    want = torch.nn.functional.rms_norm(torch.from_numpy(x), (4096,), torch.from_numpy(g), 1e-5)
    assert np.allclose(rms_norm(x, g, 1e-5), want.numpy(), rtol=1e-12, atol=1e-12)


def test_rms_norm_takes_bf16_bits():
    rng = np.random.default_rng(3)
    xb = oracle.f64_to_bf16(rng.standard_normal((3, 32)))
    gb = oracle.f64_to_bf16(rng.standard_normal(32))
    assert np.array_equal(rms_norm(xb, gb, 1e-5),
                          rms_norm(oracle.bf16_to_f64(xb), oracle.bf16_to_f64(gb), 1e-5))


def test_qkv_rope_position_zero_is_a_split():
    rng = np.random.default_rng(4)
    y = rng.standard_normal((6, (3 + 2 + 2) * 128))
    q, k, v = qkv_rope(y, np.zeros(6, dtype=np.int64), 3, 2, 2, inv_freq(128, 500000.0))
    heads = y.reshape(6, 7, 128)
    assert np.allclose(q, heads[:, :3], rtol=0, atol=0)
    assert np.allclose(k, heads[:, 3:5], rtol=0, atol=0)
    assert np.array_equal(v, heads[:, 5:])


def test_qkv_rope_head_placement():
    # one nonzero head in the fused row lands in exactly one output head
    f = inv_freq(128, 500000.0)
    for src, (part, dst) in enumerate([("q", 0), ("q", 1), ("k", 0), ("v", 0)]):
        y = np.zeros((1, 4 * 128))
        y[0, src * 128:(src + 1) * 128] = np.arange(1, 129)
        q, k, v = qkv_rope(y, np.array([17]), 2, 1, 1, f)
        out = dict(q=q, k=k, v=v)
        for name, t in out.items():
            for h in range(t.shape[1]):
                nz = np.any(t[0, h] != 0)
                assert nz == (name == part and h == dst), (src, name, h)
    # the V head is copied, not rotated
    assert np.array_equal(v[0, 0], np.arange(1, 129, dtype=np.float64))


def test_qkv_rope_matches_huggingface():
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    rng = np.random.default_rng(5)
    n, D = 11, 128
    y = rng.standard_normal((n, (4 + 2 + 2) * D))
    pos = np.sort(rng.choice(130000, n, replace=False))
    f = inv_freq(D, 500000.0)
    q, k, v = qkv_rope(y, pos, 4, 2, 2, f)
    heads = torch.from_numpy(y.reshape(n, 8, D))
    fr = torch.from_numpy(np.outer(pos.astype(np.float64), f))
    emb = torch.cat([fr, fr], dim=-1)[None]
    hq, hk = apply_rotary_pos_emb(heads[:, :4].permute(1, 0, 2)[None],
                                  heads[:, 4:6].permute(1, 0, 2)[None], emb.cos(), emb.sin())
    assert np.allclose(q, hq[0].permute(1, 0, 2).numpy(), rtol=0, atol=1e-9)
    assert np.allclose(k, hk[0].permute(1, 0, 2).numpy(), rtol=0, atol=1e-9)


def test_qkv_rope_scores_depend_on_relative_position():
    rng = np.random.default_rng(6)
    f = inv_freq(128, 500000.0)
    y = rng.standard_normal((1, 3 * 128))
    scores = []
    for p0 in (0, 1000, 70001):
        qa, _, _ = qkv_rope(y, np.array([p0 + 40]), 1, 1, 1, f)
        _, kb, _ = qkv_rope(y, np.array([p0 + 3]), 1, 1, 1, f)
        scores.append(float(np.dot(qa[0, 0], kb[0, 0])))
    assert np.allclose(scores, scores[0], rtol=1e-9, atol=1e-9)


def test_swiglu_hand_worked():
    out = swiglu(np.array([[2.0, 3.0]]), 1)[0, 0]
    assert math.isclose(out, 2.0 * 3.0 / (1.0 + math.exp(-2.0)), rel_tol=1e-15)


def test_swiglu_matches_torch_and_scipy():
    from scipy.special import expit
    rng = np.random.default_rng(7)
    gu = rng.standard_normal((9, 2 * 333)) * 4
    g, u = gu[:, :333], gu[:, 333:]
    ours = swiglu(gu, 333)
    assert np.allclose(ours, g * expit(g) * u, rtol=1e-13, atol=1e-300)
    want = torch.nn.functional.silu(torch.from_numpy(g)) * torch.from_numpy(u)
    assert np.allclose(ours, want.numpy(), rtol=1e-13, atol=1e-300)


def test_swiglu_extremes():
    gu = np.array([[0.0, -800.0, 800.0, 5.0, 5.0, 2.0]])
    out = swiglu(gu, 3)[0]
    assert out[0] == 0.0
    assert out[1] == 0.0 or abs(out[1]) < 1e-300
    assert out[2] == 800.0 * 2.0


def _hf_layer(hidden, inter, hq, hkv, theta, eps, seed):
    from transformers import LlamaConfig
    from transformers.models.llama import modeling_llama as m
    cfg = LlamaConfig(hidden_size=hidden, intermediate_size=inter, num_attention_heads=hq,
                      num_key_value_heads=hkv, head_dim=128, rope_theta=theta, rms_norm_eps=eps,
                      attn_implementation="eager")
    torch.manual_seed(seed)
    layer = m.LlamaDecoderLayer(cfg, layer_idx=0).double()
    with torch.no_grad():
        for p in layer.parameters():
            p.normal_(0.0, 0.05)
        layer.input_layernorm.weight.add_(1.0)
        layer.post_attention_layernorm.weight.add_(1.0)
    return cfg, layer, m.LlamaRotaryEmbedding(cfg)


def _weights_of(layer):
    a, mlp = layer.self_attn, layer.mlp
    t = lambda lin: lin.weight.detach().numpy().T.copy()
    return dict(norm1=layer.input_layernorm.weight.detach().numpy().copy(),
                norm2=layer.post_attention_layernorm.weight.detach().numpy().copy(),
                qkv=np.concatenate([t(a.q_proj), t(a.k_proj), t(a.v_proj)], axis=1),
                o=t(a.o_proj), gate_up=np.concatenate([t(mlp.gate_proj), t(mlp.up_proj)], axis=1),
                down=t(mlp.down_proj))


@pytest.mark.parametrize("hq,hkv", [(2, 1), (4, 2)])
def test_decoder_layer_matches_huggingface_llama(hq, hkv):
    hidden, inter, theta, eps, n = hq * 128, 384, 500000.0, 1e-5, 29
    cfg, layer, rot = _hf_layer(hidden, inter, hq, hkv, theta, eps, seed=hq)
    rng = np.random.default_rng(8)
    h = rng.standard_normal((n, hidden))
    x = torch.from_numpy(h)[None]
    pid = torch.arange(n)[None]
    mask = torch.full((n, n), float("-inf"), dtype=torch.float64).triu(1)[None, None]
    with torch.no_grad():
        want = layer(x, attention_mask=mask, position_ids=pid,
                     position_embeddings=rot(x, pid))[0].numpy()
    empty = np.zeros((n, hkv, 128))
    got = decoder_layer(h, np.arange(n), empty, empty, _weights_of(layer), hq, hkv,
                        inv_freq(128, theta), eps, round_bf16=False)["out"]
    # Hugging Face's RMSNorm and rotary tables run in float32
    assert np.allclose(got, want, rtol=1e-5, atol=1e-5)


def test_decoder_layer_selected_rows_equal_full_layer():
    # with the other rows' K/V exactly as the full layer computes them, the
    # selected rows' outputs equal the full layer's rows
    hq, hkv, hidden, inter, n = 4, 2, 512, 256, 37
    rng = np.random.default_rng(9)
    w = dict(norm1=1 + 0.1 * rng.standard_normal(hidden), norm2=1 + 0.1 * rng.standard_normal(hidden),
             qkv=0.05 * rng.standard_normal((hidden, (hq + 2 * hkv) * 128)),
             o=0.05 * rng.standard_normal((hq * 128, hidden)),
             gate_up=0.05 * rng.standard_normal((hidden, 2 * inter)),
             down=0.05 * rng.standard_normal((inter, hidden)))
    h = rng.standard_normal((n, hidden))
    f = inv_freq(128, 500000.0)
    zero = np.zeros((n, hkv, 128))
    full = decoder_layer(h, np.arange(n), zero, zero, w, hq, hkv, f, round_bf16=False)
    sel = np.sort(rng.choice(n, 12, replace=False))
    part = decoder_layer(h[sel], sel, full["k_cache"], full["v_cache"], w, hq, hkv, f,
                         round_bf16=False)
    assert np.allclose(part["out"], full["out"][sel], rtol=1e-12, atol=1e-12)
    # rows not selected keep the cache they were given
    rest = np.setdiff1d(np.arange(n), sel)
    assert np.array_equal(part["k_cache"][rest], full["k_cache"][rest])


def test_decoder_layer_rounding_stays_near_exact():
    hq, hkv, hidden, inter, n = 2, 1, 256, 256, 16
    rng = np.random.default_rng(10)
    w = dict(norm1=np.ones(hidden), norm2=np.ones(hidden),
             qkv=0.05 * rng.standard_normal((hidden, (hq + 2 * hkv) * 128)),
             o=0.05 * rng.standard_normal((hq * 128, hidden)),
             gate_up=0.05 * rng.standard_normal((hidden, 2 * inter)),
             down=0.05 * rng.standard_normal((inter, hidden)))
    w = {k: oracle.bf16_to_f64(oracle.f64_to_bf16(v)) for k, v in w.items()}
    h = oracle.bf16_to_f64(oracle.f64_to_bf16(rng.standard_normal((n, hidden))))
    f = inv_freq(128, 500000.0)
    zero = np.zeros((n, hkv, 128))
    a = decoder_layer(h, np.arange(n), zero, zero, w, hq, hkv, f, round_bf16=True)
    b = decoder_layer(h, np.arange(n), zero, zero, w, hq, hkv, f, round_bf16=False)
    # every stored value is a bfloat16 and the result stays within a few
    # bfloat16 roundings of the exact one
    assert np.array_equal(oracle.bf16_to_f64(oracle.f64_to_bf16(a["out"])), a["out"])
    assert np.allclose(a["out"], b["out"], rtol=2e-2, atol=2e-2)


def test_projection_hand_worked():
    # a = [[1, 2], [3, 4]], w rows (out x in) = e1, e2, e1 + e2
    a = np.array([[1.0, 2.0], [3.0, 4.0]])
    w = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0]])
    assert np.array_equal(projection(a, w), [[1, 2, 3], [3, 4, 7]])
    # gathered rows, one out of range (a zero row), and a residual
    r = np.array([[10.0, 20.0, 30.0]] * 3)
    assert np.array_equal(projection(a, w, rows=[1, 0, 5], residual=r),
                          [[13, 24, 37], [11, 22, 33], [10, 20, 30]])


def test_projection_integer_closed_form():
    # small integers: every product and sum is exact, equal to an integer
    # matrix product (numpy's int64 matmul)
    rng = np.random.default_rng(30)
    a = rng.integers(-50, 50, (37, 96))
    w = rng.integers(-50, 50, (24, 96))
    rows = rng.integers(0, 37, 19)
    res = rng.integers(-1000, 1000, (19, 24))
    want = (a[rows] @ w.T + res).astype(np.float64)
    got = projection(oracle.f64_to_bf16(a.astype(np.float64)), oracle.f64_to_bf16(w.astype(np.float64)),
                     rows=rows, residual=res.astype(np.float64))
    assert np.array_equal(got, want)
