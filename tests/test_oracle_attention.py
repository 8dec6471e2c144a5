"""Pins for the oracle's sparse-query causal GQA attention.

Full recomputation is plain causal attention (Section 4 setup): with every
row selected the oracle must equal PyTorch's scaled_dot_product_attention
(float64, CPU, causal) -- an independent library routine.  The causal mask
(Limitations, item 1) is pinned by perturbing keys after p_i.
"""
import numpy as np
import pytest
import torch
from scipy.special import logsumexp

from oracle import sparse_query_attention, causal_attention


def _rand(rng, *shape):
    return rng.standard_normal(shape) * rng.lognormal(0, 0.5, shape[-2:])


@pytest.mark.parametrize("hq,hkv", [(8, 2), (4, 4), (6, 1), (32, 8)])
def test_full_selection_equals_torch_causal_sdpa(hq, hkv):
    rng = np.random.default_rng(hq * 10 + hkv)
    n, D = 23, 128
    q, k, v = _rand(rng, n, hq, D), _rand(rng, n, hkv, D), _rand(rng, n, hkv, D)
    out, lse = causal_attention(q, k, v, hq, hkv)
    G = hq // hkv
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True)
    ref = ref[0].permute(1, 0, 2).numpy()
    assert np.allclose(out, ref, rtol=1e-12, atol=1e-12)
    # LSE against scipy on the explicit causal score matrix
    s = np.einsum("ihd,jhd->hij", q, np.repeat(k, G, axis=1)) / np.sqrt(D)
    s = np.where(np.tril(np.ones((n, n), bool))[None], s, -np.inf)
    assert np.allclose(lse, logsumexp(s, axis=-1).T, rtol=1e-12, atol=1e-12)


def test_sparse_rows_equal_rows_of_full_causal():
    rng = np.random.default_rng(7)
    n, hq, hkv, D = 40, 4, 2, 64
    q, k, v = _rand(rng, n, hq, D), _rand(rng, n, hkv, D), _rand(rng, n, hkv, D)
    full, full_lse = causal_attention(q, k, v, hq, hkv)
    sel = np.array([0, 3, 4, 17, 39])
    out, lse = sparse_query_attention(q[sel], sel, k, v, hq, hkv)
    assert np.array_equal(out, full[sel]) and np.array_equal(lse, full_lse[sel])


def test_future_keys_are_masked():
    rng = np.random.default_rng(8)
    n, hq, hkv, D = 30, 4, 1, 32
    q, k, v = _rand(rng, 5, hq, D), _rand(rng, n, hkv, D), _rand(rng, n, hkv, D)
    pos = np.array([2, 9, 10, 20, 29])
    out, _ = sparse_query_attention(q, pos, k, v, hq, hkv)
    k2, v2 = k.copy(), v.copy()
    k2[11:] += 50.0
    v2[11:] -= 9.0
    out2, _ = sparse_query_attention(q, pos, k2, v2, hq, hkv)
    assert np.array_equal(out[:3], out2[:3])
    assert not np.allclose(out[3:], out2[3:])


def test_single_visible_key_and_constant_values():
    rng = np.random.default_rng(9)
    hq, hkv, D = 8, 2, 16
    q, k, v = _rand(rng, 3, hq, D), _rand(rng, 12, hkv, D), _rand(rng, 12, hkv, D)
    out, lse = sparse_query_attention(q, np.array([0, 5, 11]), k, v, hq, hkv)
    G = hq // hkv
    for h in range(hq):
        assert np.allclose(out[0, h], v[0, h // G], rtol=0, atol=1e-15)
        assert np.isclose(lse[0, h], q[0, h] @ k[0, h // G] / 4.0, rtol=1e-14)
    vc = np.broadcast_to(rng.standard_normal((1, hkv, D)), (12, hkv, D))
    out, _ = sparse_query_attention(q, np.array([0, 5, 11]), k, vc, hq, hkv)
    for h in range(hq):
        assert np.allclose(out[:, h], vc[0, h // G], rtol=1e-13, atol=1e-14)


def test_explicit_scale_and_no_visible_key():
    rng = np.random.default_rng(10)
    q, k, v = _rand(rng, 2, 2, 8), _rand(rng, 4, 1, 8), _rand(rng, 4, 1, 8)
    a, la = sparse_query_attention(q, np.array([3, -1]), k, v, 2, 1, scale=0.5)
    s = 0.5 * (k[:, 0] @ q[0, 1])
    p = np.exp(s - s.max()); p /= p.sum()
    assert np.allclose(a[0, 1], p @ v[:, 0], rtol=1e-13)
    assert np.all(a[1] == 0) and np.all(la[1] == -np.inf)
