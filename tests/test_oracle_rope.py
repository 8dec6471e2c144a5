"""Pins for the oracle's RoPE rotation and chunk position adjustment.

What the paper fixes: keys are moved to their new positions (Section 1,
Section 2 PIE, Section 3.4); the composition law of rotations makes a
shift by delta equal to encoding at p + delta from scratch.  The rotation
itself is checked against a hand-worked D=4 example and against Hugging
Face's Llama implementation (an independent library routine).
"""
import math

import numpy as np
import pytest
import torch

from oracle import inv_freq, rope_rotate, rope_shift, chunk_row0, chunk_delta, f64_to_bf16


def test_inv_freq_closed_form():
    f = inv_freq(128, 500000.0)
    assert f.shape == (64,)
    assert f[0] == 1.0
    assert math.isclose(f[1], 500000.0 ** (-1.0 / 64), rel_tol=1e-15)
    assert math.isclose(f[63], 500000.0 ** (-126.0 / 128), rel_tol=1e-15)
    assert np.all(np.diff(f) < 0)


def test_rotation_hand_worked_d4():
    # D = 4, theta = 100 -> f = [1, 0.1]; pairs are (x0, x2) and (x1, x3)
    x = np.array([[[1.0, 2.0, 3.0, 4.0]]])
    out = rope_rotate(x, np.array([1]), inv_freq(4, 100.0))[0, 0]
    c1, s1, c01, s01 = math.cos(1), math.sin(1), math.cos(0.1), math.sin(0.1)
    want = [1 * c1 - 3 * s1, 2 * c01 - 4 * s01, 3 * c1 + 1 * s1, 4 * c01 + 2 * s01]
    assert np.allclose(out, want, rtol=0, atol=1e-15)


def test_rotation_matches_huggingface_llama():
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    rng = np.random.default_rng(0)
    D, H, n, theta = 128, 3, 37, 500000.0
    x = rng.standard_normal((n, H, D))
    pos = rng.integers(0, 130000, n)
    f = inv_freq(D, theta)
    ours = rope_rotate(x, pos, f)
    # HF layout: [batch, heads, seq, D]; cos/sin [batch, seq, D]
    fr = torch.from_numpy(np.outer(pos.astype(np.float64), f))
    emb = torch.cat([fr, fr], dim=-1)[None]
    xt = torch.from_numpy(x).permute(1, 0, 2)[None]
    hf, _ = apply_rotary_pos_emb(xt, xt, emb.cos(), emb.sin())
    hf = hf[0].permute(1, 0, 2).numpy()
    assert np.allclose(ours, hf, rtol=0, atol=1e-9)


def test_shift_equals_encoding_from_scratch():
    rng = np.random.default_rng(1)
    D, Hkv = 128, 2
    chunk_len = [5, 9, 3, 11]
    n = sum(chunk_len)
    f = inv_freq(D, 500000.0)
    raw = rng.standard_normal((n, Hkv, D))
    local = np.concatenate([np.arange(L) for L in chunk_len])
    cached = rope_rotate(raw, local, f)                    # chunk computed alone
    shifted = rope_shift(cached, chunk_len, f)
    scratch = rope_rotate(raw, np.arange(n), f)            # full-context positions
    assert np.allclose(shifted, scratch, rtol=0, atol=1e-10)


def test_shift_with_old_positions_and_large_offsets():
    rng = np.random.default_rng(2)
    D = 64
    chunk_len = [4, 6]
    old = [1000, 77]
    f = inv_freq(D, 10000.0)
    raw = rng.standard_normal((10, 1, D))
    cached_pos = np.concatenate([old[0] + np.arange(4), old[1] + np.arange(6)])
    cached = rope_rotate(raw, cached_pos, f)
    shifted = rope_shift(cached, chunk_len, f, old_pos0=old)
    assert np.allclose(shifted, rope_rotate(raw, np.arange(10), f), atol=1e-10)
    assert list(chunk_delta(chunk_len, old)) == [-1000, 4 - 77]


def test_delta_zero_is_identity_and_first_chunk_unmoved():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((7, 2, 16))
    f = inv_freq(16, 500000.0)
    assert np.array_equal(rope_rotate(x, np.zeros(7, dtype=int), f), x)
    out = rope_shift(x, [3, 4], f)
    assert np.array_equal(out[:3], x[:3])
    assert list(chunk_row0([3, 4])) == [0, 3]


def test_pair_norms_preserved_and_pair0_angle_is_delta():
    rng = np.random.default_rng(4)
    D = 128
    f = inv_freq(D, 500000.0)
    x = rng.standard_normal((50, 4, D))
    pos = rng.integers(-5000, 130000, 50)
    y = rope_rotate(x, pos, f)
    h = D // 2
    assert np.allclose(x[..., :h] ** 2 + x[..., h:] ** 2, y[..., :h] ** 2 + y[..., h:] ** 2, rtol=1e-12)
    # f_0 = 1: unit vector on pair 0 turns by exactly delta radians
    e = np.zeros((1, 1, D)); e[0, 0, 0] = 1.0
    for delta in (1, 250, 7750, 116250):
        z = rope_rotate(e, np.array([delta]), f)[0, 0]
        assert math.isclose(z[0], math.cos(delta), abs_tol=1e-12)
        assert math.isclose(z[h], math.sin(delta), abs_tol=1e-12)


def test_shift_accepts_bf16_bits():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((6, 1, 8))
    bits = f64_to_bf16(x)
    from oracle import bf16_to_f64
    f = inv_freq(8, 100.0)
    assert np.array_equal(rope_shift(bits, [2, 4], f), rope_shift(bf16_to_f64(bits), [2, 4], f))


def test_llama31_scaled_table_and_shift_identity():
    # the scaled table keeps the fast pairs, slows the slow ones by 8 and
    # is monotone in between; the shift identity holds for any table
    from _rope_tables import llama31_inv_freq
    f0 = inv_freq(128, 500000.0)
    f = llama31_inv_freq()
    wl = 2 * np.pi / f0
    assert np.array_equal(f[wl < 2048], f0[wl < 2048])
    assert np.allclose(f[wl > 8192], f0[wl > 8192] / 8, rtol=0, atol=0)
    assert np.all(np.diff(f) < 0) and np.all(f <= f0) and np.all(f >= f0 / 8)
    rng = np.random.default_rng(21)
    x = rng.standard_normal((5, 2, 128))
    p = np.array([0, 3, 100, 4000, 70000])
    d = 12345
    a = rope_rotate(rope_rotate(x, p, f), np.full(5, d), f)
    b = rope_rotate(x, p + d, f)
    # angles reach ~8.2e4 rad, whose float64 spacing is ~1.5e-11
    assert np.max(np.abs(a - b)) < 1e-10


def test_yarn_table_and_shift_identity():
    # YaRN (Qwen2.5): pairs that turn more than 32 times over the original
    # context keep their frequency, those turning less than once are divided
    # by the factor 4, the band between is monotone; the shift identity holds
    from _rope_tables import yarn_inv_freq
    f0 = inv_freq(128, 1e6)
    f = yarn_inv_freq()
    turns = 32768 * f0 / (2 * np.pi)
    assert np.array_equal(f[turns > 32], f0[turns > 32])
    assert np.array_equal(f[turns < 1], f0[turns < 1] / 4)
    assert 0 < np.sum((turns >= 1) & (turns <= 32)) < 64
    assert np.all(np.diff(f) < 0) and np.all(f <= f0) and np.all(f >= f0 / 4)
    rng = np.random.default_rng(23)
    x = rng.standard_normal((5, 2, 128))
    p = np.array([0, 3, 100, 40000, 120000])
    d = 65432
    a = rope_rotate(rope_rotate(x, p, f), np.full(5, d), f)
    b = rope_rotate(x, p + d, f)
    assert np.max(np.abs(a - b)) < 1e-10
