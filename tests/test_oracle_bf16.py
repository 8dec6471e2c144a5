"""Pins for the oracle's bfloat16 conversions (brute force over all bf16 values)."""
import numpy as np
import pytest
import torch

from oracle import bf16_to_f64, f64_to_bf16


def _all_finite_bf16():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    ok = np.isfinite(vals)
    return bits[ok], vals[ok]


def test_bf16_to_f64_matches_torch():
    bits, _ = _all_finite_bf16()
    t = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(bf16_to_f64(bits), t)


def test_f64_to_bf16_is_nearest_ties_even_brute_force():
    bits, vals = _all_finite_bf16()
    normal = (np.abs(vals) >= 2.0 ** -126) | (vals == 0)
    pos = np.unique(vals[normal & (vals >= 0)])           # sorted non-negative grid
    rng = np.random.default_rng(1)
    x = np.concatenate([
        rng.standard_normal(20000) * 10.0 ** rng.uniform(-30, 30, 20000),
        # exact midpoints between neighbours (ties)
        (pos[1000:1100] + pos[1001:1101]) / 2,
        -(pos[30000:30100] + pos[30001:30101]) / 2,
        [0.0, 1.0, -1.0, 3.0e38],
    ])
    x = x[(np.abs(x) >= 2.0 ** -126) & (np.abs(x) < 3.38e38)]
    got = bf16_to_f64(f64_to_bf16(x))
    ax = np.abs(x)
    i = np.searchsorted(pos, ax)                           # pos[i-1] < ax <= pos[i]
    lo, hi = pos[np.maximum(i - 1, 0)], pos[np.minimum(i, len(pos) - 1)]
    lo_bits = (lo.astype(np.float32).view(np.uint32) >> 16)
    d_lo, d_hi = ax - lo, hi - ax
    pick_lo = (d_lo < d_hi) | ((d_lo == d_hi) & (lo_bits % 2 == 0))
    want = np.where(ax == hi, hi, np.where(pick_lo, lo, hi)) * np.sign(x)
    assert np.array_equal(got, want)


def test_f64_to_bf16_rejects_out_of_range():
    with pytest.raises(ValueError):
        f64_to_bf16(np.array([np.nan]))
    with pytest.raises(ValueError):
        f64_to_bf16(np.array([1e-40]))


def test_f64_to_bf16_matches_torch_on_float32_values():
    # float32 inputs (every value a float32 holds exactly, including the
    # bf16 midpoints): torch's float32 -> bfloat16 conversion is round to
    # nearest even too
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(200000) * 10.0 ** rng.uniform(-20, 20, 200000)).astype(np.float32)
    _, vals = _all_finite_bf16()
    grid = np.unique(np.abs(vals[(np.abs(vals) >= 2.0 ** -126) & (np.abs(vals) < 2.0 ** 120)]))
    mids = ((grid[:-1] + grid[1:]) / 2).astype(np.float32)
    x = np.concatenate([x, mids, -mids])
    t = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(f64_to_bf16(x.astype(np.float64)), t)
