"""Pins for the oracle's exactly rounded squared key deviation.

Closed forms on integer-valued bfloat16 inputs, a case where only a
once-rounded sum gives the right float64, exponent gaps that force the
rational path, and the invariances of a sum of squares.
"""
from fractions import Fraction

import numpy as np

from oracle import key_deviation, f64_to_bf16, bf16_to_f64


def _bf(x):
    return f64_to_bf16(np.asarray(x, dtype=np.float64))


def test_identical_rows_give_zero():
    rng = np.random.default_rng(0)
    k = _bf(rng.standard_normal((9, 2, 128)))
    assert np.array_equal(key_deviation(k, k), np.zeros(9))


def test_small_integer_closed_form():
    # bf16 holds integers up to 256 exactly: d = sum of integer squares
    rng = np.random.default_rng(1)
    a = rng.integers(-100, 100, (5, 2, 8))
    b = rng.integers(-100, 100, (5, 2, 8))
    want = ((a - b) ** 2).reshape(5, -1).sum(axis=1).astype(np.float64)
    assert np.array_equal(key_deviation(_bf(b), _bf(a)), want)


def test_sum_is_rounded_once():
    # one term 2**54 and 1023 terms 1: exact sum 2**54 + 1023, whose nearest
    # float64 is 2**54 + 1024 (spacing 4); a left-to-right float sum gives 2**54
    a = np.zeros((1, 8, 128)); a[0, 0, 0] = 2.0 ** 27; a.reshape(-1)[1:] = 1.0
    b = np.zeros_like(a)
    d = key_deviation(_bf(b), _bf(a))
    assert d[0] == 2.0 ** 54 + 1024.0
    naive = 0.0
    for t in a.reshape(-1):
        naive += t * t
    assert naive == 2.0 ** 54


def test_large_exponent_gap_uses_exact_rationals():
    # differences with more than 26 significant bits square inexactly in
    # float64; the oracle must still return the correctly rounded sum
    a = np.array([[[2.0 ** 40, 3.0 * 2.0 ** 30, 1.0]]])
    b = np.array([[[2.0 ** -20, -(2.0 ** -35), 2.0 ** 60]]])
    d = key_deviation(_bf(b), _bf(a))
    av, bv = bf16_to_f64(_bf(a)).ravel(), bf16_to_f64(_bf(b)).ravel()
    exact = sum((Fraction(x) - Fraction(y)) ** 2 for x, y in zip(av.tolist(), bv.tolist()))
    # independent integer arithmetic: scale everything by 2**35
    ai = [int(Fraction(x) * 2 ** 35) for x in av.tolist()]
    bi = [int(Fraction(y) * 2 ** 35) for y in bv.tolist()]
    s = sum((x - y) ** 2 for x, y in zip(ai, bi))
    assert Fraction(s, 2 ** 70) == exact
    assert d[0] == float(Fraction(s, 2 ** 70))


def test_power_of_two_scaling_is_exact():
    rng = np.random.default_rng(2)
    a = _bf(rng.standard_normal((6, 2, 32)))
    b = _bf(rng.standard_normal((6, 2, 32)))
    d = key_deviation(b, a)
    for m in (-7, 3, 11):
        s = 2.0 ** m
        ds = key_deviation(_bf(bf16_to_f64(b) * s), _bf(bf16_to_f64(a) * s))
        assert np.array_equal(ds, d * s * s)


def test_symmetry_and_permutation_invariance():
    rng = np.random.default_rng(3)
    a = _bf(rng.standard_normal((4, 4, 16)))
    b = _bf(rng.standard_normal((4, 4, 16)))
    d = key_deviation(b, a)
    assert np.array_equal(d, key_deviation(a, b))
    perm = rng.permutation(64)
    ap = a.reshape(4, -1)[:, perm].reshape(a.shape)
    bp = b.reshape(4, -1)[:, perm].reshape(b.shape)
    assert np.array_equal(d, key_deviation(bp, ap))
    # sign flip of both inputs
    assert np.array_equal(d, key_deviation(b ^ np.uint16(0x8000), a ^ np.uint16(0x8000)))


def test_zeroed_separator_rows_deviate_by_squared_norm():
    # a zeroed cached row (separator tokens, Section 3.2) deviates by |k_fresh|^2
    rng = np.random.default_rng(4)
    kf = _bf(rng.standard_normal((3, 2, 16)))
    zero = np.zeros_like(kf)
    want = [float(sum(Fraction(x) ** 2 for x in bf16_to_f64(kf[r]).ravel().tolist())) for r in range(3)]
    assert np.array_equal(key_deviation(zero, kf), np.array(want))


def test_zero_cached_row_gives_the_sum_of_squares_of_the_fresh_key():
    # separator slots have all-zero cached K: d is then the squared norm of
    # the recomputed key, here integers so the exact value is known
    rng = np.random.default_rng(5)
    a = rng.integers(-200, 200, (4, 8, 128))
    want = (a.astype(np.int64) ** 2).reshape(4, -1).sum(axis=1).astype(np.float64)
    assert np.array_equal(key_deviation(np.zeros((4, 8, 128), dtype=np.uint16), _bf(a)), want)
