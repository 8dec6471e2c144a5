"""Pins for the recompute count and the top-k selection (brute force)."""
import math

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import recompute_count, select_topk, selection


def _brute(d, k):
    order = sorted(range(len(d)), key=lambda r: (-float(d[r]), r))
    return sorted(order[:k])


def test_recompute_count_values():
    assert recompute_count(0.15, 124000) == 18600
    assert recompute_count(0.15, 1024) == 153
    assert recompute_count(0.15, 4000) == 600
    assert recompute_count(0.05, 32000) == 1600
    assert recompute_count(0.30, 32000) == 9600
    assert recompute_count(1.0, 77) == 77
    assert recompute_count(0.0, 77) == 0
    assert recompute_count(-0.1, 10) == -1
    assert recompute_count(1.5, 10) == -1
    assert recompute_count(float("nan"), 10) == -1
    # the product is taken in float64: 0.29 * 100 = 28.999999999999996
    assert recompute_count(0.29, 100) == 28


@settings(max_examples=200, deadline=None)
@given(st.lists(st.integers(0, 6), min_size=1, max_size=60), st.data())
def test_topk_matches_brute_force_with_ties(vals, data):
    d = np.array(vals, dtype=np.float64) * 0.25
    k = data.draw(st.integers(0, len(d)))
    assert list(select_topk(d, k)) == _brute(d, k)


def test_topk_edge_cases():
    d = np.array([3.0, 1.0, 3.0, 2.0])
    assert list(select_topk(d, 0)) == []
    assert list(select_topk(d, 4)) == [0, 1, 2, 3]
    assert list(select_topk(np.full(9, 5.0), 4)) == [0, 1, 2, 3]
    assert list(select_topk(d, 1)) == [0]           # tie 3.0: lower row first
    assert list(select_topk(d, 3)) == [0, 2, 3]
    z = np.array([0.0, -0.0, 0.0])
    assert list(select_topk(z, 2)) == [0, 1]        # -0.0 == +0.0
    assert list(select_topk(np.array([0.0, np.inf, 1e308]), 1)) == [1]


def test_selection_appends_query_rows():
    d = np.array([0.5, 2.0, 1.0, 0.1])
    s = selection(d, 2, 4, 7)
    assert list(s) == [1, 2, 4, 5, 6]
