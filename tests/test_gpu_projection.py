"""GPU parity of the projection GEMM (kvc_projection) against the oracle.

The kernel sums exact bf16 products in float32 on the matrix cores and
rounds once to bf16 after the residual addition.  Bars:
* bit-exact where the float32 sums are exact (small integers): the result
  is then the exact value rounded once to bf16, as the oracle's;
* elsewhere one bf16 rounding plus a float32-accumulation bound derived
  from k (tests/_proj.py).
Shapes: ragged m and n (tile tails), k from 64 to 14336, gathered rows
with out-of-range entries, residuals in and out of place, and the four
projections of a Llama-3.1-8B layer on the 18,856 rows selected at 124k
(sampled rows against the oracle).
"""
import numpy as np
import pytest
import torch

import oracle
from _gpu import up, down_bf16, empty_bf16
from _proj import projection_close

pytestmark = pytest.mark.gpu


def _run(K, a, w, rows=None, res=None, in_place=False):
    m = len(rows) if rows is not None else a.shape[0]
    n, k = w.shape
    ta, tw = up(a), up(w)
    tr = up(res) if res is not None else None
    c = tr if in_place else empty_bf16(m, n)
    K.kvc_projection(m, n, k, ta, a.shape[0], None if rows is None else up(rows.astype(np.int32)), tw, tr, c)
    torch.cuda.synchronize()
    return down_bf16(c)


def _check(got_bits, a, w, rows, res, k):
    ok, excess = projection_close(got_bits, a, w, rows=rows, residual=res)
    assert ok, excess


def _bf(rng, shape, scale=1.0):
    return oracle.f64_to_bf16(rng.standard_normal(shape) * scale)


@pytest.mark.parametrize("m,n,k", [(1, 8, 64), (37, 264, 128), (255, 256, 64), (257, 520, 192), (300, 1024, 4096),
                                   (513, 776, 640)])
def test_projection_shapes(K, m, n, k):
    rng = np.random.default_rng(m + n + k)
    a, w = _bf(rng, (m, k)), _bf(rng, (n, k), 0.05)
    _check(_run(K, a, w), a, w, None, None, k)


def test_projection_small_integers_bit_exact(K):
    # products and float32 sums exact: one rounding to bf16, as the oracle
    rng = np.random.default_rng(40)
    m, n, k = 333, 264, 256
    a = oracle.f64_to_bf16(rng.integers(-3, 4, (m, k)).astype(np.float64))
    w = oracle.f64_to_bf16(rng.integers(-3, 4, (n, k)).astype(np.float64))
    res = oracle.f64_to_bf16(rng.integers(-100, 100, (m, n)).astype(np.float64))
    got = _run(K, a, w, res=res)
    want = oracle.f64_to_bf16(oracle.projection(a, w, residual=res))
    assert np.array_equal(oracle.bf16_to_f64(got), oracle.bf16_to_f64(want))


def test_projection_gather_residual_and_in_place(K):
    rng = np.random.default_rng(41)
    n_a, m, n, k = 700, 301, 512, 1024
    a, w = _bf(rng, (n_a, k)), _bf(rng, (n, k), 0.03)
    rows = rng.integers(0, n_a, m).astype(np.int64)
    rows[[3, 100, 299]] = [-1, n_a, 2**31 - 1]      # out of range: zero product rows
    res = _bf(rng, (m, n))
    got = _run(K, a, w, rows=rows, res=res)
    _check(got, a, w, rows, res, k)
    assert np.array_equal(got[[3, 100, 299]], res[[3, 100, 299]])
    # the residual updated in place gives the same bits
    assert np.array_equal(_run(K, a, w, rows=rows, res=res, in_place=True), got)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name,n,k,residual", [("qkv", 6144, 4096, False), ("o", 4096, 4096, True),
                                               ("gate_up", 28672, 4096, False), ("down", 4096, 14336, True)])
def test_projection_llama8b_selected_rows(K, name, n, k, residual):
    # the four projections of a Llama-3.1-8B layer on the 18,856 rows selected
    # at 124k, 15 %; inputs drawn on the device, 24 sampled rows (all columns)
    # checked against the oracle
    m = 18856
    g = torch.Generator(device="cuda:0")
    g.manual_seed(50 + k + n)
    a = (torch.randn((m, k), generator=g, device="cuda:0")).to(torch.bfloat16).view(torch.int16)
    w = (torch.randn((n, k), generator=g, device="cuda:0") * 0.02).to(torch.bfloat16).view(torch.int16)
    res = (torch.randn((m, n), generator=g, device="cuda:0")).to(torch.bfloat16).view(torch.int16) if residual else None
    c = empty_bf16(m, n)
    K.kvc_projection(m, n, k, a, m, None, w, res, c)
    torch.cuda.synchronize()
    rng = np.random.default_rng(n)
    rows = np.unique(np.concatenate([[0, m - 1], rng.choice(m, 22, replace=False)]))
    idx = torch.from_numpy(rows).cuda()
    a_rows, w_h = down_bf16(a[idx]), down_bf16(w)
    r_rows = down_bf16(res[idx]) if residual else None
    _check(down_bf16(c[idx]), a_rows, w_h, None, r_rows, k)
