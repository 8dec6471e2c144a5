"""GPU parity of each hot-path kernel against the CPU oracle, via the C ABI.

Bars: bit-exact for the selection indices and the scattered rows; the
adjusted keys and deviations are compared bit-exactly too (both sides round
once from float64); attention outputs within 2e-2 abs + 1e-2 rel.
"""

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from _gpu import up, down_bf16, empty_bf16, bytes_buf, within_tol, LSE_ATOL
from _inputs import build

pytestmark = pytest.mark.gpu


def _same_values(a_bits, b_bits):
    """bf16 bit arrays equal as numbers (+0 == -0)."""
    return np.array_equal(oracle.bf16_to_f64(a_bits), oracle.bf16_to_f64(b_bits))


def _plan(K, L):
    pb = K.kvc_plan_bytes(L)
    plan = bytes_buf(pb)
    plan = K.kvc_plan_upload(L, plan, pb)
    return plan


# ---------------------------------------------------------------- a1 shift
SHIFT_CASES = {
    "tiny": dict(chunk_len=[256] * 4, hkv=2, old=None),
    "4k": dict(chunk_len=[250] * 16, hkv=8, old=None),
    "ragged": dict(chunk_len=[1, 63, 64, 65, 200, 7, 129], hkv=8, old=None),
    "old_pos": dict(chunk_len=[100, 37, 64], hkv=4, old=[500, 3, 100000]),
    "many_small": dict(chunk_len=list(np.random.default_rng(9).integers(1, 40, 944)), hkv=1, old=None),
    "empty_chunks": dict(chunk_len=[0, 5, 0, 70], hkv=2, old=None),
    # 16,384 reused rows or more with fewer than 8 kv heads: tiles of 128,
    # 64 and 32 rows (1024 units each), ragged tails
    "long_1head": dict(chunk_len=[7750, 1000, 513, 9000], hkv=1, old=None),
    "long_2heads": dict(chunk_len=[20000, 3, 0, 257], hkv=2, old=[0, 17, 0, 40000]),
    "long_4heads": dict(chunk_len=[16384, 129], hkv=4, old=None),
}


@pytest.mark.parametrize("name", list(SHIFT_CASES))
@pytest.mark.parametrize("in_place", [False, True])
def test_rope_shift_matches_oracle(K, name, in_place):
    c = SHIFT_CASES[name]
    cl, hkv = c["chunk_len"], c["hkv"]
    n_r = int(sum(cl))
    rng = np.random.default_rng(len(cl) * 7 + hkv)
    k_src = oracle.f64_to_bf16(rng.standard_normal((n_r + 3, hkv, 128)) * rng.lognormal(0, 0.5, (hkv, 128)))
    L = K.Layout(cl, 3, hkv, hkv, 128, 500000.0, chunk_old_pos0=c["old"])
    plan = _plan(K, L)
    src = up(k_src)
    dst = src if in_place else up(np.zeros_like(k_src))
    K.kvc_rope_shift(L, plan, src, dst)
    got = down_bf16(dst)
    want = oracle.f64_to_bf16(oracle.rope_shift(k_src[:n_r], cl, oracle.inv_freq(128, 500000.0), c["old"]))
    assert _same_values(got[:n_r], want)
    # rows past n_reused untouched
    tail = k_src[n_r:] if in_place else np.zeros_like(k_src[n_r:])
    assert np.array_equal(got[n_r:], tail)
    ok, err = within_tol(oracle.bf16_to_f64(got[:n_r]),
                         oracle.rope_shift(k_src[:n_r], cl, oracle.inv_freq(128, 500000.0), c["old"]))
    assert ok, err


def test_rope_shift_explicit_inv_freq_and_stale_plan(K):
    cl = [64, 64]
    rng = np.random.default_rng(3)
    k_src = oracle.f64_to_bf16(rng.standard_normal((128, 2, 128)))
    f = oracle.inv_freq(128, 10000.0) * 0.25          # a rescaled table
    L = K.Layout(cl, 0, 2, 2, 128, 0.0, inv_freq=f)
    plan = _plan(K, L)
    out = up(np.zeros_like(k_src))
    K.kvc_rope_shift(L, plan, up(k_src), out)
    want = oracle.f64_to_bf16(oracle.rope_shift(k_src, cl, f))
    assert _same_values(down_bf16(out), want)
    # a plan made for another layout is refused before anything is enqueued
    L2 = K.Layout([64, 63], 0, 2, 2, 128, 500000.0)
    out2 = up(np.zeros_like(k_src))
    with pytest.raises(K.KvcError) as e:
        K.kvc_rope_shift(L2, plan, up(k_src), out2)
    assert e.value.status == K.KVC_ERR_INVALID_ARG and "another layout" in str(e.value)
    torch.cuda.synchronize()
    assert not down_bf16(out2).any()


def test_plan_upload_through_pinned_staging(K):
    # the upload only enqueues its copy when the caller supplies pinned
    # staging memory; the plan then works like one uploaded with a wait
    cl = [100, 37, 64, 300]
    rng = np.random.default_rng(4)
    k_src = oracle.f64_to_bf16(rng.standard_normal((sum(cl), 4, 128)))
    L = K.Layout(cl, 0, 8, 4, 128, 500000.0, chunk_old_pos0=[7, 0, 3, 1000])
    pb = K.kvc_plan_bytes(L)
    staging = torch.empty(pb, dtype=torch.uint8).pin_memory()
    s = torch.cuda.Stream()
    buf = bytes_buf(pb)
    with torch.cuda.stream(s):
        plan = K.kvc_plan_upload(L, buf, pb, stream=s, staging=staging)
        src = up(k_src)
        out = torch.zeros_like(src)
        K.kvc_rope_shift(L, plan, src, out, stream=s)
    s.synchronize()
    want = oracle.f64_to_bf16(oracle.rope_shift(k_src, cl, oracle.inv_freq(128, 500000.0), [7, 0, 3, 1000]))
    assert _same_values(down_bf16(out), want)


def test_rope_shift_llama31_scaled_frequencies(K):
    # Llama-3.1's rescaled RoPE table (the paper's base model) through an
    # explicit inv_freq, at offsets up to ~30k rows where the slowed pairs
    # matter
    from _rope_tables import llama31_inv_freq
    f = llama31_inv_freq()
    cl = [2000] * 16
    rng = np.random.default_rng(22)
    k_src = oracle.f64_to_bf16(rng.standard_normal((sum(cl), 8, 128)) * rng.lognormal(0, 0.5, (8, 128)))
    L = K.Layout(cl, 0, 32, 8, 128, 0.0, inv_freq=f)
    plan = _plan(K, L)
    out = up(np.zeros_like(k_src))
    K.kvc_rope_shift(L, plan, up(k_src), out)
    want = oracle.rope_shift(k_src, cl, f)
    got = down_bf16(out)
    assert _same_values(got, oracle.f64_to_bf16(want))
    ok, err = within_tol(oracle.bf16_to_f64(got), want)
    assert ok, err


def test_rope_shift_yarn_frequencies(K):
    # Qwen2.5's YaRN table (the paper's second model, Section 4.1) through
    # an explicit inv_freq, with chunks moved by up to ~120k rows
    from _rope_tables import yarn_inv_freq
    f = yarn_inv_freq()
    cl = [7750] * 16
    rng = np.random.default_rng(24)
    k_src = oracle.f64_to_bf16(rng.standard_normal((sum(cl), 2, 128)) * rng.lognormal(0, 0.5, (2, 128)))
    L = K.Layout(cl, 0, 14, 2, 128, 0.0, inv_freq=f)
    plan = _plan(K, L)
    out = up(np.zeros_like(k_src))
    K.kvc_rope_shift(L, plan, up(k_src), out)
    want = oracle.rope_shift(k_src, cl, f)
    got = down_bf16(out)
    assert _same_values(got, oracle.f64_to_bf16(want))


def _bf16_via_f32(v):
    """Round float64 to float32 and then to bfloat16, both nearest-even:
    the double rounding the kernel must avoid."""
    b = np.asarray(v, dtype=np.float64).astype(np.float32).view(np.uint32).astype(np.uint64)
    return ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)


def test_rope_shift_rounds_once_at_bf16_midpoints(K):
    # about 1 value in 65,536 rounds to a float32 that lies exactly halfway
    # between two bfloat16 values although the float64 result does not; a
    # second round-to-nearest-even step then breaks the tie, wrongly in
    # about half of these cases.  16.8M values hold a few hundred of them.
    cl = [4096] * 8
    hkv = 4
    rng = np.random.default_rng(31)
    k_src = oracle.f64_to_bf16(rng.standard_normal((sum(cl), hkv, 128)) * rng.lognormal(0, 0.5, (hkv, 128)))
    L = K.Layout(cl, 0, hkv, hkv, 128, 500000.0)
    plan = _plan(K, L)
    out = up(np.zeros_like(k_src))
    K.kvc_rope_shift(L, plan, up(k_src), out)
    got = down_bf16(out)
    r = oracle.rope_shift(k_src, cl, oracle.inv_freq(128, 500000.0))
    want = oracle.f64_to_bf16(r)
    f32 = r.astype(np.float32)
    mids = ((f32.view(np.uint32) & 0xFFFF) == 0x8000) & (f32.astype(np.float64) != r)
    naive = _bf16_via_f32(r)
    assert mids.sum() >= 100
    assert (naive[mids] != want[mids]).sum() >= 20      # the cases rounding twice gets wrong
    assert np.array_equal(naive[~mids], want[~mids])    # and only these
    assert _same_values(got[mids], want[mids])
    assert _same_values(got, want)


def _bf16_round_with_subnormals(v):
    """Nearest-even bfloat16 of float64 values of magnitude below 2^-126
    too: there bfloat16 is the fixed-point grid of step 2^-133 (its
    subnormals), so rounding is rint on v * 2^133, exact in float64."""
    v = np.asarray(v, dtype=np.float64)
    small = np.abs(v) < 2.0 ** -126
    out = np.zeros(v.shape, dtype=np.uint16)
    out[~small] = oracle.f64_to_bf16(v[~small])
    g = np.rint(v[small] * 2.0 ** 133) * 2.0 ** -133      # a multiple of 2^-133 below 2^-126 (or 2^-126 itself)
    out[small] = (g.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    return out


def test_rope_shift_subnormal_range(K):
    # keys near and below 2^-126: inputs include bfloat16 subnormals, and
    # rotated values that fall below 2^-126 round to the subnormal grid
    # (gradual underflow), not to zero
    cl = [64, 64, 64]
    rng = np.random.default_rng(32)
    n = sum(cl)
    exp = rng.integers(0, 4, (n, 1, 128)).astype(np.uint16)             # bfloat16 exponent fields 0..3
    bits = (rng.integers(0, 2, (n, 1, 128)).astype(np.uint16) << 15) | (exp << 7) | rng.integers(0, 128, (n, 1, 128)).astype(np.uint16)
    L = K.Layout(cl, 0, 1, 1, 128, 10000.0)
    plan = _plan(K, L)
    out = up(np.zeros_like(bits))
    K.kvc_rope_shift(L, plan, up(bits), out)
    got = down_bf16(out)
    r = oracle.rope_shift(bits, cl, oracle.inv_freq(128, 10000.0))
    want = _bf16_round_with_subnormals(r)
    assert (np.abs(r) < 2.0 ** -126).mean() > 0.2 and np.count_nonzero(r) > 0.9 * r.size
    assert _same_values(got, want)


# ------------------------------------------------------------ a2 deviation
def _dev_gpu(K, kc, kf):
    n, hkv = kc.shape[0], kc.shape[1]
    d = torch.empty(max(n, 1), dtype=torch.float64, device="cuda:0")
    K.kvc_kv_deviation(n, hkv, 128, up(kc), up(kf), d)
    return d[:n].cpu().numpy()


@pytest.mark.parametrize("hkv,n", [(8, 1000), (2, 333), (1, 5), (4, 1), (16, 77), (8, 4097)])
def test_kv_deviation_is_exactly_rounded(K, hkv, n):
    rng = np.random.default_rng(hkv * 1000 + n)
    kc = oracle.f64_to_bf16(rng.standard_normal((n, hkv, 128)))
    kf = oracle.f64_to_bf16(oracle.bf16_to_f64(kc) + 0.1 * rng.standard_normal((n, hkv, 128)))
    assert np.array_equal(_dev_gpu(K, kc, kf), oracle.key_deviation(kc, kf))


def test_kv_deviation_special_rows(K):
    n, hkv = 6, 8
    kc = np.zeros((n, hkv, 128), dtype=np.uint16)
    kf = np.zeros((n, hkv, 128))
    kf[0, 0, 0] = 2.0 ** 27                       # 2^54 + 1023 ones -> 2^54 + 1024
    kf[0].reshape(-1)[1:] = 1.0
    rng = np.random.default_rng(0)
    kf[1] = rng.standard_normal((hkv, 128))
    kf[2] = kf[1].reshape(-1)[rng.permutation(hkv * 128)].reshape(hkv, 128)   # same exact sum
    kf[3] = 0.0                                   # identical rows
    kf[4] = rng.standard_normal((hkv, 128)) * 1e-30
    kf[5] = rng.standard_normal((hkv, 128)) * 1e30
    kfb = oracle.f64_to_bf16(kf)
    got = _dev_gpu(K, kc, kfb)
    want = oracle.key_deviation(kc, kfb)
    assert got[0] == 2.0 ** 54 + 1024.0
    assert got[1] == got[2]
    assert got[3] == 0.0
    assert np.array_equal(got, want)


def _random_bf16_bits(rng, shape, exp_lo=0, exp_hi=254, p_zero=0.2):
    """bfloat16 bit patterns with uniform exponent fields in [exp_lo, exp_hi]
    (0 = subnormal), random mantissas and signs, and some exact zeros."""
    e = rng.integers(exp_lo, exp_hi + 1, shape).astype(np.uint16)
    m = rng.integers(0, 128, shape).astype(np.uint16)
    s = rng.integers(0, 2, shape).astype(np.uint16)
    bits = (s << 15) | (e << 7) | m
    bits[rng.random(shape) < p_zero] = 0
    return bits.astype(np.uint16)


@pytest.mark.parametrize("hkv", [1, 2, 3, 4, 8, 16])
def test_kv_deviation_rounds_once_where_double_double_does_not(K, hkv):
    # exact sum 2^53 + 1 + 2^-100: its float64 is 2^53 + 2, while a
    # double-double whose low word is rounded gives 2^53 (the tie goes to even)
    kc = np.zeros((4, hkv, 128), dtype=np.uint16)
    kf = np.zeros((4, hkv, 128))
    kf[0].reshape(-1)[:4] = [2.0 ** 26, 2.0 ** 26, 1.0, 2.0 ** -50]
    kf[1].reshape(-1)[-4:] = [2.0 ** -50, 1.0, 2.0 ** 26, 2.0 ** 26]
    kf[2].reshape(-1)[::37][:4] = [1.0, 2.0 ** 26, 2.0 ** -50, 2.0 ** 26]
    kf[3].reshape(-1)[:3] = [2.0 ** 26, 2.0 ** 26, 1.0]          # exact tie: 2^53 + 1 -> 2^53
    kfb = oracle.f64_to_bf16(kf)
    got = _dev_gpu(K, kc, kfb)
    assert list(got[:3]) == [2.0 ** 53 + 2] * 3
    assert got[3] == 2.0 ** 53
    assert np.array_equal(got, oracle.key_deviation(kc, kfb))


@pytest.mark.parametrize("hkv", [1, 2, 4, 8])
def test_kv_deviation_mixed_magnitudes(K, hkv):
    # terms spanning the whole bfloat16 range (subnormals to 2^127), signs,
    # zeros: every row leaves the float64 fast path and is summed exactly
    rng = np.random.default_rng(100 + hkv)
    n = 300
    kc = _random_bf16_bits(rng, (n, hkv, 128))
    kf = _random_bf16_bits(rng, (n, hkv, 128))
    # rows of narrower spans (30 to 60 binades), near the fast path's limits
    for i in range(0, n, 3):
        lo = int(rng.integers(1, 180))
        span = int(rng.integers(30, 60))
        kc[i] = _random_bf16_bits(rng, (hkv, 128), lo, lo + span, 0.5)
        kf[i] = _random_bf16_bits(rng, (hkv, 128), lo, lo + span, 0.5)
    assert np.array_equal(_dev_gpu(K, kc, kf), oracle.key_deviation(kc, kf))


@pytest.mark.parametrize("hkv", [1, 8])
def test_kv_deviation_permuted_rows_tie(K, hkv):
    # rows holding the same terms in different orders have the same exact
    # sum, hence the same value (what the top-k tie rule relies on)
    rng = np.random.default_rng(7 + hkv)
    for lo, span in [(100, 20), (60, 50), (1, 253)]:
        base_f = _random_bf16_bits(rng, (hkv * 128,), lo, lo + span, 0.3)
        base_c = _random_bf16_bits(rng, (hkv * 128,), lo, lo + span, 0.3)
        perms = [rng.permutation(hkv * 128) for _ in range(40)]
        kf = np.stack([base_f[p].reshape(hkv, 128) for p in perms])
        kc = np.stack([base_c[p].reshape(hkv, 128) for p in perms])
        got = _dev_gpu(K, kc, kf)
        assert np.all(got == got[0])
        assert got[0] == oracle.key_deviation(kc[:1], kf[:1])[0]


@pytest.mark.parametrize("hkv", [1, 8])
def test_kv_deviation_small_elements(K, hkv):
    # ordinary rows plus a few elements 2^28..2^36 below the rest: the
    # float64 path must certify (or redo) these rows, whose error terms are
    # no longer multiples of a coarse power of two
    rng = np.random.default_rng(31 + hkv)
    n = 2000
    c = rng.standard_normal((n, hkv, 128)) * 30
    c.reshape(n, -1)[:, :3] = rng.choice([-1, 1], (n, 3)) * 2.0 ** rng.integers(-36, -28, (n, 3))
    f = c + 30 * rng.standard_normal((n, hkv, 128))
    f.reshape(n, -1)[:, :3] = 0
    kc, kf = oracle.f64_to_bf16(c), oracle.f64_to_bf16(f)
    assert np.array_equal(_dev_gpu(K, kc, kf), oracle.key_deviation(kc, kf))


# ---------------------------------------------------------------- a3 top-k
def _topk_gpu(K, d, k):
    n = len(d)
    ws_b = K.kvc_select_topk_workspace(n)
    ws = bytes_buf(ws_b)
    out = torch.full((max(k, 1),), -7, dtype=torch.int32, device="cuda:0")
    K.kvc_select_topk(torch.from_numpy(np.ascontiguousarray(d, dtype=np.float64)).cuda(), n, k, out, ws, ws_b)
    return out[:k].cpu().numpy()


# up to 16,384 candidates the selection runs in one workgroup, up to
# 262,144 in one launch with grid barriers, above it in the multi-launch
# path: all three are covered, with both boundaries
@pytest.mark.parametrize("n,k", [(1, 0), (1, 1), (10, 3), (2047, 300), (2048, 2048), (2049, 1),
                                 (124000, 18600), (300001, 45000), (5000, 0), (5000, 4999),
                                 (16384, 2457), (16384, 16383), (16384, 1), (16385, 2457), (16385, 16384),
                                 (32000, 4800), (32768, 4915), (32768, 1), (32768, 32767), (32769, 4915),
                                 (32769, 32768), (262144, 39321), (262144, 1), (262144, 262143),
                                 (262145, 39321), (262145, 262144)])
def test_select_topk_matches_oracle(K, n, k):
    rng = np.random.default_rng(n + k)
    d = rng.standard_normal(n) ** 2 * rng.lognormal(0, 2, n)
    assert np.array_equal(_topk_gpu(K, d, k), oracle.select_topk(d, k))


@pytest.mark.parametrize("n", [9000, 20000, 40000])
@pytest.mark.parametrize("levels", [1, 2, 7, 1000])
def test_select_topk_ties_go_to_lower_rows(K, levels, n):
    rng = np.random.default_rng(levels)
    d = rng.integers(0, levels, n).astype(np.float64)
    d[rng.integers(0, n, 50)] = -0.0
    for k in (1, 1234, n // 2, n - 1):
        assert np.array_equal(_topk_gpu(K, d, k), oracle.select_topk(d, k))


@pytest.mark.parametrize("m", [3000, 12000, 20000])
def test_select_topk_signed_and_extreme_values(K, m):
    rng = np.random.default_rng(5)
    d = np.concatenate([rng.standard_normal(m) * 1e300, rng.standard_normal(m) * 1e-300,
                        [np.inf, -np.inf, 0.0, -0.0, 5e-324, -5e-324]])
    for k in (1, 7, m, 2 * m - 1):
        assert np.array_equal(_topk_gpu(K, d, k), oracle.select_topk(d, k))


# -------------------------------------------------------------- a4 scatter
@pytest.mark.parametrize("compact", [0, 1])
def test_scatter_rows(K, compact):
    rng = np.random.default_rng(compact)
    N, hkv = 300, 8
    kc = rng.integers(0, 65535, (N, hkv, 128), dtype=np.uint16)
    vc = rng.integers(0, 65535, (N, hkv, 128), dtype=np.uint16)
    sel = np.array([0, 5, 17, 299, -1, 300, 150], dtype=np.int32)   # two invalid entries skipped
    nf = len(sel) if compact else N
    kf = rng.integers(0, 65535, (nf, hkv, 128), dtype=np.uint16)
    vf = rng.integers(0, 65535, (nf, hkv, 128), dtype=np.uint16)
    tkc, tvc = up(kc), up(vc)
    K.kvc_scatter_rows(up(sel), len(sel), compact, up(kf), up(vf), nf, tkc, tvc, N, hkv, 128)
    wk, wv = kc.copy(), vc.copy()
    for i, r in enumerate(sel):
        if 0 <= r < N:
            s = i if compact else r
            wk[r], wv[r] = kf[s], vf[s]
    assert np.array_equal(down_bf16(tkc), wk) and np.array_equal(down_bf16(tvc), wv)


# ------------------------------------------------------------ a5 attention
def _attn_gpu(K, q, pos, k, v, hq, hkv, q_rows=None, scale=0.0, split=False):
    n_sel = len(pos)
    out = empty_bf16(max(n_sel, 1), hq, 128)
    lse = torch.empty((max(n_sel, 1), hq), dtype=torch.float32, device="cuda:0")
    wb = K.kvc_attention_workspace(n_sel, hq, hkv, 128) if split else 0
    ws = bytes_buf(wb) if wb else None
    K.kvc_sparse_query_attention(up(q), q.shape[0], None if q_rows is None else up(q_rows.astype(np.int32)),
                                 up(np.asarray(pos, dtype=np.int32)), n_sel, up(k), up(v), k.shape[0],
                                 hq, hkv, 128, scale, out, lse, ws, wb)
    return oracle.bf16_to_f64(down_bf16(out)[:n_sel]), lse[:n_sel].cpu().numpy()


def _qkv(rng, n_q, n_kv, hq, hkv):
    s = lambda h: rng.lognormal(0, 0.5, (h, 128))
    q = oracle.f64_to_bf16(rng.standard_normal((n_q, hq, 128)) * s(hq))
    k = oracle.f64_to_bf16(rng.standard_normal((n_kv, hkv, 128)) * s(hkv))
    v = oracle.f64_to_bf16(rng.standard_normal((n_kv, hkv, 128)) * s(hkv))
    return q, k, v


@pytest.mark.parametrize("hq,hkv", [(8, 2), (32, 8), (4, 4), (6, 2), (16, 2), (2, 1)])
def test_attention_gqa_layouts(K, hq, hkv):
    rng = np.random.default_rng(hq * 100 + hkv)
    n_kv = 777
    pos = np.sort(rng.choice(n_kv, 150, replace=False))
    q, k, v = _qkv(rng, 150, n_kv, hq, hkv)
    got, lse = _attn_gpu(K, q, pos, k, v, hq, hkv)
    want, wl = oracle.sparse_query_attention(q, pos, k, v, hq, hkv)
    ok, err = within_tol(got, want)
    assert ok, err
    assert np.allclose(lse, wl, rtol=0, atol=LSE_ATOL)


@pytest.mark.parametrize("seed", range(24))
def test_attention_random_shapes(K, seed):
    # seeded random shapes: kv heads, group size, key count, selection size,
    # sorted or unsorted positions, gather or compact queries, key-range
    # split or not, default or explicit scale
    rng = np.random.default_rng(1000 + seed)
    hkv = int(rng.choice([1, 2, 4, 8]))
    hq = hkv * int(rng.choice([1, 2, 3, 4, 8]))
    n_kv = int(rng.integers(1, 3000))
    n_sel = int(rng.integers(1, 400))
    pos = rng.integers(0, n_kv, n_sel)
    if seed % 2 == 0:
        pos = np.sort(pos)
    gather = seed % 3 == 0
    n_q = n_sel + 17 if gather else n_sel
    q, k, v = _qkv(rng, n_q, n_kv, hq, hkv)
    q_rows = rng.integers(0, n_q, n_sel) if gather else None
    scale = 0.0 if seed % 4 else float(rng.uniform(0.02, 0.2))
    got, lse = _attn_gpu(K, q, pos, k, v, hq, hkv, q_rows=q_rows, scale=scale, split=seed % 5 < 3)
    want, wl = oracle.sparse_query_attention(q if q_rows is None else q[q_rows], pos, k, v, hq, hkv, scale=scale)
    ok, err = within_tol(got, want)
    assert ok, (hq, hkv, n_kv, n_sel, err)
    assert np.allclose(lse, wl, rtol=0, atol=LSE_ATOL)


def test_attention_full_causal_and_edge_positions(K):
    rng = np.random.default_rng(11)
    n, hq, hkv = 257, 8, 2
    q, k, v = _qkv(rng, n, n, hq, hkv)
    got, lse = _attn_gpu(K, q, np.arange(n), k, v, hq, hkv)
    want, wl = oracle.causal_attention(q, k, v, hq, hkv)
    ok, err = within_tol(got, want)
    assert ok, err
    # row 0 sees only key 0: output is V[0] rounded to bf16
    assert np.array_equal(got[0], np.repeat(oracle.bf16_to_f64(v[0]), hq // hkv, axis=0))


def test_attention_gather_unsorted_clamped_and_invalid(K):
    rng = np.random.default_rng(12)
    n_kv, hq, hkv = 500, 8, 2
    q, k, v = _qkv(rng, 300, n_kv, hq, hkv)
    n_sel = 70
    q_rows = rng.integers(0, 300, n_sel)
    pos = rng.integers(0, n_kv, n_sel)               # unsorted
    pos[3] = n_kv + 50                               # clamped to n_kv - 1
    pos[4] = -3                                      # no visible key
    q_rows[5] = 300                                  # out of range row
    got, lse = _attn_gpu(K, q, pos, k, v, hq, hkv, q_rows=q_rows)
    qq = q[np.clip(q_rows, 0, 299)]
    pp = np.minimum(pos, n_kv - 1)
    pp[5] = -1
    want, wl = oracle.sparse_query_attention(qq, pp, k, v, hq, hkv)
    ok, err = within_tol(got, want)
    assert ok, err
    assert np.all(got[4] == 0) and np.all(np.isneginf(lse[4]))
    assert np.all(got[5] == 0) and np.all(np.isneginf(lse[5]))
    fin = np.isfinite(wl)
    assert np.allclose(lse[fin], wl[fin], rtol=0, atol=LSE_ATOL)


def test_attention_single_query_and_explicit_scale(K):
    rng = np.random.default_rng(13)
    q, k, v = _qkv(rng, 1, 3000, 32, 8)
    for pos in ([0], [2999], [1000]):
        got, _ = _attn_gpu(K, q, pos, k, v, 32, 8, scale=0.05)
        want, _ = oracle.sparse_query_attention(q, pos, k, v, 32, 8, scale=0.05)
        ok, err = within_tol(got, want)
        assert ok, (pos, err)


def test_attention_masks_future_keys(K):
    rng = np.random.default_rng(14)
    q, k, v = _qkv(rng, 40, 400, 8, 2)
    pos = np.sort(rng.choice(400, 40, replace=False))
    got, _ = _attn_gpu(K, q, pos, k, v, 8, 2)
    k2, v2 = k.copy(), v.copy()
    cut = pos[20] + 1
    k2[cut:] = oracle.f64_to_bf16(oracle.bf16_to_f64(k[cut:]) * 3 + 1)
    v2[cut:] = oracle.f64_to_bf16(oracle.bf16_to_f64(v[cut:]) - 5)
    got2, _ = _attn_gpu(K, q, pos, k2, v2, 8, 2)
    assert np.array_equal(got[:21], got2[:21])


def test_attention_growing_and_overflowing_maxima(K):
    # Spike keys aligned with the queries raise the row maximum by steps of
    # about 24, 48 and 200 (log2 units) at rows 100, 300 and 500; the last
    # one overflows exp2 against the earlier offset, so the kernel's rescale
    # branch must run, including the overflow case.  Negative spikes after
    # row 600 push weights far below the maximum.
    rng = np.random.default_rng(15)
    n_kv, hq, hkv = 900, 8, 2
    q = oracle.f64_to_bf16(1.0 + 0.05 * rng.standard_normal((n_kv, hq, 128)))
    kk = 0.05 * rng.standard_normal((n_kv, hkv, 128))
    for row, a in ((100, 1.5), (300, 3.0), (500, 12.0), (650, -6.0), (800, -9.0)):
        kk[row] += a
    k = oracle.f64_to_bf16(kk)
    v = oracle.f64_to_bf16(rng.standard_normal((n_kv, hkv, 128)))
    pos = np.unique(np.concatenate([[0, 99, 100, 299, 300, 499, 500, 899], rng.choice(n_kv, 150, replace=False)]))
    got, lse = _attn_gpu(K, q[pos], pos, k, v, hq, hkv)
    want, wl = oracle.sparse_query_attention(q[pos], pos, k, v, hq, hkv)
    ok, err = within_tol(got, want)
    assert ok, err
    assert np.allclose(lse, wl, rtol=0, atol=LSE_ATOL)



# ------------------------------------------------------- split key ranges
def test_attention_split_partials_far_apart(K):
    # every query sees all 5000 keys, split over 8 workgroups; keys 100-399
    # are aligned with the queries (logits near 50 in log2 units), keys
    # 4000-4099 less so (near 33), the rest are noise (near 0), so one
    # query's partial LSEs differ by 20 to 50 (log2) from split to split and
    # the merge must weight them by 2^(lse_s - max) without losing the small
    # ones' rows or overflowing
    rng = np.random.default_rng(16)
    n_kv, hq, hkv, n_q = 5000, 8, 2, 40
    assert K.kvc_attention_workspace(n_q, hq, hkv, 128) > 0
    q = oracle.f64_to_bf16(1.0 + 0.05 * rng.standard_normal((n_q, hq, 128)))
    kk = 0.05 * rng.standard_normal((n_kv, hkv, 128))
    kk[100:400] += 3.0
    kk[4000:4100] += 2.0
    k = oracle.f64_to_bf16(kk)
    v = oracle.f64_to_bf16(rng.standard_normal((n_kv, hkv, 128)))
    pos = np.sort(rng.choice(np.arange(4500, n_kv), n_q, replace=False))
    # and one query that sees only the first 2601 keys: the later splits
    # see none of its keys and must contribute nothing
    pos[0] = 2600
    got, lse = _attn_gpu(K, q, pos, k, v, hq, hkv, split=True)
    want, wl = oracle.sparse_query_attention(q, pos, k, v, hq, hkv)
    ok, err = within_tol(got, want)
    assert ok, err
    assert np.allclose(lse, wl, rtol=0, atol=LSE_ATOL)
    # the same with the large logits at the end of the key range instead
    k2 = oracle.f64_to_bf16(kk[::-1].copy())
    got2, lse2 = _attn_gpu(K, q, pos, k2, v, hq, hkv, split=True)
    want2, wl2 = oracle.sparse_query_attention(q, pos, k2, v, hq, hkv)
    ok, err = within_tol(got2, want2)
    assert ok, err
    assert np.allclose(lse2, wl2, rtol=0, atol=LSE_ATOL)



@pytest.mark.parametrize("hq,hkv,n_q,n_kv", [(32, 8, 150, 3000), (8, 2, 40, 5000), (4, 4, 300, 2100)])
def test_attention_split_key_range(K, hq, hkv, n_q, n_kv):
    # a selection too small to fill the GPU, given the optional workspace,
    # splits every query block's key tiles over several workgroups and merges
    # the partials; the result matches the oracle and the unsplit kernel
    assert K.kvc_attention_workspace(n_q, hq, hkv, 128) > 0
    rng = np.random.default_rng(n_q + n_kv)
    pos = np.sort(rng.choice(n_kv, n_q, replace=False))
    pos[0] = 0                                       # one query sees a single key
    q, k, v = _qkv(rng, n_q, n_kv, hq, hkv)
    got, lse = _attn_gpu(K, q, pos, k, v, hq, hkv, split=True)
    want, wl = oracle.sparse_query_attention(q, pos, k, v, hq, hkv)
    ok, err = within_tol(got, want)
    assert ok, err
    assert np.allclose(lse, wl, rtol=0, atol=LSE_ATOL)
    one, lse1 = _attn_gpu(K, q, pos, k, v, hq, hkv)
    assert np.max(np.abs(got - one)) <= 2 * 2.0 ** -8 * (np.max(np.abs(one)) + 1e-3)
    assert np.array_equal(got[0], np.repeat(oracle.bf16_to_f64(v[0]), hq // hkv, axis=0))


def test_attention_split_masks_future_keys_and_invalid_queries(K):
    rng = np.random.default_rng(16)
    n_kv, hq, hkv = 4000, 8, 2
    q, k, v = _qkv(rng, 60, n_kv, hq, hkv)
    pos = np.sort(rng.choice(n_kv, 60, replace=False))
    pos[7] = -1                                      # no visible key
    got, lse = _attn_gpu(K, q, pos, k, v, hq, hkv, split=True)
    k2, v2 = k.copy(), v.copy()
    cut = pos[30] + 1
    k2[cut:] = oracle.f64_to_bf16(oracle.bf16_to_f64(k[cut:]) * 3 + 1)
    v2[cut:] = oracle.f64_to_bf16(oracle.bf16_to_f64(v[cut:]) - 5)
    got2, _ = _attn_gpu(K, q, pos, k2, v2, hq, hkv, split=True)
    assert np.array_equal(got[:31], got2[:31])
    assert np.all(got[7] == 0) and np.all(np.isneginf(lse[7]))
    pp = pos.copy()
    want, wl = oracle.sparse_query_attention(q, pp, k, v, hq, hkv)
    fin = np.isfinite(wl)
    ok, err = within_tol(got, want)
    assert ok, err
    assert np.allclose(lse[fin], wl[fin], rtol=0, atol=LSE_ATOL)


def test_largest_head_count(K):
    # 64 kv heads (the largest the library takes; 16 KB rows) with 64 query
    # heads: shift, deviation and attention, unsplit and split
    rng = np.random.default_rng(31)
    hq = hkv = 64
    cl = [70, 130]
    n_r = sum(cl)
    k_src = oracle.f64_to_bf16(rng.standard_normal((n_r, hkv, 128)))
    L = K.Layout(cl, 0, hq, hkv, 128, 500000.0)
    plan = _plan(K, L)
    out = up(np.zeros_like(k_src))
    K.kvc_rope_shift(L, plan, up(k_src), out)
    want = oracle.rope_shift(k_src, cl, oracle.inv_freq(128, 500000.0))
    assert _same_values(down_bf16(out), oracle.f64_to_bf16(want))
    kf = oracle.f64_to_bf16(rng.standard_normal((n_r, hkv, 128)))
    assert np.array_equal(_dev_gpu(K, k_src, kf), oracle.key_deviation(k_src, kf))
    # 2,500 keys: 40 tiles, so the split run really splits (up to 5 ranges)
    n_q, n_kv = 40, 2500
    q, k, v = _qkv(rng, n_q, n_kv, hq, hkv)
    pos = np.sort(rng.choice(n_kv, n_q, replace=False))
    pos[-1] = n_kv - 1
    want, wl = oracle.sparse_query_attention(q, pos, k, v, hq, hkv)
    for split in (False, True):
        got, lse = _attn_gpu(K, q, pos, k, v, hq, hkv, split=split)
        ok, err = within_tol(got, want)
        assert ok, (split, err)
        assert np.allclose(lse, wl, rtol=0, atol=LSE_ATOL)
