"""The C ABI from a plain C program, without Python or torch in between.

tests/c_abi/kvc_c_demo.c allocates device memory and a stream with the HIP
runtime, uploads a plan and runs one check layer with
kvc_blend_prefill_layer; this test writes its seeded input file, runs it as
a child process and compares its output file with the oracle: selection,
adjusted and blended caches bit for bit, attention to the bf16 tolerance.
A bad ratio must come back as the library's error, through kvc_last_error.
"""
import struct
import subprocess

import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import within_tol, LSE_ATOL
from _inputs import build

pytestmark = pytest.mark.gpu


def _write_input(path, w, x, ratio):
    with open(path, "wb") as f:
        f.write(struct.pack("<i", len(w.chunk_len)))
        f.write(np.asarray(w.chunk_len, dtype="<i4").tobytes())
        f.write(struct.pack("<qiidd", w.n_query, w.n_q_heads, w.n_kv_heads, w.rope_theta, ratio))
        for name in ("k_src", "v_cache", "k_fresh", "v_fresh", "q"):
            f.write(np.ascontiguousarray(x[name]).astype("<u2").tobytes())


@pytest.mark.parametrize("name", ["tiny", "4k"])
def test_check_layer_from_c(c_demo, tmp_path, name):
    w = W.get(name)
    x = build(w, seed=4)
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    _write_input(src, w, x, w.ratio)
    r = subprocess.run([c_demo, str(src), str(dst)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    N, H, Hk = w.n_rows, w.n_q_heads, w.n_kv_heads
    n_sel = oracle.recompute_count(w.ratio, w.n_reused) + w.n_query
    raw = np.fromfile(dst, dtype=np.uint8)
    parts, off = {}, 0
    for key, dt, count in (("sel", "<i4", n_sel), ("out", "<u2", n_sel * H * 128), ("lse", "<f4", n_sel * H),
                           ("k_cache", "<u2", N * Hk * 128), ("v_cache", "<u2", N * Hk * 128)):
        nb = np.dtype(dt).itemsize * count
        parts[key] = raw[off:off + nb].view(dt)
        off += nb
    assert off == raw.size
    rows = np.unique(np.concatenate([np.arange(min(8, n_sel)), np.arange(max(n_sel - 8, 0), n_sel),
                                     np.random.default_rng(0).choice(n_sel, min(24, n_sel), replace=False)]))
    want = oracle.blend_prefill_layer(w.chunk_len, w.n_query, H, Hk, w.rope_theta, x["k_src"], x["v_cache"],
                                      x["q"], x["k_fresh"], x["v_fresh"], True, w.ratio, attn_rows=rows)
    assert np.array_equal(parts["sel"].astype(np.int64), want["sel"])
    kc = parts["k_cache"].reshape(N, Hk, 128)
    assert np.array_equal(oracle.bf16_to_f64(kc), oracle.bf16_to_f64(want["k_cache"]))
    assert np.array_equal(parts["v_cache"].reshape(N, Hk, 128), want["v_cache"])
    got = oracle.bf16_to_f64(parts["out"].reshape(n_sel, H, 128)[rows])
    ok, err = within_tol(got, want["out"])
    assert ok, err
    assert np.allclose(parts["lse"].reshape(n_sel, H)[rows], want["lse"], rtol=0, atol=LSE_ATOL)


def test_error_from_c(c_demo, tmp_path):
    w = W.get("tiny")
    x = build(w, seed=4)
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    _write_input(src, w, x, 1.5)
    r = subprocess.run([c_demo, str(src), str(dst)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 2, (r.returncode, r.stderr)
    assert "kvc_blend_prefill_layer" in r.stderr and "ratio" in r.stderr
