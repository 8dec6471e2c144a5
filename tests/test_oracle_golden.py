"""The oracle reproduces its stored regression fixture (tests/golden)."""
import json
import os

import numpy as np

import oracle
import workloads as W
from _inputs import build

HERE = os.path.dirname(os.path.abspath(__file__))


def test_tiny_seed0_fixture():
    with open(os.path.join(HERE, "golden", "tiny_seed0.json")) as fh:
        fix = json.load(fh)
    w = W.get("tiny")
    x = build(w, seed=0)
    r = oracle.blend_prefill_layer(w.chunk_len, w.n_query, w.n_q_heads, w.n_kv_heads,
                                   w.rope_theta, x["k_src"], x["v_cache"], x["q"],
                                   x["k_fresh"], x["v_fresh"], True, w.ratio)
    assert [int(i) for i in r["sel"]] == fix["sel"]
    assert len(fix["sel"]) == 153 + 64
    assert np.sort(r["dev"])[::-1][:5].tolist() == fix["dev_top5"]
    assert np.allclose(r["out"][0, 0, :8], fix["out_row0_head0_first8"], rtol=1e-12, atol=0)
    assert np.allclose(r["lse"][0], fix["lse_row0"], rtol=1e-12, atol=0)
