"""Writes the oracle regression fixtures in this folder.

Calls only ``oracle/`` (and the seeded raw draws of ``workloads``):
    python tests/golden/make_golden.py
The paper prints no worked numerical example of the computation, so these
fixtures pin the oracle against its own earlier, reviewed output; the
paper-facing pins live in tests/test_oracle_*.py.
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
sys.path.insert(0, os.path.dirname(HERE))

import workloads as W          # noqa: E402
import oracle                  # noqa: E402
from _inputs import build      # noqa: E402


def main():
    w = W.get("tiny")
    x = build(w, seed=0)
    r = oracle.blend_prefill_layer(w.chunk_len, w.n_query, w.n_q_heads, w.n_kv_heads,
                                   w.rope_theta, x["k_src"], x["v_cache"], x["q"],
                                   x["k_fresh"], x["v_fresh"], True, w.ratio)
    fix = {
        "what": "Tiny workload (4 x 256 reused + 64 query rows, 8/2 heads, D 128, "
                "theta 500000, ratio 0.15, seed 0), check layer, from the oracle",
        "sel": [int(i) for i in r["sel"]],
        "dev_top5": [float(v) for v in np.sort(r["dev"])[::-1][:5]],
        "out_row0_head0_first8": [float(v) for v in r["out"][0, 0, :8]],
        "lse_row0": [float(v) for v in r["lse"][0]],
        "k_shift_sum": float(oracle.bf16_to_f64(r["k_shift"]).sum()),
    }
    with open(os.path.join(HERE, "tiny_seed0.json"), "w") as fh:
        json.dump(fix, fh, indent=1)


if __name__ == "__main__":
    main()
