"""CPU oracle for the selective-recompute prefill -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 numpy implementation of what the GPU path computes,
written from the paper ("Fine-Tuning a KV Cache Concatenation-Aware Model
or Recomputing KV Caches? Why Not Both?", arXiv 2609.09768).  It exists to
check the HIP library; only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it.  The product path never
calls it, and it shares no code with the HIP kernels or the C ABI.

Modules (each function cites the passage it follows):

* ``bf16``      -- bfloat16 bit patterns <-> float64 (exact / round-to-nearest-even)
* ``rope``      -- RoPE rotation and the per-chunk position adjustment (A1)
* ``deviation`` -- per-token squared key deviation, exactly rounded (A2)
* ``select``    -- recompute count and top-k token selection (A3)
* ``attention`` -- causal GQA attention of sparse queries (A5)
* ``blend``     -- one layer of the selective-recompute prefill (A4 + A6)
* ``layer``     -- the decoder-layer steps around the attention for the
                   selected tokens: RMS normalisation, Q/K/V split with RoPE,
                   gated SiLU, the projections, and the whole layer composed

Every function here is pinned by ``tests/test_oracle_*.py`` against closed
forms, invariants, brute force or independent library routines.
"""
from . import bf16, rope, deviation, select, attention, blend, layer  # noqa: F401
from .bf16 import bf16_to_f64, f64_to_bf16
from .rope import inv_freq, rope_rotate, chunk_row0, chunk_delta, rope_shift
from .deviation import key_deviation
from .select import recompute_count, select_topk, selection
from .attention import sparse_query_attention, causal_attention
from .blend import blend_prefill_layer
from .layer import rms_norm, qkv_rope, swiglu, projection, decoder_layer

__all__ = [
    "bf16_to_f64", "f64_to_bf16", "inv_freq", "rope_rotate", "chunk_row0",
    "chunk_delta", "rope_shift", "key_deviation", "recompute_count",
    "select_topk", "selection", "sparse_query_attention", "causal_attention",
    "blend_prefill_layer", "rms_norm", "qkv_rope", "swiglu", "projection", "decoder_layer",
]
