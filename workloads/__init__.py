"""Seeded synthetic workloads for the selective-recompute prefill.

This module only draws random numbers and fixes shapes.  It holds none of
the method's arithmetic (no rotation, no deviation, no selection, no
attention): both the CPU oracle (via ``tests/``) and the GPU benchmark
consume what it returns and build their own inputs from it.

Shapes follow the Llama-3.1-8B attention layout used by the paper's
experiments (Section 4: 32 query heads, 8 key/value heads, head size 128,
RoPE base 500000) at the context lengths of its TTFT study (Section 4.3).
Value distributions are a stand-in for real per-chunk KV caches, which are
not available: per-channel scales drawn from lognormal(0, 0.5), Gaussian
entries, and a recomputed ("fresh") key/value that differs from the cached
one by N(0, 0.1) noise, which plays the part of the missing
cross-attention between chunks (Section 1, Section 3.2).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

__all__ = ["Workload", "CONFIGS", "get", "draw_raw", "f32_to_bf16_bits", "documents"]


@dataclass(frozen=True)
class Workload:
    """Shape of one prefill request: reused chunks followed by a query chunk."""

    name: str
    chunk_len: tuple
    n_query: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int = 128
    rope_theta: float = 500000.0
    ratio: float = 0.15
    noise: float = 0.1
    # chunks whose first tokens get a larger deviation (attention-sink-like)
    structured: bool = False
    chunk_old_pos0: tuple | None = None
    # reused chunks whose cached K/V are all zero: the two special tokens
    # between documents, whose cache entries the paper sets to zero
    # (Section 3.1; implementation notes of Section 4)
    zero_kv_chunks: tuple = ()
    extra: dict = field(default_factory=dict)

    @property
    def n_reused(self) -> int:
        return int(sum(self.chunk_len))

    @property
    def n_rows(self) -> int:
        return self.n_reused + int(self.n_query)

    @property
    def zero_kv_flags(self) -> list:
        """One flag per reused chunk: True where the cached K/V are zero."""
        z = set(self.zero_kv_chunks)
        return [i in z for i in range(len(self.chunk_len))]

    @property
    def zero_rows(self) -> np.ndarray:
        """Row indices of the zero-K/V chunks (int64, ascending)."""
        row0 = np.concatenate([[0], np.cumsum(self.chunk_len)[:-1]]).astype(np.int64)
        parts = [np.arange(row0[i], row0[i] + self.chunk_len[i], dtype=np.int64) for i in self.zero_kv_chunks]
        return np.concatenate(parts) if parts else np.zeros(0, dtype=np.int64)

    def with_(self, **kw) -> "Workload":
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)


def documents(name: str, n_reused: int, mean_len: float, n_query: int, n_q_heads: int, n_kv_heads: int,
              max_len: int = 512, min_len: int = 16, sep: int = 2, seed: int = 0) -> Workload:
    """A retrieval-style context of exactly ``n_reused`` reused rows:
    documents of mixed length, each one its own precomputed chunk, with a
    sep-token separator slot of zero K/V before every document and after
    the last one: [sep][doc 0][sep][doc 1] ... [doc n-1][sep], then the
    query chunk.

    Document lengths are lognormal with mean ``mean_len`` (sigma 0.6),
    clipped to [min_len, max_len]; the last document takes what is left.
    The paper's non-QA contexts use documents of at most 512 tokens and its
    QA contexts the benchmark's own passages, which at 124k tokens makes
    over 200 and over 700 chunks (Section 4.2).
    """
    rng = np.random.default_rng([int(seed), 99])
    mu = np.log(mean_len) - 0.5 * 0.6 ** 2
    chunk_len, zero, used = [], [], 0
    while True:
        left = n_reused - used - 2 * sep       # room for this document and the closing separator
        if left < min_len:
            break
        n = int(np.clip(np.rint(rng.lognormal(mu, 0.6)), min_len, max_len))
        if left - n < min_len + sep:           # too little would remain for another document
            n = left
        zero.append(len(chunk_len))
        chunk_len += [sep, n]
        used += sep + n
    zero.append(len(chunk_len))
    chunk_len.append(n_reused - used)          # the closing separator (sep rows)
    assert chunk_len[-1] == sep and sum(chunk_len) == n_reused
    return Workload(name, tuple(chunk_len), n_query, n_q_heads, n_kv_heads, zero_kv_chunks=tuple(zero))


CONFIGS = {
    # 4 chunks x 256 tokens + 64-token query chunk, 8 q heads / 2 kv heads
    "tiny": Workload("tiny", (256,) * 4, 64, 8, 2),
    # 16 chunks x 250 tokens + 96-token query (~4.1k context)
    "4k": Workload("4k", (250,) * 16, 96, 32, 8),
    # 16 chunks x 2,000 tokens + 256-token query (32,256 rows)
    "32k": Workload("32k", (2000,) * 16, 256, 32, 8),
    # 16 chunks x 7,750 tokens + 256-token query (124,256 rows)
    "124k": Workload("124k", (7750,) * 16, 256, 32, 8),
    # one GPU's share of the 124k layer split 8 ways by kv head (tensor
    # parallel, Llama's layout): 1 kv head and its 4 query heads
    "124k-tp8": Workload("124k-tp8", (7750,) * 16, 256, 4, 1),
    # document layouts with two-token zero-K/V separators
    "sep-tiny": documents("sep-tiny", 480, 40.0, 32, 8, 2, max_len=96),
    "sep-4k": documents("sep-4k", 4000, 170.0, 96, 32, 8),
    "qa-32k": documents("qa-32k", 32000, 175.0, 256, 32, 8),
    # 124,000 reused rows of short QA-like passages (~700 documents)
    "qa-124k": documents("qa-124k", 124000, 170.0, 256, 32, 8),
    # 124,000 reused rows of documents of up to 512 tokens (~250 documents)
    "docs-124k": documents("docs-124k", 124000, 480.0, 256, 32, 8),
}


def get(name: str) -> Workload:
    return CONFIGS[name]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); uint16 bits.

    Input preparation only (the generator's own data-type conversion).
    Values are finite by construction.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def _rng(seed: int, layer: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(layer), int(stream)])


def draw_raw(w: Workload, seed: int = 0, layer: int = 0, q_rows=None,
             parts=("k", "v", "q")) -> dict:
    """Draw the raw float32 tensors of one layer of one request.

    Returns a dict of float32 arrays (no positional encoding applied):

    * ``k_raw``  [N, Hkv, D] pre-RoPE key of every token (cached side)
    * ``k_noise`` [N, Hkv, D] recomputed key = k_raw + k_noise
    * ``v``      [N, Hkv, D] cached value
    * ``v_noise`` [N, Hkv, D] recomputed value = v + v_noise
    * ``q_raw``  [N, Hq, D] (or only the rows in ``q_rows``) pre-RoPE query

    Each tensor comes from its own counter-keyed stream, so drawing a subset
    of query rows gives the same values as drawing all of them, and ``parts``
    (a subset of "k", "v", "q") skips the tensors not needed.
    """
    N, Hq, Hkv, D = w.n_rows, w.n_q_heads, w.n_kv_heads, w.head_dim
    g = _rng(seed, layer, 0)
    s_k = g.lognormal(0.0, 0.5, size=(Hkv, D)).astype(np.float32)
    s_v = g.lognormal(0.0, 0.5, size=(Hkv, D)).astype(np.float32)
    s_q = g.lognormal(0.0, 0.5, size=(Hq, D)).astype(np.float32)

    out = {}
    if "k" in parts:
        k_raw = _rng(seed, layer, 1).standard_normal((N, Hkv, D), dtype=np.float32) * s_k
        k_noise = _rng(seed, layer, 2).standard_normal((N, Hkv, D), dtype=np.float32)
        k_noise *= np.float32(w.noise)
        out.update(k_raw=k_raw, k_noise=k_noise)
    if "v" in parts:
        v = _rng(seed, layer, 3).standard_normal((N, Hkv, D), dtype=np.float32) * s_v
        v_noise = _rng(seed, layer, 4).standard_normal((N, Hkv, D), dtype=np.float32)
        v_noise *= np.float32(w.noise)
        out.update(v=v, v_noise=v_noise)
    if w.structured:
        # first 4 tokens of each reused chunk deviate 4x more
        row0 = np.concatenate([[0], np.cumsum(w.chunk_len)[:-1]])
        for r in row0:
            for key in ("k_noise", "v_noise"):
                if key in out:
                    out[key][r:r + 4] *= np.float32(4.0)
    if "q" not in parts:
        return out

    # queries are drawn in fixed blocks of 256 rows, each from its own
    # stream, so any subset of rows can be drawn without the rest
    rows = np.arange(N, dtype=np.int64) if q_rows is None else np.asarray(q_rows, dtype=np.int64)
    q_raw = np.empty((len(rows), Hq, D), dtype=np.float32)
    blk_of = rows // 256
    for b in np.unique(blk_of):
        gb = np.random.default_rng([int(seed), int(layer), 5, int(b)])
        blk = gb.standard_normal((256, Hq, D), dtype=np.float32) * s_q
        idx = np.nonzero(blk_of == b)[0]
        q_raw[idx] = blk[rows[idx] - b * 256]
    out["q_raw"] = q_raw
    return out
