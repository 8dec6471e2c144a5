"""Decoder-layer steps around the attention of the selected tokens (test
infrastructure only).

The paper's base models (Section 4.1: Llama-3.1-8B-Instruct, and
Qwen2.5-7B-Instruct) are decoder-only transformers with pre-norm layers: an
RMS normalisation, a projection to queries, keys and values, RoPE on the
queries and keys at each token's position, attention, an output projection
added to the residual stream, a second RMS normalisation and a gated SiLU
feed-forward block added to the residual stream.  With selective recompute
only the selected tokens and the query chunk pass through a layer; every
other token keeps its cached K/V (Section 3.4; Section 4 setup), so these
steps run on the selected rows only.

The steps follow the published definitions the models use: RMSNorm (Zhang
and Sennrich, 2019), the SwiGLU feed-forward block (Shazeer, 2020) and RoPE
in the half-split form (Su et al.; see ``rope``).  Readings fixed here:

* RMS normalisation: y = x / sqrt(mean(x^2) + eps) * gamma, exact and
  rounded once (the models' library code rounds x / rms to bfloat16 before
  the product with gamma);
* the fused projection's output row is [Q heads | K heads | V heads], each
  head D wide; Q and K pairs (x[j], x[j + D/2]) are rotated by pos * f_j at
  the token's absolute position; V is passed through;
* the feed-forward input row is [gate (I) | up (I)]; the activation is
  silu(gate) * up with silu(g) = g / (1 + exp(-g));
* every tensor stored between two steps is bfloat16, rounded to nearest
  even (``decoder_layer`` with ``round_bf16=True``); matrix products
  (``projection``) accumulate in float64 and round once, after the residual
  addition where there is one.
"""
import numpy as np

from .bf16 import bf16_to_f64, f64_to_bf16
from .rope import rope_rotate
from .attention import sparse_query_attention


def _f64(x):
    x = np.asarray(x)
    return bf16_to_f64(x) if x.dtype == np.uint16 else x.astype(np.float64)


def rms_norm(x, gamma, eps: float) -> np.ndarray:
    """Row-wise RMS normalisation: x / sqrt(mean(x^2) + eps) * gamma.

    x: [rows, hidden], gamma: [hidden]; bfloat16 bits or floats.
    Returns float64 [rows, hidden].
    """
    x = _f64(x)
    g = _f64(gamma)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + float(eps)) * g[None, :]


def qkv_rope(y, pos, n_q_heads: int, n_k_heads: int, n_v_heads: int, freqs,
             head_dim: int = 128):
    """Split fused projection rows into Q, K, V; rotate Q and K at ``pos``.

    y: [rows, (n_q + n_k + n_v) * D]; pos: [rows] absolute positions.
    Returns float64 (q [rows, n_q, D], k [rows, n_k, D], v [rows, n_v, D]).
    """
    y = _f64(y)
    n = y.shape[0]
    D = int(head_dim)
    assert y.shape[1] == (n_q_heads + n_k_heads + n_v_heads) * D
    heads = y.reshape(n, n_q_heads + n_k_heads + n_v_heads, D)
    q = heads[:, :n_q_heads]
    k = heads[:, n_q_heads:n_q_heads + n_k_heads]
    v = heads[:, n_q_heads + n_k_heads:]
    pos = np.asarray(pos, dtype=np.int64)
    return rope_rotate(q, pos, freqs), rope_rotate(k, pos, freqs), v.copy()


def swiglu(gu, inter: int) -> np.ndarray:
    """Gated SiLU of the feed-forward block: silu(gate) * up.

    gu: [rows, 2 * inter] with the gate in the first half of each row.
    Returns float64 [rows, inter].
    """
    gu = _f64(gu)
    assert gu.shape[1] == 2 * int(inter)
    g, u = gu[:, :inter], gu[:, inter:]
    # g / (1 + e^-g) written without overflow: for g < 0, g e^g / (1 + e^g)
    e = np.exp(-np.abs(g))
    silu = np.where(g >= 0, g / (1.0 + e), g * e / (1.0 + e))
    return silu * u


def projection(a, w, rows=None, residual=None) -> np.ndarray:
    """One linear map of the layer on the selected rows:
        c = a[rows] w^T  (+ residual)
    Only the selected tokens pass through a layer under selective recompute
    (Section 3.4; Section 4 setup), so each of its projections (fused Q/K/V,
    O, gate/up, down) multiplies the selected rows by a weight matrix.

    a: [n_a, k]; w: [n, k], the [out, in] layout of a linear layer; rows:
    [m] indices into a, or None for all rows (an index outside [0, n_a)
    stands for a zero row); residual: [m, n] or None.  bfloat16 bits or
    floats.  The products of bfloat16 values are exact in float64 and are
    summed in float64.  Returns float64 [m, n].
    """
    a = _f64(a)
    w = _f64(w)
    if rows is not None:
        rows = np.asarray(rows, dtype=np.int64)
        ok = (rows >= 0) & (rows < a.shape[0])
        a = np.where(ok[:, None], a[np.where(ok, rows, 0)], 0.0)
    c = a @ w.T
    if residual is not None:
        c = c + _f64(residual)
    return c


def decoder_layer(h, pos, k_cache, v_cache, w, n_q_heads: int, n_kv_heads: int,
                  freqs, eps: float = 1e-5, round_bf16: bool = True):
    """One pre-norm decoder layer for the selected rows ``h``.

    h: [n, hidden] residual-stream rows of the tokens at positions ``pos``
    (ascending); k_cache, v_cache: [N, Hkv, D] blended cache whose rows at
    ``pos`` are replaced by the rows' fresh K/V before the attention (the
    other rows are the reused cache).  w: dict of weights with
    y = x @ W conventions: ``norm1``/``norm2`` [hidden], ``qkv``
    [hidden, (Hq + 2 Hkv) D], ``o`` [Hq D, hidden], ``gate_up``
    [hidden, 2 I], ``down`` [I, hidden].  With every row selected
    (pos = 0..N-1) this is the full causal layer.

    Returns a dict of the intermediates (x, q, k, v, attn, h_mid, x2, gu,
    act) and the layer output ``out`` [n, hidden], all float64 (holding
    bfloat16 values when round_bf16), plus the blended ``k_cache`` and
    ``v_cache``.
    """
    rnd = (lambda t: bf16_to_f64(f64_to_bf16(t))) if round_bf16 else (lambda t: t)
    W = {name: _f64(t) for name, t in w.items()}
    h = _f64(h)
    pos = np.asarray(pos, dtype=np.int64)
    n = h.shape[0]
    D = _f64(k_cache).shape[-1]
    inter = W["down"].shape[0]

    x = rnd(rms_norm(h, W["norm1"], eps))
    y = rnd(projection(x, W["qkv"].T))
    q, k, v = qkv_rope(y, pos, n_q_heads, n_kv_heads, n_kv_heads, freqs, D)
    q, k, v = rnd(q), rnd(k), rnd(v)
    kc = np.array(_f64(k_cache), copy=True)
    vc = np.array(_f64(v_cache), copy=True)
    kc[pos] = k
    vc[pos] = v
    attn, _ = sparse_query_attention(q, pos, kc, vc, n_q_heads, n_kv_heads)
    attn = rnd(attn)
    h_mid = rnd(projection(attn.reshape(n, n_q_heads * D), W["o"].T, residual=h))
    x2 = rnd(rms_norm(h_mid, W["norm2"], eps))
    gu = rnd(projection(x2, W["gate_up"].T))
    act = rnd(swiglu(gu, inter))
    out = rnd(projection(act, W["down"].T, residual=h_mid))
    return dict(x=x, q=q, k=k, v=v, attn=attn, h_mid=h_mid, x2=x2, gu=gu, act=act,
                out=out, k_cache=kc, v_cache=vc)
