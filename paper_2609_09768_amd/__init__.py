"""Python binding of libkvc, the MI355X selective-recompute prefill library.

Argument marshalling only: every function here forwards to the C entry
point of the same name declared in ``include/kvc.h`` (ctypes), and every
step of the computation runs in the library's HIP kernels.  Pointer
arguments accept a torch tensor (its ``data_ptr()``), an integer address or
None (NULL); ``stream`` accepts a ``torch.cuda.Stream``, a raw hipStream_t
integer, or None for torch's current stream.  A non-OK status raises
``KvcError`` carrying the library's message.

The library must have been built (``python paper_2609_09768_amd/build_lib.py``);
importing this package without it raises, there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvc.so")

KVC_OK, KVC_ERR_INVALID_ARG, KVC_ERR_UNSUPPORTED, KVC_ERR_WORKSPACE, KVC_ERR_DEVICE = range(5)
_STATUS_NAMES = {0: "KVC_OK", 1: "KVC_ERR_INVALID_ARG", 2: "KVC_ERR_UNSUPPORTED",
                 3: "KVC_ERR_WORKSPACE", 4: "KVC_ERR_DEVICE"}


class KvcError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing; build it with "
                      "`python paper_2609_09768_amd/build_lib.py` (hipcc, gfx950)")

_lib = ctypes.CDLL(LIB_PATH)

_vp, _i32, _i64, _f32, _f64, _sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                    ctypes.c_float, ctypes.c_double, ctypes.c_size_t)


class kvc_layout(ctypes.Structure):
    _fields_ = [("n_chunks", _i32), ("chunk_len", ctypes.POINTER(_i32)),
                ("chunk_old_pos0", ctypes.POINTER(_i64)), ("n_query", _i64),
                ("n_q_heads", _i32), ("n_kv_heads", _i32), ("head_dim", _i32),
                ("rope_theta", _f64), ("inv_freq", ctypes.POINTER(_f64)),
                ("zero_kv", ctypes.POINTER(ctypes.c_uint8))]


class kvc_plan(ctypes.Structure):
    _fields_ = [("device", _vp), ("bytes", _sz), ("layout_id", ctypes.c_uint64)]


_LP = ctypes.POINTER(kvc_layout)
_PLP = ctypes.POINTER(kvc_plan)
_PP = ctypes.POINTER(_vp)
_SIGS = {
    "kvc_abi_version": (_i32, []),
    "kvc_last_error": (ctypes.c_char_p, []),
    "kvc_recompute_count": (_i64, [_f64, _i64]),
    "kvc_layout_id": (_i32, [_LP, ctypes.POINTER(ctypes.c_uint64)]),
    "kvc_plan_bytes": (_i32, [_LP, ctypes.POINTER(_sz)]),
    "kvc_plan_upload": (_i32, [_LP, _vp, _sz, _vp, _PLP, _vp]),
    "kvc_rope_shift": (_i32, [_LP, _PLP, _vp, _vp, _vp]),
    "kvc_kv_deviation": (_i32, [_i64, _i32, _i32, _vp, _vp, _vp, _vp]),
    "kvc_select_topk_workspace": (_i32, [_i64, ctypes.POINTER(_sz)]),
    "kvc_select_topk": (_i32, [_vp, _i64, _i64, _vp, _vp, _sz, _vp]),
    "kvc_scatter_rows": (_i32, [_vp, _i64, _i32, _vp, _vp, _i64, _vp, _vp, _i64, _i32, _i32, _vp]),
    "kvc_attention_workspace": (_i32, [_i64, _i32, _i32, _i32, ctypes.POINTER(_sz)]),
    "kvc_sparse_query_attention": (_i32, [_vp, _i64, _vp, _vp, _i64, _vp, _vp, _i64, _i32, _i32,
                                          _i32, _f32, _vp, _vp, _vp, _sz, _vp]),
    "kvc_blend_workspace": (_i32, [_LP, ctypes.POINTER(_sz)]),
    "kvc_blend_prefill_layer": (_i32, [_LP, _PLP, _i32, _f64, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                       _i64, _vp, _vp, _vp, _sz, _vp]),
    "kvc_blend_prefill_layer_noalloc": (_i32, [_LP, _PLP, _i32, _f64, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                               _i64, _vp, _vp, _vp]),
    "kvc_select_tokens": (_i32, [_LP, _PLP, _f64, _vp, _vp, _vp, _vp, _i64, _vp, _sz, _vp]),
    "kvc_rms_norm": (_i32, [_vp, _i64, _vp, _i64, _i32, _vp, _f32, _vp, _vp, _vp]),
    "kvc_qkv_rope": (_i32, [_vp, _i64, _i32, _i32, _i32, _i32, _vp, _f64, ctypes.POINTER(_f64), _vp,
                            _vp, _vp, _vp]),
    "kvc_swiglu": (_i32, [_vp, _i64, _i64, _vp, _vp]),
    "kvc_projection": (_i32, [_i64, _i64, _i64, _vp, _i64, _vp, _vp, _vp, _vp, _vp]),
    "kvc_stage_layer": (_i32, [_LP, _PLP, _PP, _PP, _vp, _vp, _vp]),
    "kvc_stage_layers": (_i32, [_LP, _PLP, _i32, _PP, _PP, _PP, _PP, _PP, _vp]),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def _ptr(x):
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    return int(x)


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if hasattr(s, "cuda_stream"):
        return s.cuda_stream
    return int(s)


def _check(st: int):
    if st != KVC_OK:
        raise KvcError(st, _lib.kvc_last_error().decode())


class Layout:
    """Owns the host arrays behind a ``kvc_layout`` (see include/kvc.h)."""

    def __init__(self, chunk_len, n_query, n_q_heads, n_kv_heads, head_dim=128,
                 rope_theta=500000.0, chunk_old_pos0=None, inv_freq=None, zero_kv=None):
        cl = [int(x) for x in chunk_len]
        self.chunk_len = list(cl)
        self.n_query = int(n_query)
        self.n_q_heads, self.n_kv_heads, self.head_dim = int(n_q_heads), int(n_kv_heads), int(head_dim)
        self._cl = (_i32 * max(len(cl), 1))(*cl)
        self._old = None if chunk_old_pos0 is None else (_i64 * len(cl))(*[int(x) for x in chunk_old_pos0])
        self._inv = None if inv_freq is None else (_f64 * len(inv_freq))(*[float(x) for x in inv_freq])
        # zero_kv: one flag per chunk (true: cached K/V all zero)
        self._zero = None
        if zero_kv is not None:
            flags = [int(bool(v)) for v in zero_kv]
            if len(flags) != len(cl):
                raise ValueError(f"zero_kv has {len(flags)} flags for {len(cl)} chunks")
            self._zero = (ctypes.c_uint8 * max(len(cl), 1))(*flags)
        self.struct = kvc_layout(
            len(cl), ctypes.cast(self._cl, ctypes.POINTER(_i32)),
            None if self._old is None else ctypes.cast(self._old, ctypes.POINTER(_i64)),
            self.n_query, self.n_q_heads, self.n_kv_heads, self.head_dim, float(rope_theta),
            None if self._inv is None else ctypes.cast(self._inv, ctypes.POINTER(_f64)),
            None if self._zero is None else ctypes.cast(self._zero, ctypes.POINTER(ctypes.c_uint8)))

    @property
    def n_reused(self) -> int:
        return sum(self.chunk_len)

    @property
    def n_rows(self) -> int:
        return self.n_reused + self.n_query

    def ref(self):
        return ctypes.byref(self.struct)


def _lref(layout):
    return None if layout is None else layout.ref()


class Plan:
    """A ``kvc_plan`` descriptor (see include/kvc.h) plus references to the
    device buffer (and host staging memory) it describes, which stay alive
    as long as the descriptor.  ``kvc_plan_upload`` returns one; tests may
    also build one from raw values."""

    def __init__(self, device, nbytes, layout_id, keep=()):
        self.struct = kvc_plan(_ptr(device), int(nbytes), int(layout_id))
        self._keep = (device,) + tuple(keep)

    @property
    def layout_id(self) -> int:
        return int(self.struct.layout_id)

    def ref(self):
        return ctypes.byref(self.struct)


def _pref(plan):
    return None if plan is None else plan.ref()


def kvc_abi_version() -> int:
    return int(_lib.kvc_abi_version())


def kvc_last_error() -> str:
    return _lib.kvc_last_error().decode()


def kvc_recompute_count(ratio: float, n_reused: int) -> int:
    return int(_lib.kvc_recompute_count(float(ratio), int(n_reused)))


def kvc_plan_bytes(layout) -> int:
    b = _sz(0)
    _check(_lib.kvc_plan_bytes(_lref(layout), ctypes.byref(b)))
    return b.value


def kvc_layout_id(layout) -> int:
    v = ctypes.c_uint64(0)
    _check(_lib.kvc_layout_id(_lref(layout), ctypes.byref(v)))
    return int(v.value)


def kvc_plan_upload(layout, plan, plan_bytes, stream=None, staging=None) -> Plan:
    """Uploads the plan into the device buffer ``plan`` and returns its
    descriptor.  ``staging``: None (the call waits for its copy) or pinned
    host memory of at least plan_bytes bytes (a CPU tensor or an address)
    that the caller leaves unchanged until the copy has run."""
    out = kvc_plan()
    _check(_lib.kvc_plan_upload(_lref(layout), _ptr(plan), int(plan_bytes), _ptr(staging),
                                ctypes.byref(out), _stream(stream)))
    p = Plan(plan, out.bytes, out.layout_id, keep=() if staging is None else (staging,))
    p.struct.device = out.device
    return p


def kvc_rope_shift(layout, plan, k_src, k_dst, stream=None):
    _check(_lib.kvc_rope_shift(_lref(layout), _pref(plan), _ptr(k_src), _ptr(k_dst), _stream(stream)))


def kvc_kv_deviation(n_rows, n_kv_heads, head_dim, k_cached, k_fresh, dev_out, stream=None):
    _check(_lib.kvc_kv_deviation(int(n_rows), int(n_kv_heads), int(head_dim), _ptr(k_cached),
                                 _ptr(k_fresh), _ptr(dev_out), _stream(stream)))


def kvc_select_topk_workspace(n) -> int:
    b = _sz(0)
    _check(_lib.kvc_select_topk_workspace(int(n), ctypes.byref(b)))
    return b.value


def kvc_select_topk(dev, n, k, idx_out, ws, ws_bytes, stream=None):
    _check(_lib.kvc_select_topk(_ptr(dev), int(n), int(k), _ptr(idx_out), _ptr(ws), int(ws_bytes),
                                _stream(stream)))


def kvc_scatter_rows(sel, n_sel, fresh_is_compact, k_fresh, v_fresh, n_fresh_rows, k_cache, v_cache,
                     n_rows, n_kv_heads, head_dim, stream=None):
    _check(_lib.kvc_scatter_rows(_ptr(sel), int(n_sel), int(fresh_is_compact), _ptr(k_fresh),
                                 _ptr(v_fresh), int(n_fresh_rows), _ptr(k_cache), _ptr(v_cache),
                                 int(n_rows), int(n_kv_heads), int(head_dim), _stream(stream)))


def kvc_attention_workspace(n_sel, n_q_heads, n_kv_heads, head_dim) -> int:
    b = _sz(0)
    _check(_lib.kvc_attention_workspace(int(n_sel), int(n_q_heads), int(n_kv_heads), int(head_dim),
                                        ctypes.byref(b)))
    return b.value


def kvc_sparse_query_attention(q, n_q_rows, q_rows, q_pos, n_sel, k, v, n_kv, n_q_heads, n_kv_heads,
                               head_dim, softmax_scale, out, lse, ws=None, ws_bytes=0, stream=None):
    _check(_lib.kvc_sparse_query_attention(
        _ptr(q), int(n_q_rows), _ptr(q_rows), _ptr(q_pos), int(n_sel), _ptr(k), _ptr(v), int(n_kv),
        int(n_q_heads), int(n_kv_heads), int(head_dim), float(softmax_scale), _ptr(out), _ptr(lse),
        _ptr(ws), int(ws_bytes), _stream(stream)))


def kvc_blend_workspace(layout) -> int:
    b = _sz(0)
    _check(_lib.kvc_blend_workspace(_lref(layout), ctypes.byref(b)))
    return b.value


def kvc_blend_prefill_layer(layout, plan, is_check_layer, ratio, k_src, k_cache, v_cache, q_fresh,
                            k_fresh, v_fresh, sel, n_sel, out, lse, ws, ws_bytes, stream=None):
    _check(_lib.kvc_blend_prefill_layer(
        _lref(layout), _pref(plan), int(bool(is_check_layer)), float(ratio), _ptr(k_src),
        _ptr(k_cache), _ptr(v_cache), _ptr(q_fresh), _ptr(k_fresh), _ptr(v_fresh), _ptr(sel),
        int(n_sel), _ptr(out), _ptr(lse), _ptr(ws), int(ws_bytes), _stream(stream)))


def kvc_blend_prefill_layer_noalloc(layout, plan, is_check_layer, ratio, k_src, k_cache, v_cache, q_fresh,
                                    k_fresh, v_fresh, sel, n_sel, out, lse, stream=None):
    _check(_lib.kvc_blend_prefill_layer_noalloc(
        _lref(layout), _pref(plan), int(bool(is_check_layer)), float(ratio), _ptr(k_src),
        _ptr(k_cache), _ptr(v_cache), _ptr(q_fresh), _ptr(k_fresh), _ptr(v_fresh), _ptr(sel),
        int(n_sel), _ptr(out), _ptr(lse), _stream(stream)))


STATIC_SCRATCH_BYTES = 16 << 20   # KVC_STATIC_SCRATCH_BYTES in include/kvc.h


def kvc_select_tokens(layout, plan, ratio, k_src, k_cache, k_fresh, sel, n_sel, ws, ws_bytes, stream=None):
    _check(_lib.kvc_select_tokens(_lref(layout), _pref(plan), float(ratio), _ptr(k_src), _ptr(k_cache),
                                  _ptr(k_fresh), _ptr(sel), int(n_sel), _ptr(ws), int(ws_bytes),
                                  _stream(stream)))


def kvc_rms_norm(x, n_x_rows, rows, n, hidden, gamma, eps, out, res_out=None, stream=None):
    _check(_lib.kvc_rms_norm(_ptr(x), int(n_x_rows), _ptr(rows), int(n), int(hidden), _ptr(gamma),
                             float(eps), _ptr(out), _ptr(res_out), _stream(stream)))


def kvc_qkv_rope(y, n, n_q_heads, n_k_heads, n_v_heads, head_dim, pos, rope_theta, q, k, v,
                 inv_freq=None, stream=None):
    """inv_freq: None or a sequence of head_dim/2 floats (host)."""
    f = None if inv_freq is None else (_f64 * len(inv_freq))(*[float(x) for x in inv_freq])
    _check(_lib.kvc_qkv_rope(_ptr(y), int(n), int(n_q_heads), int(n_k_heads), int(n_v_heads),
                             int(head_dim), _ptr(pos), float(rope_theta),
                             None if f is None else ctypes.cast(f, ctypes.POINTER(_f64)),
                             _ptr(q), _ptr(k), _ptr(v), _stream(stream)))


def kvc_swiglu(gate_up, n, inter, out, stream=None):
    _check(_lib.kvc_swiglu(_ptr(gate_up), int(n), int(inter), _ptr(out), _stream(stream)))


def kvc_projection(m, n, k, a, n_a_rows, a_rows, w, residual, c, stream=None):
    _check(_lib.kvc_projection(int(m), int(n), int(k), _ptr(a), int(n_a_rows), _ptr(a_rows), _ptr(w),
                               _ptr(residual), _ptr(c), _stream(stream)))


def _ptrs(items):
    """ctypes array of pointers (tensors, integer addresses or None)."""
    if items is None:
        return None
    vals = [_ptr(x) for x in items]
    return (_vp * max(len(vals), 1))(*vals)


def kvc_stage_layer(layout, plan, k_chunks, v_chunks, k_cache, v_cache, stream=None):
    kc, vc = _ptrs(k_chunks), _ptrs(v_chunks)
    _check(_lib.kvc_stage_layer(_lref(layout), _pref(plan), kc, vc, _ptr(k_cache), _ptr(v_cache),
                                _stream(stream)))


def kvc_stage_layers(layout, plan, n_layers, k_chunks, v_chunks, k_cache, v_cache, events=None, stream=None):
    """k_chunks / v_chunks: flat lists, layer l's chunk i at l * n_chunks + i; k_cache, v_cache:
    one device tensor per layer; events: one per layer (torch.cuda.Event, raw hipEvent_t
    integer or None) or None."""
    ev = None
    if events is not None:
        ev = [None if e is None else (e.cuda_event if hasattr(e, "cuda_event") else int(e)) for e in events]
    _check(_lib.kvc_stage_layers(_lref(layout), _pref(plan), int(n_layers), _ptrs(k_chunks), _ptrs(v_chunks),
                                 _ptrs(k_cache), _ptrs(v_cache), _ptrs(ev), _stream(stream)))


__all__ = [n for n in _SIGS] + ["Layout", "Plan", "KvcError", "LIB_PATH", "kvc_layout", "kvc_plan"]
