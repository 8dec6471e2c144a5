"""Helpers for GPU tests: move bfloat16 bit arrays to and from cuda:0."""
import numpy as np
import torch


def dev():
    return torch.device("cuda:0")


def up(a, dtype=None):
    """numpy -> cuda tensor; uint16 bf16 bits travel as int16."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    t = torch.from_numpy(a).to(dev())
    return t if dtype is None else t.to(dtype)


def down_bf16(t):
    return t.detach().cpu().numpy().view(np.uint16)


def empty_bf16(*shape):
    return torch.empty(shape, dtype=torch.int16, device=dev())


def bytes_buf(n):
    return torch.empty(max(int(n), 16), dtype=torch.uint8, device=dev())


def within_tol(got, want, atol=2e-2, rtol=1e-2):
    """|got - want| <= atol + rtol |want| everywhere (bf16 output tolerance)."""
    err = np.abs(got - want)
    return bool(np.all(err <= atol + rtol * np.abs(want))), float(err.max() if err.size else 0.0)
