"""Helpers for GPU tests: move bfloat16 bit arrays to and from cuda:0."""
import math

import numpy as np
import torch

# Attention LSE tolerance.  The kernel normalises by the sum of the
# bfloat16-rounded softmax weights it multiplies V with (so O is an exact
# weighted average).  bfloat16 has 8 significant bits, so round-to-nearest
# moves each weight, and hence their sum, by at most 2^-8 of itself: the LSE
# is off by at most ln(1 + 2^-8) = 3.90e-3 (every weight rounded the same
# way), plus 1e-4 for the float32 exponentials, sums and logarithm.
LSE_ATOL = math.log1p(2.0 ** -8) + 1e-4


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


def device_normal_bf16(shape, seed, scale=1.0):
    """Seeded N(0, scale^2) draws rounded to bfloat16 on cuda:0 (int16 bits),
    for inputs too large to build on the host.  Drawn in slices of 2^28 so
    the float32 temporaries stay at 1 GiB."""
    g = torch.Generator(device=dev())
    g.manual_seed(seed)
    out = torch.empty(shape, dtype=torch.int16, device=dev())
    flat = out.view(-1)
    step = 1 << 28
    for i in range(0, flat.numel(), step):
        n = min(step, flat.numel() - i)
        flat[i:i + n] = (torch.randn(n, generator=g, device=dev()) * scale).to(torch.bfloat16).view(torch.int16)
    return out
