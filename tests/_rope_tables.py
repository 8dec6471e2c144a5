"""RoPE frequency tables of the models the paper evaluates (test inputs).

Llama-3.1 rescales the base table f_j = 500000^(-2j/128) by wavelength,
with factor 8, low/high-frequency factors 1 and 4 and an original context of
8192 tokens: wavelengths shorter than 8192/4 keep their frequency, those
longer than 8192/1 are divided by 8, and the band between interpolates
linearly in 8192/wavelength.  Written from that published definition.

Qwen2.5 (the paper's other model, Section 4.1) extends its context with
YaRN: with base 1e6, scale factor s = 4 and an original context of L = 32768
tokens, each pair's frequency f_j is blended between f_j / s (interpolated)
and f_j (kept) by a ramp in r_j = L / wavelength_j: gamma = 0 for r_j < 1,
1 for r_j > 32, linear between; f'_j = (1 - gamma) f_j / s + gamma f_j.
Written from the YaRN paper's definition ("NTK-by-parts" with alpha = 1,
beta = 32); YaRN's attention temperature scales logits, not frequencies,
and is not part of the table.
"""
import numpy as np

import oracle


def llama31_inv_freq(head_dim=128, theta=500000.0, factor=8.0, low=1.0, high=4.0, ctx=8192.0):
    f = oracle.inv_freq(head_dim, theta)
    wavelen = 2.0 * np.pi / f
    out = f.copy()
    long_ = wavelen > ctx / low
    out[long_] = f[long_] / factor
    mid = ~long_ & ~(wavelen < ctx / high)
    t = (ctx / wavelen[mid] - low) / (high - low)
    out[mid] = (1.0 - t) * f[mid] / factor + t * f[mid]
    return out


def yarn_inv_freq(head_dim=128, theta=1000000.0, factor=4.0, ctx=32768.0, alpha=1.0, beta=32.0):
    f = oracle.inv_freq(head_dim, theta)
    r = ctx / (2.0 * np.pi / f)
    gamma = np.clip((r - alpha) / (beta - alpha), 0.0, 1.0)
    return (1.0 - gamma) * f / factor + gamma * f
