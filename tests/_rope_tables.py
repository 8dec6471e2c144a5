"""RoPE frequency tables of the models the paper evaluates (test inputs).

Llama-3.1 rescales the base table f_j = 500000^(-2j/128) by wavelength,
with factor 8, low/high-frequency factors 1 and 4 and an original context of
8192 tokens: wavelengths shorter than 8192/4 keep their frequency, those
longer than 8192/1 are divided by 8, and the band between interpolates
linearly in 8192/wavelength.  Written from that published definition.
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
