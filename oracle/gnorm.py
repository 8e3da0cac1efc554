"""Float64 oracle of the gated normalization of the Frac layer's output (Sec. 3.3:
the mixer output is processed by gated normalization before the output projection).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: imported by ``tests/`` and
nothing in the product package.

The paper names the operation only; the form here is the gated RMS normalization of
the Mamba-2 block the layer follows (gate applied before the normalization), over
groups of `group` consecutive channels of each token:
  u = x * silu(z)
  y = u / sqrt(mean_group(u^2) + eps) * weight
"""
from __future__ import annotations

import numpy as np


def _silu(v):
    return v * 0.5 * (1.0 + np.tanh(0.5 * v))


def _grouped(a, group):
    B, L, C = a.shape
    return a.reshape(B, L, C // group, group)


def gnorm_forward(x, z, weight, group, eps=1e-5):
    x, z, w = (np.asarray(a, dtype=np.float64) for a in (x, z, weight))
    u = _grouped(x * _silu(z), group)
    r = 1.0 / np.sqrt(np.mean(u * u, axis=-1, keepdims=True) + eps)
    return (u * r).reshape(x.shape) * w


def gnorm_backward(x, z, weight, dy, group, eps=1e-5):
    """Returns dict(dx, dz, dweight) by the chain rule through gnorm_forward."""
    x, z, w, dy = (np.asarray(a, dtype=np.float64) for a in (x, z, weight, dy))
    sg = 0.5 * (1.0 + np.tanh(0.5 * z))
    s = z * sg
    u = _grouped(x * s, group)
    r = 1.0 / np.sqrt(np.mean(u * u, axis=-1, keepdims=True) + eps)
    yh = u * r
    gw = _grouped(dy * w, group)
    du = r * (gw - yh * np.mean(gw * yh, axis=-1, keepdims=True))
    du = du.reshape(x.shape)
    dsilu = sg * (1.0 + z * (1.0 - sg))
    return dict(dx=du * s, dz=du * x * dsilu,
                dweight=np.sum(dy * yh.reshape(x.shape), axis=(0, 1)))
