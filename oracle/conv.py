"""Float64 oracle of the content branch's causal depthwise 1-D convolution
(FracMixer, Sec. 3.3: a local depthwise causal convolution along the sequence;
convolution size 4 in the experiments).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: imported by ``tests/`` and
nothing in the product package.

Per batch b, token t, channel c, with weight w [C, K] and bias [C]:
  pre[b,t,c] = bias[c] + sum_{j=0}^{K-1} w[c,j] x[b, t-(K-1)+j, c]   (x = 0 before t = 0)
  y = silu(pre) = pre * sigmoid(pre)      (or y = pre without the activation)
The SiLU after the convolution follows the Mamba-2 block the paper builds on; the
paper does not name the activation.
"""
from __future__ import annotations

import numpy as np


def _sigmoid(v):
    return 0.5 * (1.0 + np.tanh(0.5 * v))


def conv_pre(x, w, bias=None):
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    B, L, C = x.shape
    K = w.shape[1]
    pre = np.zeros((B, L, C)) if bias is None else np.broadcast_to(np.asarray(bias, np.float64), (B, L, C)).copy()
    for j in range(K):
        shift = K - 1 - j  # tap j reads the token `shift` steps back
        if shift >= L:
            continue
        pre[:, shift:, :] += w[None, None, :, j] * x[:, :L - shift, :]
    return pre


def conv_forward(x, w, bias=None, activation=True):
    pre = conv_pre(x, w, bias)
    return pre * _sigmoid(pre) if activation else pre


def conv_backward(x, w, dy, bias=None, activation=True):
    """Returns dict(dx [B,L,C], dw [C,K], dbias [C])."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    B, L, C = x.shape
    K = w.shape[1]
    pre = conv_pre(x, w, bias)
    if activation:
        s = _sigmoid(pre)
        g = dy * (s + pre * s * (1.0 - s))
    else:
        g = dy
    dx = np.zeros_like(x)
    dw = np.zeros((C, K))
    for j in range(K):
        shift = K - 1 - j
        if shift >= L:
            continue
        dx[:, :L - shift, :] += w[None, None, :, j] * g[:, shift:, :]
        dw[:, j] = np.sum(g[:, shift:, :] * x[:, :L - shift, :], axis=(0, 1))
    return dict(dx=dx, dw=dw, dbias=g.sum(axis=(0, 1)))
