"""Float64 oracle of the control-branch parameter construction (FracMixer, Sec. 3.3;
clipping ranges of the experimental setup; gated read / write maps of the appendix
on the state-transition algorithm).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: imported by ``tests/`` and
nothing in the product package.

Per batch b, token t, head h (and mode m for the logits):
  dt          = clip(softplus(z_dt + dt_bias_h), dt_min, dt_max)   softplus as in Mamba
  alpha       = sigmoid(z_alpha)                                   0 < alpha < 1
  lambda      = clip(softplus(z_lambda), lambda_min, lambda_max)
  read_logit  = sigmoid(p_read)  * v_read                          v = W u from the caller's GEMM
  write_logit = sigmoid(p_write) * v_write
The paper clips dt to [1e-4, 1] and lambda to [0.25, 4].  The derivative of a clip is
taken as 1 on the closed interval and 0 outside it.
"""
from __future__ import annotations

import numpy as np

DT_RANGE = (1e-4, 1.0)
LAMBDA_RANGE = (0.25, 4.0)


def softplus(x):
    """log(1 + e^x), evaluated without overflow."""
    x = np.asarray(x, dtype=np.float64)
    return np.maximum(x, 0.0) + np.log1p(np.exp(-np.abs(x)))


def sigmoid(x):
    x = np.asarray(x, dtype=np.float64)
    return 0.5 * (1.0 + np.tanh(0.5 * x))


def _clip_pass(v, lo, hi):
    return ((v >= lo) & (v <= hi)).astype(np.float64)


def params_forward(z_dt, dt_bias, z_alpha, z_lambda=None, v_read=None, v_write=None, p_read=0.0, p_write=0.0,
                   dt_range=DT_RANGE, lambda_range=LAMBDA_RANGE):
    """Returns dict(dt, alpha, lambda, read_logit, write_logit) (absent inputs give None)."""
    z_dt = np.asarray(z_dt, dtype=np.float64)
    s = softplus(z_dt + np.asarray(dt_bias, dtype=np.float64))
    out = dict(dt=np.clip(s, *dt_range), alpha=sigmoid(z_alpha), **{"lambda": None},
               read_logit=None, write_logit=None)
    if z_lambda is not None:
        out["lambda"] = np.clip(softplus(z_lambda), *lambda_range)
    if v_read is not None:
        out["read_logit"] = sigmoid(p_read) * np.asarray(v_read, dtype=np.float64)
    if v_write is not None:
        out["write_logit"] = sigmoid(p_write) * np.asarray(v_write, dtype=np.float64)
    return out


def params_backward(z_dt, dt_bias, z_alpha, z_lambda=None, v_read=None, v_write=None, p_read=0.0, p_write=0.0,
                    ddt=None, dalpha=None, dlambda=None, dread_logit=None, dwrite_logit=None,
                    dt_range=DT_RANGE, lambda_range=LAMBDA_RANGE):
    """Chain rule through params_forward: returns dict(dz_dt, ddt_bias [H], dz_alpha,
    dz_lambda, dv_read, dv_write, dp_read, dp_write); gradients of absent outputs are
    taken as zero."""
    z_dt = np.asarray(z_dt, dtype=np.float64)
    zeros = np.zeros_like(z_dt)
    g = lambda a: zeros if a is None else np.asarray(a, dtype=np.float64)
    x = z_dt + np.asarray(dt_bias, dtype=np.float64)
    dz_dt = g(ddt) * _clip_pass(softplus(x), *dt_range) * sigmoid(x)
    sa = sigmoid(z_alpha)
    out = dict(dz_dt=dz_dt, ddt_bias=dz_dt.reshape(-1, dz_dt.shape[-1]).sum(axis=0),
               dz_alpha=g(dalpha) * sa * (1.0 - sa), dz_lambda=None, dv_read=None, dv_write=None,
               dp_read=0.0, dp_write=0.0)
    if z_lambda is not None:
        zl = np.asarray(z_lambda, dtype=np.float64)
        out["dz_lambda"] = g(dlambda) * _clip_pass(softplus(zl), *lambda_range) * sigmoid(zl)
    for side, v, dl, p in (("read", v_read, dread_logit, p_read), ("write", v_write, dwrite_logit, p_write)):
        if v is None:
            continue
        v = np.asarray(v, dtype=np.float64)
        dl = np.zeros_like(v) if dl is None else np.asarray(dl, dtype=np.float64)
        sp = float(sigmoid(p))
        out["dv_" + side] = sp * dl
        out["dp_" + side] = float(np.sum(dl * v)) * sp * (1.0 - sp)
    return out
