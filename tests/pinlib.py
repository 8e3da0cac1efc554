"""Test-side reference formulations used to pin the oracle (independent of oracle/).

Each helper restates one formulation of the method from the paper in numpy,
structured differently from the oracle's sequential recurrence, so that a
mistake in either one shows up as a disagreement.
"""
from __future__ import annotations

import numpy as np
from scipy.special import softmax


def token_coefficients(dt, alpha, tau, lam=None, read_logit=None, write_logit=None):
    """rho, kappa, c, w per token and mode (last axis = mode).

    rho = exp(-dt lambda^(1/alpha) / tau_m)          eq. rho-beta-def-frac
    beta = 1 - rho (computed as -expm1)              Algorithm step 3 and the remark after it
    c, w = softmax_m(-alpha ln tau_m + logits)       eq. read-softmax (write: same form)
    kappa = beta * w                                 eq. frac-selective-update
    """
    dt = np.asarray(dt, np.float64)[..., None]
    alpha = np.broadcast_to(np.asarray(alpha, np.float64), dt.shape[:-1])[..., None]
    lam = 1.0 if lam is None else np.broadcast_to(np.asarray(lam, np.float64), dt.shape[:-1])[..., None]
    tau = np.asarray(tau, np.float64)
    arg = -dt * lam ** (1.0 / alpha) / tau
    rho = np.exp(arg)
    beta = -np.expm1(arg)
    prior = -alpha * np.log(tau)
    c = softmax(prior + (0.0 if read_logit is None else read_logit), axis=-1)
    w = softmax(prior + (0.0 if write_logit is None else write_logit), axis=-1)
    return rho, beta * w, c, w


def brute_force(x, dt, Bm, Cm, alpha, tau, lam=None, read_logit=None, write_logit=None, D=None,
                init_state=None):
    """O(L^2) pairwise form of the scan (appendix on the efficient implementation):

        y_t = sum_{k<=t} (C_t . B_k) Gamma_{t,k} x_k + sum_m c_{t,m} e^{l_{t,m}} C_t^T S0_m + D x_t
        Gamma_{t,k} = sum_m c_{t,m} kappa_{k,m} exp(l_{t,m} - l_{k,m})

    with l the inclusive cumulative log-retention along the whole sequence (tiny
    inputs only).  Also returns the final state in the same pairwise form."""
    x = np.asarray(x, np.float64)
    Bsz, L, H, P = x.shape
    G, N = Bm.shape[2], Bm.shape[3]
    M = len(tau)
    rho, kappa, c, _ = token_coefficients(np.broadcast_to(dt, (Bsz, L, H)), np.broadcast_to(alpha, (Bsz, L, H)),
                                          tau, lam, read_logit, write_logit)
    ell = np.cumsum(np.log(rho), axis=1)  # [B,L,H,M]
    y = np.zeros_like(x) if D is None else np.asarray(D, np.float64)[None, None, :, None] * x
    fs = np.zeros((Bsz, H, M, N, P))
    tri = np.tril(np.ones((L, L), bool))
    for b in range(Bsz):
        for h in range(H):
            g = h * G // H
            e = ell[b, :, h, :]
            diff = np.where(tri[:, :, None], e[:, None, :] - e[None, :, :], -np.inf)
            gam = np.einsum("tm,km,tkm->tk", c[b, :, h], kappa[b, :, h], np.exp(diff))
            cb = Cm[b, :, g] @ Bm[b, :, g].T
            y[b, :, h] += (cb * gam) @ x[b, :, h]
            wend = kappa[b, :, h] * np.exp(e[-1][None, :] - e)  # [k, m]
            fs[b, h] = np.einsum("km,kn,kp->mnp", wend, Bm[b, :, g], x[b, :, h])
            if init_state is not None:
                S0 = np.asarray(init_state, np.float64)[b, h]
                y[b, :, h] += np.einsum("tm,tn,mnp->tp", c[b, :, h] * np.exp(e), Cm[b, :, g], S0)
                fs[b, h] += np.exp(e[-1])[:, None, None] * S0
    return y, fs
