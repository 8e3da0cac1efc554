"""Mittag-Leffler function tools for the oracle pins (test-side, independent of oracle/).

E_alpha(-s^alpha) is evaluated from the diffusive (spectral) representation of
Appendix A (density eq. r-density with lambda = 1), integrated in log-timescale
u = ln(tau) with the trapezoid rule (the integrand is smooth and decays doubly
exponentially for u -> -inf); the slowly decaying u -> +inf tail is split off
and integrated in closed form / by a short moment series.  The power series of
eq. Ea is provided for small arguments.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import gamma as Gamma


def ml_series(alpha: float, z, beta: float = 1.0, terms: int = 400):
    """E_{alpha,beta}(z) by its defining power series (eq. Ea / eq. frac-impulse)."""
    z = np.asarray(z, dtype=np.float64)
    out = np.zeros_like(z)
    for k in range(terms):
        g = alpha * k + beta
        if g > 170:
            break
        out = out + z ** k / Gamma(g)
    return out


def _r_tilde(alpha: float, u):
    """tau * R_{alpha,1}(tau) at tau = e^u (density eq. r-density times tau)."""
    sa = math.sin(math.pi * alpha)
    ca = math.cos(math.pi * alpha)
    ea = np.exp(alpha * np.asarray(u))
    return (sa / math.pi) / (ea + 2.0 * ca + 1.0 / ea)


def ml_neg_power(alpha: float, s, h: float = 0.01, u_lo: float = -12.0):
    """E_alpha(-s^alpha) for s > 0, 0 < alpha < 1, via the diffusive representation.

    E = int e^{-s e^{-u}} R~(u) du.  Split at u1 with s_max e^{-u1} = 1e-3: below u1
    trapezoid rule; above u1 expand e^{-s e^{-u}} = sum_k (-s)^k e^{-k u}/k!, with the
    k = 0 moment in closed form and k >= 1 moments by quadrature."""
    s = np.atleast_1d(np.asarray(s, dtype=np.float64))
    u1 = math.log(float(s.max()) * 1e3)
    n = int(math.ceil((u1 - u_lo) / h)) + 1
    u = np.linspace(u_lo, u1, n)
    w = np.full(u.shape, u[1] - u[0])
    w[0] = w[-1] = 0.5 * (u[1] - u[0])
    rt = _r_tilde(alpha, u) * w
    main = np.exp(-np.outer(s, np.exp(-u))) @ rt
    # tail moments  m_k = int_{u1}^{inf} R~(u) e^{-k u} du
    sa, ca = math.sin(math.pi * alpha), math.cos(math.pi * alpha)
    v1 = math.exp(alpha * u1)
    m0 = (math.pi / 2 - math.atan((v1 + ca) / sa)) / (math.pi * alpha)
    nt = int(math.ceil(60.0 / h)) + 1
    ut = np.linspace(u1, u1 + 60.0, nt)
    wt = np.full(ut.shape, ut[1] - ut[0])
    wt[0] = wt[-1] = 0.5 * (ut[1] - ut[0])
    rtt = _r_tilde(alpha, ut) * wt
    tail = np.full(s.shape, m0)
    for k in range(1, 8):
        mk = float(np.exp(-k * ut) @ rtt)
        tail = tail + (-s) ** k / math.factorial(k) * mk
    return main + tail
