"""Float64 CPU oracle for the Frac selective mode-bank scan.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py``; never by the product package.  The
arithmetic lives in ``frac_oracle.c`` (sequential float64 recurrence of Sec. 3.2
and the Appendix-D algorithm, with its reverse-mode derivative); this module only
marshals numpy arrays into it and builds it with gcc on first use.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "frac_oracle.c")
_LIB = os.path.join(_HERE, "libfrac_oracle.so")

TAU_MIN = 1.0
TAU_MAX = 2.0 ** 17


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (IEEE float64, no fast-math) into oracle/."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-fno-fast-math",
               "-ffp-contract=off", "-o", tmp, _SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB)
    return _LIB


class _Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in
                ("batch", "seqlen", "nheads", "headdim", "dstate", "ngroups", "nmodes")]


_DP = ctypes.POINTER(ctypes.c_double)


class _Inputs(ctypes.Structure):
    _fields_ = [(n, _DP) for n in ("x", "dt", "alpha", "lam", "Bm", "Cm", "read_logit",
                                   "write_logit", "tau", "D", "init_state")]


class _Grads(ctypes.Structure):
    _fields_ = [(n, _DP) for n in ("dx", "ddt", "dBm", "dCm", "dalpha", "dlambda",
                                   "dread_logit", "dwrite_logit", "dD", "dinit_state")]


_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        lib.frac_oracle_forward.argtypes = [ctypes.POINTER(_Dims), ctypes.POINTER(_Inputs), _DP, _DP]
        lib.frac_oracle_forward.restype = ctypes.c_int
        lib.frac_oracle_backward.argtypes = [ctypes.POINTER(_Dims), ctypes.POINTER(_Inputs), _DP, _DP,
                                             ctypes.POINTER(_Grads)]
        lib.frac_oracle_backward.restype = ctypes.c_int
        lib.frac_oracle_default_tau.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_double, _DP]
        lib.frac_oracle_default_tau.restype = None
        lib.frac_oracle_num_threads.argtypes = []
        lib.frac_oracle_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _f64(a):
    return None if a is None else np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(_DP)


def num_threads() -> int:
    """OpenMP threads the oracle runs on (OMP_NUM_THREADS, else all host cores)."""
    return int(_load().frac_oracle_num_threads())


def default_tau(M: int, tau_min: float = TAU_MIN, tau_max: float = TAU_MAX) -> np.ndarray:
    """Endpoint-inclusive geometric timescale bank on [tau_min, tau_max] (Appendix E)."""
    out = np.empty(M, dtype=np.float64)
    _load().frac_oracle_default_tau(int(M), float(tau_min), float(tau_max), _ptr(out))
    return out


def _prepare(x, dt, Bm, Cm, alpha, tau, lam, read_logit, write_logit, D, init_state):
    x = _f64(x)
    Bsz, L, H, P = x.shape
    Bm, Cm = _f64(Bm), _f64(Cm)
    G, N = Bm.shape[2], Bm.shape[3]
    assert Bm.shape == (Bsz, L, G, N) and Cm.shape == Bm.shape
    tau = _f64(tau)
    M = tau.shape[0]
    dt = _f64(np.broadcast_to(np.asarray(dt, np.float64), (Bsz, L, H)))
    alpha = _f64(np.broadcast_to(np.asarray(alpha, np.float64), (Bsz, L, H)))
    lam = None if lam is None else _f64(np.broadcast_to(np.asarray(lam, np.float64), (Bsz, L, H)))
    rl = None if read_logit is None else _f64(np.broadcast_to(read_logit, (Bsz, L, H, M)))
    wl = None if write_logit is None else _f64(np.broadcast_to(write_logit, (Bsz, L, H, M)))
    D = None if D is None else _f64(np.broadcast_to(np.asarray(D, np.float64), (H,)))
    init_state = None if init_state is None else _f64(init_state)
    if init_state is not None:
        assert init_state.shape == (Bsz, H, M, N, P)
    dims = _Dims(Bsz, L, H, P, N, G, M)
    arrays = dict(x=x, dt=dt, alpha=alpha, lam=lam, Bm=Bm, Cm=Cm, read_logit=rl, write_logit=wl,
                  tau=tau, D=D, init_state=init_state)
    inp = _Inputs(**{k: _ptr(v) for k, v in arrays.items()})
    return dims, inp, arrays


def forward(x, dt, Bm, Cm, alpha, tau, lam=None, read_logit=None, write_logit=None, D=None,
            init_state=None):
    """Sequential float64 scan.  Returns (y [B,L,H,P], final_state [B,H,M,N,P])."""
    dims, inp, arrays = _prepare(x, dt, Bm, Cm, alpha, tau, lam, read_logit, write_logit, D, init_state)
    Bsz, L, H, P = arrays["x"].shape
    N, M = dims.dstate, dims.nmodes
    y = np.empty((Bsz, L, H, P), np.float64)
    fs = np.empty((Bsz, H, M, N, P), np.float64)
    rc = _load().frac_oracle_forward(ctypes.byref(dims), ctypes.byref(inp), _ptr(y), _ptr(fs))
    if rc != 0:
        raise RuntimeError("frac_oracle_forward failed (%d)" % rc)
    return y, fs


def backward(x, dt, Bm, Cm, alpha, tau, dy, lam=None, read_logit=None, write_logit=None, D=None,
             init_state=None, d_final_state=None):
    """Reverse-mode derivative of ``forward``.

    Returns a dict with dx, ddt, dBm, dCm (summed over the heads of a group),
    dalpha [B,L,H], dlambda [B,L,H] (zeros when lam is None), dread_logit,
    dwrite_logit [B,L,H,M], dD [H] and dinit_state [B,H,M,N,P].
    """
    dims, inp, arrays = _prepare(x, dt, Bm, Cm, alpha, tau, lam, read_logit, write_logit, D, init_state)
    Bsz, L, H, P = arrays["x"].shape
    N, M, G = dims.dstate, dims.nmodes, dims.ngroups
    dy = _f64(dy)
    assert dy.shape == (Bsz, L, H, P)
    dfs = _f64(d_final_state)
    out = dict(dx=np.empty((Bsz, L, H, P)), ddt=np.empty((Bsz, L, H)), dBm=np.empty((Bsz, L, G, N)),
               dCm=np.empty((Bsz, L, G, N)), dalpha=np.empty((Bsz, L, H)), dlambda=np.empty((Bsz, L, H)),
               dread_logit=np.empty((Bsz, L, H, M)), dwrite_logit=np.empty((Bsz, L, H, M)),
               dD=np.empty((H,)), dinit_state=np.empty((Bsz, H, M, N, P)))
    grads = _Grads(**{k: _ptr(v) for k, v in out.items()})
    rc = _load().frac_oracle_backward(ctypes.byref(dims), ctypes.byref(inp), _ptr(dy), _ptr(dfs),
                                      ctypes.byref(grads))
    if rc != 0:
        raise RuntimeError("frac_oracle_backward failed (%d)" % rc)
    return out


def decode_step(state, x, dt, Bm, Cm, alpha, tau, lam=None, read_logit=None, write_logit=None, D=None):
    """One token of the recurrence: the forward loop with L = 1 from ``state``.

    x [B,H,P], dt/alpha [B,H], Bm/Cm [B,G,N], state [B,H,M,N,P].
    Returns (y [B,H,P], new_state)."""
    ex = lambda a: None if a is None else np.asarray(a)[:, None]
    lam_e = None if lam is None else np.broadcast_to(np.asarray(lam, np.float64), np.shape(dt))[:, None]
    y, fs = forward(ex(x), ex(dt), ex(Bm), ex(Cm),
                    np.broadcast_to(np.asarray(alpha, np.float64), np.shape(dt))[:, None], tau, lam=lam_e,
                    read_logit=ex(read_logit), write_logit=ex(write_logit), D=D, init_state=state)
    return y[:, 0], fs
