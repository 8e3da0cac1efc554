"""Frac selective mode-bank scan for MI355X (gfx950).

Python face of the C ABI in ``include/frac.h``.  The functions keep the C names
without the ``frac_`` prefix: ``scan_fwd``, ``scan_bwd``, ``decode_step``,
``scan_workspace_size``, ``default_tau``.  They take PyTorch tensors (device
memory), allocate outputs and workspace with PyTorch, and launch on the current
stream; the arithmetic runs in libfrac.so.
"""
from __future__ import annotations

import ctypes
from typing import Optional

import torch

from . import _lib
from ._lib import FracError, FracShape, FracFwdArgs, FracBwdArgs, FracStepArgs, FRAC_BF16, FRAC_F32

__all__ = ["scan_fwd", "scan_bwd", "decode_step", "scan_workspace_size", "default_tau", "FracError",
           "CHUNK"]

CHUNK = 64
TAU_MIN = 1.0
TAU_MAX = 2.0 ** 17


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _io_dtype(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return FRAC_BF16
    if t.dtype == torch.float32:
        return FRAC_F32
    raise TypeError("x/Bm/Cm must be float32 or bfloat16, got %s" % t.dtype)


def _f32(t, name):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.dtype != torch.float32:
        raise TypeError("%s must be a float32 tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t


_scalars = {}


def _scalar_tensor(v: float, device) -> torch.Tensor:
    """A cached one-element float32 device tensor holding v (read-only by the library)."""
    key = (float(v), str(device))
    t = _scalars.get(key)
    if t is None:
        if len(_scalars) > 256:
            _scalars.clear()
        t = torch.full((1,), float(v), dtype=torch.float32, device=device)
        _scalars[key] = t
    return t


def _strided(v, shape, device, name):
    """float32 scalar / broadcastable tensor -> (tensor, element strides over `shape`)."""
    if v is None:
        return None, (0,) * len(shape)
    if not isinstance(v, torch.Tensor):
        v = _scalar_tensor(v, device)
    if v.dtype != torch.float32:
        raise TypeError("%s must be float32" % name)
    e = v.expand(shape)
    return v, tuple(int(s) for s in e.stride())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _shape(x, Bm, nmodes, chunk, seqlen=None):
    """Bm None: the form without B/C projections (dstate 1, B = C = 1)."""
    if x.dim() == 4:
        Bsz, L, H, P = x.shape
        G, N = (1, 1) if Bm is None else (Bm.shape[2], Bm.shape[3])
    else:
        Bsz, H, P = x.shape
        L = 1
        G, N = (1, 1) if Bm is None else (Bm.shape[1], Bm.shape[2])
    return FracShape(Bsz, L if seqlen is None else seqlen, H, P, N, G, nmodes, chunk, _io_dtype(x))


def scan_workspace_size(shape: FracShape, backward: bool = False) -> int:
    """Bytes of workspace frac_scan_fwd / frac_scan_bwd need (frac_scan_workspace_size)."""
    return int(_lib.load().frac_scan_workspace_size(ctypes.byref(shape), int(bool(backward))))


def default_tau(M: int, tau_min: float = TAU_MIN, tau_max: float = TAU_MAX, device=None) -> torch.Tensor:
    """The paper's base timescale bank (frac_default_tau), as a float32 tensor."""
    out = (ctypes.c_float * M)()
    _lib.check(_lib.load().frac_default_tau(int(M), float(tau_min), float(tau_max), out))
    t = torch.tensor(list(out), dtype=torch.float32)
    return t if device is None else t.to(device)


def _fwd_struct(x, dt, Bm, Cm, alpha, tau, lam, read_logit, write_logit, D, init_state, y, final_state,
                chunk_states=None):
    Bsz, L, H, P = x.shape
    if (Bm is None) != (Cm is None):
        raise TypeError("Bm and Cm are both given or both None (B = C = 1)")
    if Bm is not None and (Bm.dtype != x.dtype or Cm.dtype != x.dtype):
        raise TypeError("x, Bm and Cm must share one dtype")
    for t, n in ((x, "x"), (Bm, "Bm"), (Cm, "Cm")):
        if t is not None and not t.is_contiguous():
            raise ValueError("%s must be contiguous" % n)
    alpha_t, a_str = _strided(alpha, (Bsz, L, H), x.device, "alpha")
    lam_t, l_str = _strided(lam, (Bsz, L, H), x.device, "lambda")
    a = FracFwdArgs()
    a.x, a.dt, a.Bm, a.Cm = _ptr(x), _ptr(_f32(dt, "dt")), _ptr(Bm), _ptr(Cm)
    a.alpha, a.alpha_stride = _ptr(alpha_t), (ctypes.c_int64 * 3)(*a_str)
    a.lam, a.lambda_stride = _ptr(lam_t), (ctypes.c_int64 * 3)(*l_str)
    a.read_logit, a.write_logit = _ptr(_f32(read_logit, "read_logit")), _ptr(_f32(write_logit, "write_logit"))
    a.tau, a.D = _ptr(_f32(tau, "tau")), _ptr(_f32(D, "D"))
    a.init_state = _ptr(_f32(init_state, "init_state"))
    a.y, a.final_state = _ptr(y), _ptr(final_state)
    a.chunk_states = _ptr(_f32(chunk_states, "chunk_states"))
    keep = (alpha_t, lam_t)
    return a, keep


def scan_fwd(x, dt, Bm, Cm, alpha, tau, *, lam=None, read_logit=None, write_logit=None, D=None,
             init_state=None, return_final_state=False, chunk=0, y=None, final_state=None, workspace=None,
             chunk_states=None):
    """Chunked parallel scan, forward (frac_scan_fwd).

    x [B,L,H,P], Bm/Cm [B,L,G,N] (float32 or bfloat16, one dtype), or both None for the
    form without B/C (B = C = 1, state [B,H,M,1,P], headdim <= 256, up to 32 modes); dt [B,L,H] f32;
    alpha, lam: float or f32 tensor broadcastable to [B,L,H]; read/write logits
    [B,L,H,M] f32; tau [M] f32; D [H] f32; init_state [B,H,M,N,P] f32.
    chunk_states (the form without B/C): an f32 tensor of chunk_states_size bytes the
    forward fills with the state entering each 64-token chunk, for scan_bwd.
    Returns y, or (y, final_state) when return_final_state."""
    M = int(tau.shape[0])
    shape = _shape(x, Bm, M, chunk)
    Bsz, L, H, P = x.shape
    N = int(shape.dstate)
    if y is None:
        y = torch.empty_like(x)
    if return_final_state and final_state is None:
        final_state = torch.empty((Bsz, H, M, N, P), dtype=torch.float32, device=x.device)
    args, keep = _fwd_struct(x, dt, Bm, Cm, alpha, tau, lam, read_logit, write_logit, D, init_state, y,
                             final_state if return_final_state else None, chunk_states)
    ws_bytes = scan_workspace_size(shape, False)
    if workspace is None and ws_bytes:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=x.device)
    _lib.check(_lib.load().frac_scan_fwd(ctypes.byref(shape), ctypes.byref(args), _ptr(workspace),
                                         ws_bytes if workspace is not None else 0, _stream()))
    del keep
    return (y, final_state) if return_final_state else y


def chunk_states_size(shape):
    """Bytes of the chunk states scan_fwd keeps for scan_bwd (frac_chunk_states_size; the
    form without B/C only)."""
    n = ctypes.c_size_t(0)
    _lib.check(_lib.load().frac_chunk_states_size(ctypes.byref(shape), ctypes.byref(n)))
    return int(n.value)


def chunk_states_like(x, nmodes):
    """An f32 tensor for the chunk states of x [B,L,H,P] with nmodes modes (no B/C)."""
    return torch.empty(chunk_states_size(_shape(x, None, nmodes, 0)) // 4, dtype=torch.float32, device=x.device)


def scan_fwd_noalloc(x, dt, Bm, Cm, alpha, tau, *, y, lam=None, read_logit=None, write_logit=None, D=None,
                     init_state=None, final_state=None, chunk=0):
    """frac_scan_fwd_noalloc: the forward with the library's static scratch in place of a
    workspace.  The outputs y (and final_state, when wanted) are the caller's; the library
    call allocates no device memory.  (A Python float for alpha or lam is turned into a
    cached one-element device tensor the first time it is seen: pass tensors where no
    allocation at all may happen.)"""
    M = int(tau.shape[0])
    shape = _shape(x, Bm, M, chunk)
    args, keep = _fwd_struct(x, dt, Bm, Cm, alpha, tau, lam, read_logit, write_logit, D, init_state, y, final_state)
    _lib.check(_lib.load().frac_scan_fwd_noalloc(ctypes.byref(shape), ctypes.byref(args), _stream()))
    del keep
    return y


def scan_fwd_noalloc_limit():
    """Bytes of the static scratch of scan_fwd_noalloc."""
    return int(_lib.load().frac_scan_fwd_noalloc_limit())


def scan_bwd(x, dt, Bm, Cm, alpha, tau, dy, *, lam=None, read_logit=None, write_logit=None, D=None,
             init_state=None, d_final_state=None, chunk=0, workspace=None, all_grads=False, chunk_states=None):
    """Chunked parallel scan, backward (frac_scan_bwd).

    Returns dict(dx, ddt, dBm, dCm, dD) with dD None when D is None.  With
    all_grads also dalpha [B,L,H], dlambda [B,L,H], dread_logit, dwrite_logit
    [B,L,H,M] and dinit_state [B,H,M,N,P] (N = 1 without B/C).  chunk_states: the tensor
    scan_fwd filled for these inputs (the form without B/C), read instead of recomputed."""
    M = int(tau.shape[0])
    shape = _shape(x, Bm, M, chunk)
    Bsz, L, H, P = x.shape
    if dy.dtype != x.dtype or not dy.is_contiguous():
        raise TypeError("dy must be contiguous with the dtype of x")
    fwd, keep = _fwd_struct(x, dt, Bm, Cm, alpha, tau, lam, read_logit, write_logit, D, init_state, None, None,
                            chunk_states)
    out = dict(dx=torch.empty_like(x), ddt=torch.empty_like(dt), dBm=None if Bm is None else torch.empty_like(Bm),
               dCm=None if Cm is None else torch.empty_like(Cm), dD=None if D is None else torch.empty_like(D))
    if all_grads:
        f32 = dict(dtype=torch.float32, device=x.device)
        out.update(dalpha=torch.empty((Bsz, L, H), **f32), dlambda=torch.empty((Bsz, L, H), **f32),
                   dread_logit=torch.empty((Bsz, L, H, M), **f32), dwrite_logit=torch.empty((Bsz, L, H, M), **f32),
                   dinit_state=torch.empty((Bsz, H, M, int(shape.dstate), P), **f32))
    a = FracBwdArgs()
    a.fwd = fwd
    a.dy, a.d_final_state = _ptr(dy), _ptr(_f32(d_final_state, "d_final_state"))
    a.dx, a.ddt, a.dBm, a.dCm, a.dD = (_ptr(out["dx"]), _ptr(out["ddt"]), _ptr(out["dBm"]), _ptr(out["dCm"]),
                                       _ptr(out["dD"]))
    if all_grads:
        a.dalpha, a.dlambda = _ptr(out["dalpha"]), _ptr(out["dlambda"])
        a.dread_logit, a.dwrite_logit = _ptr(out["dread_logit"]), _ptr(out["dwrite_logit"])
        a.dinit_state = _ptr(out["dinit_state"])
    ws_bytes = scan_workspace_size(shape, True)
    if workspace is None and ws_bytes:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=x.device)
    _lib.check(_lib.load().frac_scan_bwd(ctypes.byref(shape), ctypes.byref(a), _ptr(workspace),
                                         ws_bytes if workspace is not None else 0, _stream()))
    del keep
    return out


def decode_step(state, x, dt, Bm, Cm, alpha, tau, *, lam=None, read_logit=None, write_logit=None, D=None,
                y=None):
    """One decode token (frac_decode_step): updates `state` [B,H,M,N,P] f32 in place,
    returns y [B,H,P].  x [B,H,P], dt [B,H], Bm/Cm [B,G,N] (both None: B = C = 1, dstate 1)."""
    M = int(tau.shape[0])
    shape = _shape(x, Bm, M, 0, seqlen=1)
    Bsz, H, P = x.shape
    if (Bm is None) != (Cm is None):
        raise TypeError("Bm and Cm are both given or both None (B = C = 1)")
    if Bm is not None and (Bm.dtype != x.dtype or Cm.dtype != x.dtype):
        raise TypeError("x, Bm and Cm must share one dtype")
    alpha_t, a_str = _strided(alpha, (Bsz, H), x.device, "alpha")
    lam_t, l_str = _strided(lam, (Bsz, H), x.device, "lambda")
    if y is None:
        y = torch.empty_like(x)
    a = FracStepArgs()
    a.x, a.dt, a.Bm, a.Cm = _ptr(x), _ptr(_f32(dt, "dt")), _ptr(Bm), _ptr(Cm)
    a.alpha, a.alpha_stride = _ptr(alpha_t), (ctypes.c_int64 * 2)(*a_str)
    a.lam, a.lambda_stride = _ptr(lam_t), (ctypes.c_int64 * 2)(*l_str)
    a.read_logit, a.write_logit = _ptr(_f32(read_logit, "read_logit")), _ptr(_f32(write_logit, "write_logit"))
    a.tau, a.D = _ptr(_f32(tau, "tau")), _ptr(_f32(D, "D"))
    a.state, a.y = _ptr(_f32(state, "state")), _ptr(y)
    _lib.check(_lib.load().frac_decode_step(ctypes.byref(shape), ctypes.byref(a), _stream()))
    del alpha_t, lam_t
    return y


DT_RANGE = (1e-4, 1.0)       # the paper's clipping of the step
LAMBDA_RANGE = (0.25, 4.0)   # and of the fractional scale


def _params_struct(z_dt, dt_bias, z_alpha, z_lambda, v_read, v_write, p_read, p_write, dt_range, lambda_range):
    keep = [_f32(t, n) for t, n in ((z_dt, "z_dt"), (dt_bias, "dt_bias"), (z_alpha, "z_alpha"),
                                    (z_lambda, "z_lambda"), (v_read, "v_read"), (v_write, "v_write"),
                                    (p_read, "p_read"), (p_write, "p_write"))]
    a = _lib.FracParamsArgs()
    (a.z_dt, a.dt_bias, a.z_alpha, a.z_lambda, a.v_read, a.v_write, a.p_read, a.p_write) = (_ptr(t) for t in keep)
    a.dt_min, a.dt_max = dt_range
    a.lambda_min, a.lambda_max = lambda_range
    return a, keep


def _params_shape(z_dt, v):
    B, L, H = z_dt.shape
    return FracShape(B, L, H, 1, 1, 1, 1 if v is None else int(v.shape[-1]), 0, FRAC_F32)


def params_fwd(z_dt, z_alpha, *, dt_bias=None, z_lambda=None, v_read=None, v_write=None, p_read=None, p_write=None,
               dt_range=DT_RANGE, lambda_range=LAMBDA_RANGE):
    """Control-branch parameter construction (frac_params_fwd): z_* [B,L,H], dt_bias [H],
    v_* [B,L,H,M], p_* one-element tensors (all float32 on the device).  Returns
    dict(dt, alpha, lam, read_logit, write_logit), None for what has no input."""
    v = v_read if v_read is not None else v_write
    shape = _params_shape(z_dt, v)
    a, keep = _params_struct(z_dt, dt_bias, z_alpha, z_lambda, v_read, v_write, p_read, p_write, dt_range,
                             lambda_range)
    out = dict(dt=torch.empty_like(z_dt), alpha=torch.empty_like(z_dt),
               lam=None if z_lambda is None else torch.empty_like(z_dt),
               read_logit=None if v_read is None else torch.empty_like(v_read),
               write_logit=None if v_write is None else torch.empty_like(v_write))
    a.dt, a.alpha, a.lam = _ptr(out["dt"]), _ptr(out["alpha"]), _ptr(out["lam"])
    a.read_logit, a.write_logit = _ptr(out["read_logit"]), _ptr(out["write_logit"])
    _lib.check(_lib.load().frac_params_fwd(ctypes.byref(shape), ctypes.byref(a), _stream()))
    del keep
    return out


def params_bwd(z_dt, z_alpha, *, dt_bias=None, z_lambda=None, v_read=None, v_write=None, p_read=None, p_write=None,
               ddt=None, dalpha=None, dlambda=None, dread_logit=None, dwrite_logit=None, dt_range=DT_RANGE,
               lambda_range=LAMBDA_RANGE):
    """Backward of params_fwd (frac_params_bwd).  Returns dict(dz_dt, ddt_bias, dz_alpha,
    dz_lambda, dv_read, dv_write, dp_read, dp_write), None for what has no input."""
    v = v_read if v_read is not None else v_write
    shape = _params_shape(z_dt, v)
    f, keep = _params_struct(z_dt, dt_bias, z_alpha, z_lambda, v_read, v_write, p_read, p_write, dt_range,
                             lambda_range)
    grads = [_f32(t, n) for t, n in ((ddt, "ddt"), (dalpha, "dalpha"), (dlambda, "dlambda"),
                                     (dread_logit, "dread_logit"), (dwrite_logit, "dwrite_logit"))]
    H = z_dt.shape[-1]
    e = lambda t: None if t is None else torch.empty_like(t)
    out = dict(dz_dt=torch.empty_like(z_dt), ddt_bias=torch.empty(H, dtype=torch.float32, device=z_dt.device),
               dz_alpha=torch.empty_like(z_dt), dz_lambda=e(z_lambda), dv_read=e(v_read), dv_write=e(v_write),
               dp_read=None if v_read is None else torch.empty(1, dtype=torch.float32, device=z_dt.device),
               dp_write=None if v_write is None else torch.empty(1, dtype=torch.float32, device=z_dt.device))
    a = _lib.FracParamsBwdArgs()
    a.fwd = f
    a.ddt, a.dalpha, a.dlambda, a.dread_logit, a.dwrite_logit = (_ptr(t) for t in grads)
    for k in out:
        setattr(a, k, _ptr(out[k]))
    ws = torch.empty(_lib.load().frac_params_workspace_size(ctypes.byref(shape)), dtype=torch.uint8,
                     device=z_dt.device)
    _lib.check(_lib.load().frac_params_bwd(ctypes.byref(shape), ctypes.byref(a), _ptr(ws), ws.numel(), _stream()))
    del keep, grads
    return out


def _conv_struct(x, w, bias, activation):
    if x.dim() != 3 or not x.is_contiguous():
        raise ValueError("x must be a contiguous [B, L, C] tensor")
    C = x.shape[2]
    if w.dim() != 2 or w.shape[0] != C:
        raise ValueError("w must be [C, K]")
    keep = [_f32(w, "w"), _f32(bias, "bias")]
    a = _lib.FracConvArgs()
    a.x, a.w, a.bias = _ptr(x), _ptr(keep[0]), _ptr(keep[1])
    a.channels, a.width, a.activation = C, int(w.shape[1]), int(bool(activation))
    B, L, _ = x.shape
    shape = FracShape(B, L, 1, 1, 1, 1, 1, 0, _io_dtype(x))
    return a, shape, keep


def conv_fwd(x, w, *, bias=None, activation=True, y=None):
    """Causal depthwise convolution of the content branch (frac_conv_fwd): x [B,L,C]
    (bfloat16 or float32), w [C,K] and bias [C] float32; returns y like x."""
    a, shape, keep = _conv_struct(x, w, bias, activation)
    y = torch.empty_like(x) if y is None else y
    a.y = _ptr(y)
    _lib.check(_lib.load().frac_conv_fwd(ctypes.byref(shape), ctypes.byref(a), _stream()))
    del keep
    return y


def conv_bwd(x, w, dy, *, bias=None, activation=True):
    """Backward of conv_fwd (frac_conv_bwd): returns dict(dx, dw, dbias) (dbias None
    without a bias)."""
    a, shape, keep = _conv_struct(x, w, bias, activation)
    if dy.shape != x.shape or dy.dtype != x.dtype or not dy.is_contiguous():
        raise ValueError("dy must be contiguous, with the shape and dtype of x")
    out = dict(dx=torch.empty_like(x), dw=torch.empty_like(w),
               dbias=None if bias is None else torch.empty_like(bias))
    b = _lib.FracConvBwdArgs()
    b.fwd = a
    b.dy, b.dx, b.dw, b.dbias = _ptr(dy), _ptr(out["dx"]), _ptr(out["dw"]), _ptr(out["dbias"])
    nbytes = _lib.load().frac_conv_workspace_size(ctypes.byref(shape), a.channels, a.width)
    ws = torch.empty(max(1, nbytes), dtype=torch.uint8, device=x.device)
    _lib.check(_lib.load().frac_conv_bwd(ctypes.byref(shape), ctypes.byref(b), _ptr(ws), nbytes, _stream()))
    del keep
    return out


def _gnorm_struct(x, z, weight, group, eps):
    if x.dim() != 3 or not x.is_contiguous() or z.shape != x.shape or z.dtype != x.dtype or not z.is_contiguous():
        raise ValueError("x and z must be contiguous [B, L, C] tensors of one dtype")
    C = x.shape[2]
    keep = [_f32(weight, "weight")]
    a = _lib.FracGnormArgs()
    a.x, a.z, a.weight = _ptr(x), _ptr(z), _ptr(keep[0])
    a.channels, a.group, a.eps = C, C if group is None else int(group), float(eps)
    B, L, _ = x.shape
    return a, FracShape(B, L, 1, 1, 1, 1, 1, 0, _io_dtype(x)), keep


def gnorm_fwd(x, z, weight, *, group=None, eps=1e-5, y=None):
    """Gated RMS normalization of the layer output (frac_gnorm_fwd): x, z [B,L,C]
    (bfloat16 or float32), weight [C] float32, over groups of `group` channels (all C
    by default).  Returns y like x."""
    a, shape, keep = _gnorm_struct(x, z, weight, group, eps)
    y = torch.empty_like(x) if y is None else y
    a.y = _ptr(y)
    _lib.check(_lib.load().frac_gnorm_fwd(ctypes.byref(shape), ctypes.byref(a), _stream()))
    del keep
    return y


def gnorm_bwd(x, z, weight, dy, *, group=None, eps=1e-5):
    """Backward of gnorm_fwd (frac_gnorm_bwd): returns dict(dx, dz, dweight)."""
    a, shape, keep = _gnorm_struct(x, z, weight, group, eps)
    if dy.shape != x.shape or dy.dtype != x.dtype or not dy.is_contiguous():
        raise ValueError("dy must be contiguous, with the shape and dtype of x")
    out = dict(dx=torch.empty_like(x), dz=torch.empty_like(x), dweight=torch.empty_like(weight))
    b = _lib.FracGnormBwdArgs()
    b.fwd = a
    b.dy, b.dx, b.dz, b.dweight = _ptr(dy), _ptr(out["dx"]), _ptr(out["dz"]), _ptr(out["dweight"])
    nbytes = _lib.load().frac_gnorm_workspace_size(ctypes.byref(shape), a.channels)
    ws = torch.empty(max(1, nbytes), dtype=torch.uint8, device=x.device)
    _lib.check(_lib.load().frac_gnorm_bwd(ctypes.byref(shape), ctypes.byref(b), _ptr(ws), nbytes, _stream()))
    del keep
    return out
