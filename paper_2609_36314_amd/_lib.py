"""ctypes binding of the C ABI in include/frac.h (libfrac.so).

Argument marshalling only: every step of the scan runs in the HIP kernels of
libfrac.so.  Tensors are PyTorch device tensors; they supply device pointers and
the current HIP stream.  Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import c_int, c_int32, c_int64, c_size_t, c_void_p, c_char_p, c_double, POINTER

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libfrac.so")

FRAC_F32 = 0
FRAC_BF16 = 1

STATUS = {0: "FRAC_OK", -1: "FRAC_ERR_INVALID_ARG", -2: "FRAC_ERR_UNSUPPORTED", -3: "FRAC_ERR_WORKSPACE",
          -4: "FRAC_ERR_HIP"}

# every symbol include/frac.h declares
EXPORTS = ("frac_scan_workspace_size", "frac_chunk_states_size", "frac_scan_fwd", "frac_scan_bwd", "frac_decode_step",
           "frac_default_tau", "frac_status_string", "frac_last_error", "frac_params_fwd", "frac_params_workspace_size",
           "frac_params_bwd", "frac_conv_fwd", "frac_conv_workspace_size", "frac_conv_bwd",
           "frac_gnorm_fwd", "frac_gnorm_workspace_size", "frac_gnorm_bwd", "frac_scan_fwd_noalloc",
           "frac_scan_fwd_noalloc_limit")


class FracShape(ctypes.Structure):
    _fields_ = [("batch", c_int64), ("seqlen", c_int64), ("nheads", c_int64), ("headdim", c_int64),
                ("dstate", c_int64), ("ngroups", c_int64), ("nmodes", c_int64), ("chunk", c_int64),
                ("io_dtype", c_int32)]


class FracFwdArgs(ctypes.Structure):
    _fields_ = [("x", c_void_p), ("dt", c_void_p), ("Bm", c_void_p), ("Cm", c_void_p),
                ("alpha", c_void_p), ("alpha_stride", c_int64 * 3),
                ("lam", c_void_p), ("lambda_stride", c_int64 * 3),
                ("read_logit", c_void_p), ("write_logit", c_void_p), ("tau", c_void_p), ("D", c_void_p),
                ("init_state", c_void_p), ("y", c_void_p), ("final_state", c_void_p),
                ("chunk_states", c_void_p)]


class FracBwdArgs(ctypes.Structure):
    _fields_ = [("fwd", FracFwdArgs), ("dy", c_void_p), ("d_final_state", c_void_p), ("dx", c_void_p),
                ("ddt", c_void_p), ("dBm", c_void_p), ("dCm", c_void_p), ("dD", c_void_p),
                ("dalpha", c_void_p), ("dlambda", c_void_p), ("dread_logit", c_void_p),
                ("dwrite_logit", c_void_p), ("dinit_state", c_void_p)]


class FracStepArgs(ctypes.Structure):
    _fields_ = [("x", c_void_p), ("dt", c_void_p), ("Bm", c_void_p), ("Cm", c_void_p),
                ("alpha", c_void_p), ("alpha_stride", c_int64 * 2),
                ("lam", c_void_p), ("lambda_stride", c_int64 * 2),
                ("read_logit", c_void_p), ("write_logit", c_void_p), ("tau", c_void_p), ("D", c_void_p),
                ("state", c_void_p), ("y", c_void_p)]


class FracParamsArgs(ctypes.Structure):
    _fields_ = [("z_dt", c_void_p), ("dt_bias", c_void_p), ("z_alpha", c_void_p), ("z_lambda", c_void_p),
                ("v_read", c_void_p), ("v_write", c_void_p), ("p_read", c_void_p), ("p_write", c_void_p),
                ("dt_min", ctypes.c_float), ("dt_max", ctypes.c_float), ("lambda_min", ctypes.c_float),
                ("lambda_max", ctypes.c_float), ("dt", c_void_p), ("alpha", c_void_p), ("lam", c_void_p),
                ("read_logit", c_void_p), ("write_logit", c_void_p)]


class FracParamsBwdArgs(ctypes.Structure):
    _fields_ = [("fwd", FracParamsArgs), ("ddt", c_void_p), ("dalpha", c_void_p), ("dlambda", c_void_p),
                ("dread_logit", c_void_p), ("dwrite_logit", c_void_p), ("dz_dt", c_void_p), ("ddt_bias", c_void_p),
                ("dz_alpha", c_void_p), ("dz_lambda", c_void_p), ("dv_read", c_void_p), ("dv_write", c_void_p),
                ("dp_read", c_void_p), ("dp_write", c_void_p)]


class FracConvArgs(ctypes.Structure):
    _fields_ = [("x", c_void_p), ("w", c_void_p), ("bias", c_void_p), ("y", c_void_p), ("channels", c_int64),
                ("width", ctypes.c_int32), ("activation", ctypes.c_int32)]


class FracConvBwdArgs(ctypes.Structure):
    _fields_ = [("fwd", FracConvArgs), ("dy", c_void_p), ("dx", c_void_p), ("dw", c_void_p), ("dbias", c_void_p)]


class FracGnormArgs(ctypes.Structure):
    _fields_ = [("x", c_void_p), ("z", c_void_p), ("weight", c_void_p), ("y", c_void_p), ("channels", c_int64),
                ("group", c_int64), ("eps", ctypes.c_float)]


class FracGnormBwdArgs(ctypes.Structure):
    _fields_ = [("fwd", FracGnormArgs), ("dy", c_void_p), ("dx", c_void_p), ("dz", c_void_p),
                ("dweight", c_void_p)]


class FracError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s: %s" % (STATUS.get(status, str(status)), message))
        self.status = status


_lib = None


def load():
    """Load libfrac.so (built by paper_2609_36314_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libfrac.so is not built (%s); run `python -m paper_2609_36314_amd.build`" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    lib.frac_scan_workspace_size.argtypes = [POINTER(FracShape), c_int]
    lib.frac_scan_workspace_size.restype = c_size_t
    lib.frac_chunk_states_size.argtypes = [POINTER(FracShape), POINTER(c_size_t)]
    lib.frac_chunk_states_size.restype = c_int
    lib.frac_scan_fwd.argtypes = [POINTER(FracShape), POINTER(FracFwdArgs), c_void_p, c_size_t, c_void_p]
    lib.frac_scan_fwd.restype = c_int
    lib.frac_scan_fwd_noalloc.argtypes = [POINTER(FracShape), POINTER(FracFwdArgs), c_void_p]
    lib.frac_scan_fwd_noalloc.restype = c_int
    lib.frac_scan_fwd_noalloc_limit.argtypes = []
    lib.frac_scan_fwd_noalloc_limit.restype = c_size_t
    lib.frac_scan_bwd.argtypes = [POINTER(FracShape), POINTER(FracBwdArgs), c_void_p, c_size_t, c_void_p]
    lib.frac_scan_bwd.restype = c_int
    lib.frac_decode_step.argtypes = [POINTER(FracShape), POINTER(FracStepArgs), c_void_p]
    lib.frac_decode_step.restype = c_int
    lib.frac_default_tau.argtypes = [c_int, c_double, c_double, POINTER(ctypes.c_float)]
    lib.frac_default_tau.restype = c_int
    lib.frac_status_string.argtypes = [c_int]
    lib.frac_status_string.restype = c_char_p
    lib.frac_last_error.argtypes = []
    lib.frac_last_error.restype = c_char_p
    lib.frac_params_fwd.argtypes = [POINTER(FracShape), POINTER(FracParamsArgs), c_void_p]
    lib.frac_params_fwd.restype = c_int
    lib.frac_params_workspace_size.argtypes = [POINTER(FracShape)]
    lib.frac_params_workspace_size.restype = c_size_t
    lib.frac_params_bwd.argtypes = [POINTER(FracShape), POINTER(FracParamsBwdArgs), c_void_p, c_size_t, c_void_p]
    lib.frac_params_bwd.restype = c_int
    lib.frac_conv_fwd.argtypes = [POINTER(FracShape), POINTER(FracConvArgs), c_void_p]
    lib.frac_conv_fwd.restype = c_int
    lib.frac_conv_workspace_size.argtypes = [POINTER(FracShape), c_int64, c_int]
    lib.frac_conv_workspace_size.restype = c_size_t
    lib.frac_conv_bwd.argtypes = [POINTER(FracShape), POINTER(FracConvBwdArgs), c_void_p, c_size_t, c_void_p]
    lib.frac_conv_bwd.restype = c_int
    lib.frac_gnorm_fwd.argtypes = [POINTER(FracShape), POINTER(FracGnormArgs), c_void_p]
    lib.frac_gnorm_fwd.restype = c_int
    lib.frac_gnorm_workspace_size.argtypes = [POINTER(FracShape), c_int64]
    lib.frac_gnorm_workspace_size.restype = c_size_t
    lib.frac_gnorm_bwd.argtypes = [POINTER(FracShape), POINTER(FracGnormBwdArgs), c_void_p, c_size_t, c_void_p]
    lib.frac_gnorm_bwd.restype = c_int
    _lib = lib
    return lib


def check(status: int):
    if status != 0:
        msg = load().frac_last_error().decode()
        raise FracError(status, msg)
