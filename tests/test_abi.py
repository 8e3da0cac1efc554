"""Host-side checks of the C ABI (no GPU needed): the library loads, exports every
function include/frac.h declares, validates arguments before touching the device,
and builds the paper's timescale bank like the oracle does."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2609_36314_amd import _lib
from paper_2609_36314_amd._lib import FracShape, FracFwdArgs, FracBwdArgs, FracStepArgs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "frac.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(frac_[a-z_]+)\s*\(", src)))


def test_header_declares_the_bound_symbols():
    assert _declared() == sorted(_lib.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = _lib.load()
    for name in _declared():
        assert hasattr(lib, name), name
    out = os.popen("nm -D --defined-only %s" % _lib.LIB_PATH).read()
    for name in _declared():
        assert re.search(r"\bT %s\b" % name, out), name


def test_status_strings():
    lib = _lib.load()
    for s in (0, -1, -2, -3, -4):
        assert lib.frac_status_string(s).decode().startswith(_lib.STATUS[s])


def test_default_tau_matches_oracle_grid():
    lib = _lib.load()
    for M in (1, 2, 4, 8, 16, 32):
        out = (ctypes.c_float * M)()
        assert lib.frac_default_tau(M, 1.0, 2.0 ** 17, out) == 0
        assert np.array_equal(np.array(out, np.float32), oracle.default_tau(M).astype(np.float32))
    assert lib.frac_default_tau(0, 1.0, 2.0, (ctypes.c_float * 1)()) == -1
    assert lib.frac_default_tau(3, 2.0, 1.0, (ctypes.c_float * 3)()) == -1


def _shape(**kw):
    d = dict(batch=1, seqlen=64, nheads=4, headdim=64, dstate=128, ngroups=1, nmodes=4, chunk=0, io_dtype=1)
    d.update(kw)
    return FracShape(**d)


@pytest.mark.parametrize("kw,status", [
    (dict(nheads=6, ngroups=4), -1),
    (dict(nmodes=0), -1),
    (dict(batch=-1), -1),
    (dict(io_dtype=7), -1),
    (dict(nmodes=33), -2),
    (dict(dstate=1, headdim=264), -2),
    (dict(dstate=12), -2),
    (dict(dstate=256), -2),
    (dict(headdim=20), -2),
    (dict(headdim=136, dstate=128), -2),
    (dict(headdim=136, dstate=16), -2),
    (dict(chunk=128), -2),
])
def test_invalid_shapes_are_rejected_on_the_host(kw, status):
    lib = _lib.load()
    sh = _shape(**kw)
    a = FracFwdArgs()
    assert lib.frac_scan_fwd(ctypes.byref(sh), ctypes.byref(a), None, 0, None) == status
    assert lib.frac_last_error().decode() != ""
    b = FracBwdArgs()
    assert lib.frac_scan_bwd(ctypes.byref(sh), ctypes.byref(b), None, 0, None) == status
    assert lib.frac_scan_workspace_size(ctypes.byref(sh), 0) == 0


def test_mode_blocks_are_sized_on_the_host():
    """More than 8 modes (up to 32) run the scan in blocks of eight: the shape is
    accepted and both workspaces hold the float32 partial output."""
    lib = _lib.load()
    for M in (9, 16, 32):
        sh = _shape(nmodes=M)
        for bwd in (0, 1):
            need = lib.frac_scan_workspace_size(ctypes.byref(sh), bwd)
            assert need >= sh.batch * sh.seqlen * sh.nheads * sh.headdim * 4, (M, bwd)
        a = FracFwdArgs()
        assert lib.frac_scan_fwd(ctypes.byref(sh), ctypes.byref(a), None, 0, None) == -1  # pointers missing
        b = FracBwdArgs()
        assert lib.frac_scan_bwd(ctypes.byref(sh), ctypes.byref(b), None, 0, None) == -1


def test_missing_pointers_are_rejected():
    lib = _lib.load()
    sh = _shape()
    a = FracFwdArgs()
    assert lib.frac_scan_fwd(ctypes.byref(sh), ctypes.byref(a), None, 0, None) == -1
    assert lib.frac_scan_fwd(None, ctypes.byref(a), None, 0, None) == -1
    st = FracStepArgs()
    sh1 = _shape(seqlen=1)
    assert lib.frac_decode_step(ctypes.byref(sh1), ctypes.byref(st), None) == -1
    assert lib.frac_decode_step(ctypes.byref(_shape(seqlen=2)), ctypes.byref(st), None) == -1


def test_misaligned_pointer_is_rejected():
    lib = _lib.load()
    sh = _shape()
    a = FracFwdArgs()
    for f in ("x", "dt", "Bm", "Cm", "alpha", "tau", "y"):
        setattr(a, f, ctypes.c_void_p(0x10000))
    a.x = ctypes.c_void_p(0x10002)
    assert lib.frac_scan_fwd(ctypes.byref(sh), ctypes.byref(a), None, 0, None) == -1
    assert "aligned" in lib.frac_last_error().decode()


def test_workspace_is_required_and_checked():
    lib = _lib.load()
    sh = _shape(batch=2, seqlen=200)
    need = lib.frac_scan_workspace_size(ctypes.byref(sh), 0)
    assert need > 0
    a = FracFwdArgs()
    for f in ("x", "dt", "Bm", "Cm", "alpha", "tau", "y"):
        setattr(a, f, ctypes.c_void_p(0x10000))
    assert lib.frac_scan_fwd(ctypes.byref(sh), ctypes.byref(a), None, 0, None) == -3
    assert lib.frac_scan_fwd(ctypes.byref(sh), ctypes.byref(a), ctypes.c_void_p(0x20000), need - 1, None) == -3


def test_noalloc_forward_rejects_shapes_beyond_its_scratch():
    """frac_scan_fwd_noalloc checks the shape's workspace against its static scratch on
    the host, before any device call."""
    lib = _lib.load()
    limit = lib.frac_scan_fwd_noalloc_limit()
    assert limit == 64 << 20
    sh = _shape(batch=16, seqlen=65536)
    assert lib.frac_scan_workspace_size(ctypes.byref(sh), 0) > limit
    a = FracFwdArgs()
    for f in ("x", "dt", "Bm", "Cm", "alpha", "tau", "y"):
        setattr(a, f, ctypes.c_void_p(0x10000))
    assert lib.frac_scan_fwd_noalloc(ctypes.byref(sh), ctypes.byref(a), None) == -3
    assert "static scratch" in lib.frac_last_error().decode()
    assert lib.frac_scan_fwd_noalloc(None, ctypes.byref(a), None) == -1


@pytest.mark.parametrize("nmodes,status", [(33, -2), (0, -1)])
def test_decode_mode_range_is_checked_on_the_host(nmodes, status):
    """frac_decode_step takes up to 32 modes; the shape is checked before any argument."""
    lib = _lib.load()
    sh = _shape(seqlen=1, nmodes=nmodes)
    a = FracStepArgs()
    assert lib.frac_decode_step(ctypes.byref(sh), ctypes.byref(a), None) == status


def test_projection_free_form_checks_its_arguments_on_the_host():
    """dstate 1 means B = C = 1: Bm and Cm (dBm, dCm) must be NULL there (and are
    required otherwise); its forward needs no workspace, its backward does."""
    lib = _lib.load()
    sh = _shape(dstate=1, headdim=256, nmodes=16)
    assert lib.frac_scan_workspace_size(ctypes.byref(sh), 0) == 0
    assert lib.frac_scan_workspace_size(ctypes.byref(sh), 1) > 0
    a = FracFwdArgs()
    buf = (ctypes.c_float * 64)()
    a.x = a.dt = a.alpha = a.tau = a.y = ctypes.cast(buf, ctypes.c_void_p)
    a.Bm = ctypes.cast(buf, ctypes.c_void_p)  # given although dstate is 1
    assert lib.frac_scan_fwd(ctypes.byref(sh), ctypes.byref(a), None, 0, None) == -1
    b = FracBwdArgs()
    b.fwd = a
    b.dy = b.dx = b.ddt = ctypes.cast(buf, ctypes.c_void_p)
    assert lib.frac_scan_bwd(ctypes.byref(sh), ctypes.byref(b), None, 0, None) == -1
    a.Bm = None
    b.fwd = a
    b.dBm = ctypes.cast(buf, ctypes.c_void_p)
    assert lib.frac_scan_bwd(ctypes.byref(sh), ctypes.byref(b), None, 0, None) == -1
    b.dBm = None
    assert lib.frac_scan_bwd(ctypes.byref(sh), ctypes.byref(b), None, 0, None) == -3  # no workspace


@pytest.mark.parametrize("field", ["dalpha", "dlambda", "dread_logit", "dwrite_logit", "dinit_state"])
def test_further_gradients_are_accepted_for_both_forms(field):
    """dalpha, dlambda, the logit gradients and dinit_state are produced with and without
    B/C projections: with every required pointer given, the call passes validation and
    stops only at the missing workspace (nothing is launched)."""
    lib = _lib.load()
    buf = (ctypes.c_float * 64)()
    p = ctypes.cast(buf, ctypes.c_void_p)
    for dstate in (16, 1):
        sh = _shape()
        sh.dstate = dstate
        a = FracFwdArgs()
        a.x = a.dt = a.alpha = a.tau = p
        if dstate > 1:
            a.Bm = a.Cm = p
        b = FracBwdArgs()
        b.fwd = a
        b.dy = b.dx = b.ddt = p
        if dstate > 1:
            b.dBm = b.dCm = p
        setattr(b, field, p)
        assert lib.frac_scan_bwd(ctypes.byref(sh), ctypes.byref(b), None, 0, None) == -3, lib.frac_last_error()


def test_parameter_construction_arguments_are_checked_on_the_host():
    from paper_2609_36314_amd._lib import FracParamsArgs, FracParamsBwdArgs
    lib = _lib.load()
    sh = _shape()
    buf = (ctypes.c_float * 64)()
    p = ctypes.cast(buf, ctypes.c_void_p)
    a = FracParamsArgs()
    a.dt_min, a.dt_max, a.lambda_min, a.lambda_max = 1e-4, 1.0, 0.25, 4.0
    assert lib.frac_params_fwd(ctypes.byref(sh), ctypes.byref(a), None) == -1  # no inputs
    a.z_dt = a.z_alpha = p
    assert lib.frac_params_fwd(ctypes.byref(sh), ctypes.byref(a), None) == -1  # no outputs
    a.dt = a.alpha = p
    a.v_read = p
    assert lib.frac_params_fwd(ctypes.byref(sh), ctypes.byref(a), None) == -1  # v_read without p_read
    assert "p_read" in lib.frac_last_error().decode()
    a.v_read = None
    a.z_lambda = p
    assert lib.frac_params_fwd(ctypes.byref(sh), ctypes.byref(a), None) == -1  # z_lambda without lambda
    a.z_lambda = None
    a.dt_min, a.dt_max = 1.0, 1e-4
    assert lib.frac_params_fwd(ctypes.byref(sh), ctypes.byref(a), None) == -1
    a.dt_min, a.dt_max = 1e-4, 1.0
    assert lib.frac_params_workspace_size(ctypes.byref(sh)) > 0
    b = FracParamsBwdArgs()
    b.fwd = a
    assert lib.frac_params_bwd(ctypes.byref(sh), ctypes.byref(b), None, 0, None) == -3  # no workspace


def test_convolution_arguments_are_checked_on_the_host():
    from paper_2609_36314_amd._lib import FracConvArgs, FracConvBwdArgs
    lib = _lib.load()
    sh = _shape()
    buf = (ctypes.c_float * 64)()
    p = ctypes.cast(buf, ctypes.c_void_p)
    a = FracConvArgs()
    a.channels, a.width, a.activation = 64, 4, 1
    assert lib.frac_conv_fwd(ctypes.byref(sh), ctypes.byref(a), None) == -1  # no pointers
    a.x = a.w = a.y = p
    for ch, wd, st in ((60, 4, -2), (64, 5, -2), (64, 0, -2), (0, 4, -2)):
        a.channels, a.width = ch, wd
        assert lib.frac_conv_fwd(ctypes.byref(sh), ctypes.byref(a), None) == st, (ch, wd)
    a.channels, a.width = 64, 4
    a.x = ctypes.c_void_p(ctypes.addressof(buf) + 4)
    assert lib.frac_conv_fwd(ctypes.byref(sh), ctypes.byref(a), None) == -1  # misaligned
    a.x = p
    assert lib.frac_conv_workspace_size(ctypes.byref(sh), 64, 4) > 0
    assert lib.frac_conv_workspace_size(ctypes.byref(sh), 64, 9) == 0
    b = FracConvBwdArgs()
    b.fwd = a
    b.dy = b.dx = b.dw = p
    assert lib.frac_conv_bwd(ctypes.byref(sh), ctypes.byref(b), None, 0, None) == -3  # no workspace


def test_gated_norm_arguments_are_checked_on_the_host():
    from paper_2609_36314_amd._lib import FracGnormArgs, FracGnormBwdArgs
    lib = _lib.load()
    sh = _shape()
    buf = (ctypes.c_float * 64)()
    p = ctypes.cast(buf, ctypes.c_void_p)
    a = FracGnormArgs()
    a.channels, a.group, a.eps = 64, 64, 1e-5
    assert lib.frac_gnorm_fwd(ctypes.byref(sh), ctypes.byref(a), None) == -1  # no pointers
    a.x = a.z = a.weight = a.y = p
    for ch, grp, st in ((64, 24, -2), (64, 48, -2), (60, 60, -2), (8192, 64, -2), (64, 128, -2)):
        a.channels, a.group = ch, grp
        assert lib.frac_gnorm_fwd(ctypes.byref(sh), ctypes.byref(a), None) == st, (ch, grp)
    a.channels, a.group, a.eps = 64, 16, -1.0
    assert lib.frac_gnorm_fwd(ctypes.byref(sh), ctypes.byref(a), None) == -1
    a.eps = 1e-5
    assert lib.frac_gnorm_workspace_size(ctypes.byref(sh), 64) > 0
    b = FracGnormBwdArgs()
    b.fwd = a
    b.dy = b.dx = b.dz = b.dweight = p
    assert lib.frac_gnorm_bwd(ctypes.byref(sh), ctypes.byref(b), None, 0, None) == -3  # no workspace


def test_chunk_states_are_sized_and_checked_on_the_host():
    """The forward keeps the per-chunk states for the backward only without B/C: there
    they are B H (ceil(L / 64) + 1) M P floats; with B/C the size query and a forward or
    backward given chunk_states are refused before anything is launched."""
    lib = _lib.load()
    n = ctypes.c_size_t(7)
    sh1 = _shape(dstate=1, headdim=256, nmodes=16, batch=2, seqlen=200)
    assert lib.frac_chunk_states_size(ctypes.byref(sh1), ctypes.byref(n)) == 0
    assert n.value == 2 * sh1.nheads * (4 + 1) * 16 * 256 * 4
    assert lib.frac_chunk_states_size(ctypes.byref(sh1), None) == -1
    sh = _shape()  # with B/C
    assert lib.frac_chunk_states_size(ctypes.byref(sh), ctypes.byref(n)) == -2 and n.value == 0
    buf = (ctypes.c_float * 64)()
    p = ctypes.cast(buf, ctypes.c_void_p)
    a = FracFwdArgs()
    a.x = a.dt = a.alpha = a.tau = a.y = a.Bm = a.Cm = p
    a.chunk_states = p
    assert lib.frac_scan_fwd(ctypes.byref(sh), ctypes.byref(a), None, 0, None) == -2
    assert "dstate 1" in lib.frac_last_error().decode()
    b = FracBwdArgs()
    b.fwd = a
    b.dy = b.dx = b.ddt = b.dBm = b.dCm = p
    assert lib.frac_scan_bwd(ctypes.byref(sh), ctypes.byref(b), None, 0, None) == -2
    a.chunk_states = ctypes.c_void_p(0x10004)  # misaligned, without B/C
    a.Bm = a.Cm = None
    assert lib.frac_scan_fwd(ctypes.byref(sh1), ctypes.byref(a), None, 0, None) == -1
    assert "aligned" in lib.frac_last_error().decode()
