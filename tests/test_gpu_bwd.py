"""GPU parity of the chunked backward scan (frac_scan_bwd) against the float64 oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36314_amd as frac
from paper_2609_36314_amd.workloads import TRAIN, Workload
from harness import TOL, assert_close, device_inputs, f64

pytestmark = pytest.mark.gpu


def _tau(M):
    t32 = oracle.default_tau(M).astype(np.float32)
    return torch.from_numpy(t32).cuda(), t32.astype(np.float64)


def _alpha64(inp, shape):
    a = inp["alpha"]
    if isinstance(a, torch.Tensor) and a.dim() == 1:
        return np.broadcast_to(f64(a)[None, None, :], shape)
    return np.broadcast_to(f64(a), shape)


def _run_bwd(inp, tau_d, dfs=None):
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state") if k in inp}
    return frac.scan_bwd(inp["x"], inp["dt"], inp["Bm"], inp["Cm"], inp["alpha"], tau_d, inp["dy"],
                         d_final_state=dfs, **kw)


def _oracle_bwd(inp, tau64, dfs=None, b=None, h=None):
    x, dt, Bm, Cm, dy = (f64(inp[k]) for k in ("x", "dt", "Bm", "Cm", "dy"))
    alpha = _alpha64(inp, dt.shape)
    kw = {k: f64(inp[k]) for k in ("lam", "read_logit", "write_logit", "D", "init_state") if k in inp}
    dF = None if dfs is None else f64(dfs)
    if b is not None:
        H = x.shape[2]
        G = Bm.shape[2]
        hs = slice(h, h + 1) if h is not None else slice(None)
        x, dt, alpha, dy = x[b:b + 1, :, hs], dt[b:b + 1, :, hs], alpha[b:b + 1, :, hs], dy[b:b + 1, :, hs]
        if h is not None:
            gi = h * G // H
            Bm, Cm = Bm[b:b + 1, :, gi:gi + 1], Cm[b:b + 1, :, gi:gi + 1]
        else:
            Bm, Cm = Bm[b:b + 1], Cm[b:b + 1]
        for k in ("lam",):
            if k in kw:
                kw[k] = kw[k][b:b + 1, :, hs]
        for k in ("read_logit", "write_logit"):
            if k in kw:
                kw[k] = kw[k][b:b + 1, :, hs]
        if "D" in kw:
            kw["D"] = kw["D"][hs]
        if "init_state" in kw:
            kw["init_state"] = kw["init_state"][b:b + 1, hs]
        if dF is not None:
            dF = dF[b:b + 1, hs]
    return oracle.backward(x, dt, Bm, Cm, alpha, tau64, dy, d_final_state=dF, **kw)


CASES = {
    "f32 extras dfinal": Workload("t", 1, 150, 2, 32, 32, 3, io_dtype="f32", extras=True, init_state=True,
                                  backward=True, final_state=True),
    "f32 tiny": Workload("t", 1, 256, 2, 16, 16, 4, io_dtype="f32", backward=True),
    "bf16 ragged": Workload("t", 2, 200, 4, 64, 128, 4, backward=True),
    "bf16 M8": Workload("t", 1, 130, 2, 64, 128, 8, backward=True, final_state=True),
    "bf16 groups extras": Workload("t", 2, 100, 4, 64, 64, 4, ngroups=2, extras=True, init_state=True,
                                   backward=True, final_state=True),
    "bf16 G=H M2 N32 P48": Workload("t", 1, 80, 2, 48, 32, 2, ngroups=2, backward=True),
    "bf16 M1 N16 P16": Workload("t", 2, 70, 3, 16, 16, 1, backward=True),
    "bf16 L1": Workload("t", 2, 1, 2, 64, 128, 4, backward=True, final_state=True, init_state=True),
    # float32 with 8 modes and a full-width state (single-buffered tiles and weights)
    "f32 M8 N128 extras dfinal": Workload("t", 1, 140, 2, 64, 128, 8, io_dtype="f32", extras=True, init_state=True,
                                          backward=True, final_state=True),
    # an odd mode count and state width, several chunks and a ragged tail
    "bf16 M5 N96 P32 extras": Workload("t", 2, 333, 2, 32, 96, 5, extras=True, init_state=True, backward=True,
                                       final_state=True),
    # 8 modes with heads in two groups (per-head dB, dC partials summed per group)
    "bf16 M8 groups P48": Workload("t", 1, 190, 4, 48, 64, 8, ngroups=2, backward=True),
    # banks of more than 8 modes: the sweeps once per block of eight modes
    "bf16 M16 extras dfinal": Workload("t", 1, 200, 2, 64, 128, 16, extras=True, init_state=True, backward=True,
                                       final_state=True),
    "f32 M12 N64 extras dfinal": Workload("t", 1, 150, 2, 32, 64, 12, io_dtype="f32", extras=True, init_state=True,
                                          backward=True, final_state=True),
    "bf16 M32 groups": Workload("t", 1, 140, 4, 64, 64, 32, ngroups=2, backward=True, final_state=True),
    # headdim above 64: groups of 64 columns, their sums over P in slots of their own
    "bf16 P128 extras dfinal": Workload("t", 1, 150, 2, 128, 128, 8, extras=True, init_state=True, backward=True,
                                        final_state=True),
    "f32 P96 M16 extras": Workload("t", 1, 130, 2, 96, 64, 16, io_dtype="f32", extras=True, init_state=True,
                                   backward=True, final_state=True),
    # the largest sizes built: four mode blocks x two column groups
    "bf16 max M32 N128 P128": Workload("t", 1, 100, 2, 128, 128, 32, extras=True, init_state=True, backward=True,
                                       final_state=True),
}


@pytest.mark.parametrize("name", list(CASES))
def test_bwd_parity_small(name):
    w = CASES[name]
    inp = device_inputs(w, seed=1)
    tau_d, tau64 = _tau(w.nmodes)
    dfs = inp.get("d_final_state")
    print("case", name, w, flush=True)
    g = _run_bwd(inp, tau_d, dfs)
    torch.cuda.synchronize()
    ref = _oracle_bwd(inp, tau64, dfs)
    tol = TOL[w.io_dtype]
    assert_close("dx", f64(g["dx"]), ref["dx"], tol)
    assert_close("ddt", f64(g["ddt"]), ref["ddt"], tol)
    assert_close("dB", f64(g["dBm"]), ref["dBm"], tol)
    assert_close("dC", f64(g["dCm"]), ref["dCm"], tol)
    if "D" in inp:
        assert_close("dD", f64(g["dD"]), ref["dD"], tol)


ALL_GRAD_CASES = ["f32 extras dfinal", "f32 M8 N128 extras dfinal", "bf16 M5 N96 P32 extras", "bf16 groups extras",
                  "bf16 M8", "bf16 L1", "bf16 M16 extras dfinal", "f32 M12 N64 extras dfinal", "bf16 M32 groups",
                  "bf16 P128 extras dfinal", "f32 P96 M16 extras", "bf16 max M32 N128 P128"]


@pytest.mark.parametrize("moderate", [False, True])
@pytest.mark.parametrize("name", ALL_GRAD_CASES)
def test_bwd_all_gradients(name, moderate):
    """With B/C projections: the gradients of alpha, lambda, both logits and the
    initial state beside dx, ddt, dB, dC, dD.  The extras draw alpha and lambda over
    the paper's ranges; `moderate` redraws them from alpha ~ U[0.3, 0.9], lambda ~
    U[0.5, 2] (factors lambda^{1/alpha} up to 10, long runs of chunks below the cut)."""
    w = CASES[name]
    if moderate and not w.extras:
        pytest.skip("no lambda or per-token alpha to redraw")
    inp = device_inputs(w, seed=5)
    if moderate:
        g0 = torch.Generator().manual_seed(55)
        shp = inp["dt"].shape
        inp["alpha"] = (torch.rand(shp, generator=g0) * 0.6 + 0.3).cuda()
        inp["lam"] = (torch.rand(shp, generator=g0) * 1.5 + 0.5).cuda()
    tau_d, tau64 = _tau(w.nmodes)
    dfs = inp.get("d_final_state")
    print("case", name, w, flush=True)
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state") if k in inp}
    g = frac.scan_bwd(inp["x"], inp["dt"], inp["Bm"], inp["Cm"], inp["alpha"], tau_d, inp["dy"],
                      d_final_state=dfs, all_grads=True, **kw)
    torch.cuda.synchronize()
    ref = _oracle_bwd(inp, tau64, dfs)
    tol = TOL[w.io_dtype]
    # (dalpha is per (b, t, h) on both sides, also where alpha is broadcast)
    for k in ("dx", "ddt", "dBm", "dCm", "dinit_state", "dread_logit", "dwrite_logit", "dalpha"):
        assert_close(k, f64(g[k]), ref[k], tol)
    if "lam" in inp:
        assert_close("dlambda", f64(g["dlambda"]), ref["dlambda"], tol)
    if "D" in inp:
        assert_close("dD", f64(g["dD"]), ref["dD"], tol)


@pytest.mark.parametrize("io,M,N", [("f32", 4, 32), ("bf16", 4, 32), ("bf16", 8, 128)])
def test_bwd_large_steps_use_direct_decay(io, M, N):
    """Steps large enough that r A_Q exceeds the factorisation bound for the fast
    modes (the per-pair exponential path), in float32 and bfloat16."""
    w = Workload("t", 1, 140, 2, 32, N, M, io_dtype=io, backward=True)
    inp = device_inputs(w, seed=3)
    inp["dt"] = (inp["dt"] * 8.0).contiguous()
    tau_d, tau64 = _tau(M)
    print("case", io, M, N, flush=True)
    g = _run_bwd(inp, tau_d)
    torch.cuda.synchronize()
    ref = _oracle_bwd(inp, tau64)
    for k, rk in (("dx", "dx"), ("ddt", "ddt"), ("dBm", "dBm"), ("dCm", "dCm")):
        assert_close(io + " " + k, f64(g[k]), ref[rk], TOL[io])


def test_bwd_deterministic():
    w = Workload("t", 2, 192, 4, 64, 128, 4, backward=True)
    inp = device_inputs(w, seed=4)
    tau_d, _ = _tau(4)
    g1 = _run_bwd(inp, tau_d)
    g2 = _run_bwd(inp, tau_d)
    torch.cuda.synchronize()
    for k in ("dx", "ddt", "dBm", "dCm"):
        assert torch.equal(g1[k], g2[k]), k


def test_bwd_full_size_sampled_bank_of_16():
    """The training workload with the paper's bank of 16 modes (two blocks of eight),
    at full size: dx and ddt on sampled heads, the last batch element and last head
    among them."""
    w = TRAIN.scaled(nmodes=16)
    inp = device_inputs(w, seed=6)
    tau_d, tau64 = _tau(w.nmodes)
    print("full-size", w.name, "M16", flush=True)
    g = _run_bwd(inp, tau_d)
    torch.cuda.synchronize()
    for k in ("dx", "ddt", "dBm", "dCm"):
        assert torch.isfinite(g[k].float()).all(), k
    for (b, h) in [(0, 0), (3, 63)]:
        ref = _oracle_bwd(inp, tau64, b=b, h=h)
        assert_close("dx[%d,:,%d]" % (b, h), f64(g["dx"][b:b + 1, :, h:h + 1]), ref["dx"], TOL["bf16"])
        assert_close("ddt[%d,:,%d]" % (b, h), f64(g["ddt"][b:b + 1, :, h:h + 1]), ref["ddt"], TOL["bf16"])


def test_bwd_full_size_all_grads_sampled():
    """The training workload at full size with lambda, both logits, D, an initial
    state and a final-state gradient drawn over the paper's ranges, all gradients
    (the all-gradients launch the benchmark times): every per-head gradient of the
    first and the last (batch, head) recomputed by the oracle."""
    w = TRAIN.scaled(extras=True, init_state=True, final_state=True)
    inp = device_inputs(w, seed=7)
    tau_d, tau64 = _tau(w.nmodes)
    dfs = inp["d_final_state"]
    print("full-size", w.name, "all gradients", flush=True)
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state")}
    g = frac.scan_bwd(inp["x"], inp["dt"], inp["Bm"], inp["Cm"], inp["alpha"], tau_d, inp["dy"], d_final_state=dfs,
                      all_grads=True, **kw)
    torch.cuda.synchronize()
    tol = TOL["bf16"]
    for (b, h) in [(0, 0), (3, 63)]:
        ref = _oracle_bwd(inp, tau64, dfs, b=b, h=h)
        print("slice", b, h, flush=True)
        for k in ("dx", "ddt", "dalpha", "dlambda", "dread_logit", "dwrite_logit"):
            assert_close("%s[%d,:,%d]" % (k, b, h), f64(g[k][b:b + 1, :, h:h + 1]), ref[k], tol)
        assert_close("dinit_state[%d,%d]" % (b, h), f64(g["dinit_state"][b:b + 1, h:h + 1]), ref["dinit_state"], tol)


def test_bwd_full_size_sampled():
    """The training workload at full size (batch 4, L 4096, 64 heads, M 8), as the
    benchmark launches it.  dx and ddt are checked on sampled heads (they depend
    on their own head only); dB and dC, summed over all 64 heads, on batch
    element 0 recomputed by the oracle for every head."""
    w = TRAIN
    inp = device_inputs(w, seed=0)
    tau_d, tau64 = _tau(w.nmodes)
    print("full-size", w.name, flush=True)
    g = _run_bwd(inp, tau_d)
    torch.cuda.synchronize()
    for k in ("dx", "ddt", "dBm", "dCm"):
        assert torch.isfinite(g[k].float()).all(), k
    for (b, h) in [(1, 5), (3, 60)]:
        ref = _oracle_bwd(inp, tau64, b=b, h=h)
        assert_close("dx[%d,:,%d]" % (b, h), f64(g["dx"][b:b + 1, :, h:h + 1]), ref["dx"], TOL["bf16"])
        assert_close("ddt[%d,:,%d]" % (b, h), f64(g["ddt"][b:b + 1, :, h:h + 1]), ref["ddt"], TOL["bf16"])
    ref = _oracle_bwd(inp, tau64, b=0)
    assert_close("dB[0]", f64(g["dBm"][0:1]), ref["dBm"], TOL["bf16"])
    assert_close("dC[0]", f64(g["dCm"][0:1]), ref["dCm"], TOL["bf16"])
    assert_close("dx[0]", f64(g["dx"][0:1]), ref["dx"], TOL["bf16"])


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_custom_tau_bank(io):
    """A caller's own timescale bank instead of the geometric default: unsorted, with
    modes faster than one step (tau < 1, rates above 1) beside very slow ones; the
    forward and every gradient against the oracle on the same bank."""
    M = 6
    w = Workload("t", 1, 170, 2, 64, 64, M, io_dtype=io, extras=True, init_state=True, backward=True,
                 final_state=True)
    inp = device_inputs(w, seed=21)
    t32 = np.array([30.0, 0.25, 4000.0, 1.0, 0.6, 150000.0], dtype=np.float32)
    tau_d, tau64 = torch.from_numpy(t32).cuda(), t32.astype(np.float64)
    dfs = inp["d_final_state"]
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state")}
    print("custom tau", io, flush=True)
    y, fin = frac.scan_fwd(inp["x"], inp["dt"], inp["Bm"], inp["Cm"], inp["alpha"], tau_d, return_final_state=True,
                           **kw)
    g = frac.scan_bwd(inp["x"], inp["dt"], inp["Bm"], inp["Cm"], inp["alpha"], tau_d, inp["dy"], d_final_state=dfs,
                      all_grads=True, **kw)
    torch.cuda.synchronize()
    okw = {k: f64(inp[k]) for k in ("lam", "read_logit", "write_logit", "D", "init_state")}
    args = (f64(inp["x"]), f64(inp["dt"]), f64(inp["Bm"]), f64(inp["Cm"]), f64(inp["alpha"]), tau64)
    ry, rfin = oracle.forward(*args, **okw)
    ref = oracle.backward(*args, f64(inp["dy"]), d_final_state=f64(dfs), **okw)
    tol = TOL[io]
    assert_close("y", f64(y), ry, tol)
    for m in range(M):
        assert_close("final_state mode %d" % m, f64(fin)[:, :, m], rfin[:, :, m], tol)
    for k in ("dx", "ddt", "dBm", "dCm", "dinit_state", "dread_logit", "dwrite_logit", "dalpha", "dlambda", "dD"):
        assert_close(k, f64(g[k]), ref[k], tol)
