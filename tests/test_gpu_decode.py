"""GPU parity of the decode step (frac_decode_step) against the float64 oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36314_amd as frac
from paper_2609_36314_amd.workloads import DECODE, Workload
from harness import TOL, assert_close, device_inputs, f64

pytestmark = pytest.mark.gpu


def _tau(M):
    t32 = oracle.default_tau(M).astype(np.float32)
    return torch.from_numpy(t32).cuda(), t32.astype(np.float64)


def _step_kw(inp, s):
    kw = {}
    for k in ("lam", "read_logit", "write_logit"):
        if k in inp:
            kw[k] = inp[k][s].contiguous()
    if "D" in inp:
        kw["D"] = inp["D"]
    a = inp["alpha"]
    alpha = a[s].contiguous() if isinstance(a, torch.Tensor) and a.dim() == 3 else a
    return alpha, kw


def _oracle_step(inp, s, state, tau64, sl=None):
    alpha, kw = _step_kw(inp, s)
    x, dt, Bm, Cm = f64(inp["x"][s]), f64(inp["dt"][s]), f64(inp["Bm"][s]), f64(inp["Cm"][s])
    H = x.shape[1]
    al = f64(alpha)
    al = np.broadcast_to(al if np.ndim(al) != 1 else al[None, :], dt.shape)
    okw = {k: f64(v) for k, v in kw.items()}
    if sl is not None:
        b, h = sl
        g = h * Bm.shape[1] // H
        x, dt, al = x[b:b + 1, h:h + 1], dt[b:b + 1, h:h + 1], al[b:b + 1, h:h + 1]
        Bm, Cm = Bm[b:b + 1, g:g + 1], Cm[b:b + 1, g:g + 1]
        for k in ("lam", "read_logit", "write_logit"):
            if k in okw:
                okw[k] = okw[k][b:b + 1, h:h + 1]
        if "D" in okw:
            okw["D"] = okw["D"][h:h + 1]
    return oracle.decode_step(state, x, dt, Bm, Cm, al, tau64, **okw)


CASES = {
    "bf16": Workload("t", 3, 1, 4, 64, 128, 4, decode_steps=6, init_state=True),
    "f32 extras groups": Workload("t", 2, 1, 4, 32, 64, 3, ngroups=2, io_dtype="f32", decode_steps=5,
                                  init_state=True, extras=True),
    "bf16 M8 P16": Workload("t", 2, 1, 2, 16, 32, 8, decode_steps=4, init_state=True),
    # the paper's bank sizes beyond the scan's 8 modes
    "bf16 M16 P128": Workload("t", 2, 1, 2, 128, 64, 16, decode_steps=3, init_state=True, extras=True),
    "f32 M32 N16": Workload("t", 1, 1, 3, 32, 16, 32, io_dtype="f32", decode_steps=3, init_state=True,
                            extras=True),
    "bf16 M11": Workload("t", 2, 1, 2, 64, 32, 11, decode_steps=3, init_state=True, extras=True),
}


@pytest.mark.parametrize("name", list(CASES))
def test_decode_parity_small(name):
    w = CASES[name]
    inp = device_inputs(w, seed=1)
    tau_d, tau64 = _tau(w.nmodes)
    state = inp["init_state"].clone()
    ref_state = f64(inp["init_state"])
    tol = TOL[w.io_dtype]
    for s in range(w.decode_steps):
        alpha, kw = _step_kw(inp, s)
        y = frac.decode_step(state, inp["x"][s], inp["dt"][s], inp["Bm"][s], inp["Cm"][s], alpha, tau_d, **kw)
        torch.cuda.synchronize()
        yr, ref_state = _oracle_step(inp, s, ref_state, tau64)
        assert_close("y step %d" % s, f64(y), yr, tol)
    for m in range(w.nmodes):
        assert_close("state mode %d" % m, f64(state)[:, :, m], ref_state[:, :, m], tol)


def test_decode_matches_prefill():
    """Decode steps from a state == the chunked forward over the same tokens."""
    w = Workload("t", 2, 1, 4, 64, 128, 4, decode_steps=70, init_state=True)
    inp = device_inputs(w, seed=2)
    tau_d, _ = _tau(4)
    state = inp["init_state"].clone()
    ys = []
    for s in range(w.decode_steps):
        ys.append(frac.decode_step(state, inp["x"][s], inp["dt"][s], inp["Bm"][s], inp["Cm"][s], 0.5, tau_d))
    seq = lambda k: inp[k].transpose(0, 1).contiguous()
    y_f, fs = frac.scan_fwd(seq("x"), seq("dt"), seq("Bm"), seq("Cm"), 0.5, tau_d, init_state=inp["init_state"],
                            return_final_state=True)
    torch.cuda.synchronize()
    assert_close("y", f64(torch.stack(ys, 1)), f64(y_f), TOL["bf16"])
    assert_close("state", f64(state), f64(fs), 1e-3)


@pytest.mark.parametrize("M", [16, 32])
def test_prefill_then_decode_with_the_paper_bank(M):
    """The hand-off at the paper's bank sizes with B/C: a chunked forward over a prompt
    (modes in blocks of eight) returns the final state, decode steps continue from it,
    and the tokens decoded match the chunked forward over prompt and continuation."""
    w = Workload("t", 2, 1, 2, 64, 128, M, decode_steps=150, init_state=True, extras=True)
    inp = device_inputs(w, seed=3)
    tau_d, _ = _tau(M)
    seq = lambda k: inp[k].transpose(0, 1).contiguous()
    x, dt, Bm, Cm, lam, rl, wl = (seq(k) for k in ("x", "dt", "Bm", "Cm", "lam", "read_logit", "write_logit"))
    alpha = seq("alpha")
    kw = lambda sl: dict(lam=lam[:, sl].contiguous(), read_logit=rl[:, sl].contiguous(),
                         write_logit=wl[:, sl].contiguous(), D=inp["D"])
    P0 = 130  # prompt: two chunks and a ragged third
    _, st = frac.scan_fwd(x[:, :P0].contiguous(), dt[:, :P0].contiguous(), Bm[:, :P0].contiguous(),
                          Cm[:, :P0].contiguous(), alpha[:, :P0].contiguous(), tau_d, init_state=inp["init_state"],
                          return_final_state=True, **kw(slice(0, P0)))
    ys = []
    for s in range(P0, w.decode_steps):
        c = lambda t: t[:, s].contiguous()
        ys.append(frac.decode_step(st, c(x), c(dt), c(Bm), c(Cm), c(alpha), tau_d,
                                   lam=c(lam), read_logit=c(rl), write_logit=c(wl), D=inp["D"]))
    y_f, fs = frac.scan_fwd(x, dt, Bm, Cm, alpha, tau_d, init_state=inp["init_state"], return_final_state=True,
                            **kw(slice(None)))
    torch.cuda.synchronize()
    print("prefill then decode, M", M, flush=True)
    assert_close("decoded y", f64(torch.stack(ys, 1)), f64(y_f[:, P0:]), TOL["bf16"])
    for m in range(M):  # (the chunked update rounds its matrix-core operands to bfloat16, decode does not)
        assert_close("state mode %d" % m, f64(st)[:, :, m], f64(fs)[:, :, m], TOL["bf16"])


def test_decode_full_size_sampled():
    """The decode workload at full size (2 GiB float32 state), three steps as the
    benchmark runs them, checked on sampled (batch, head) slices."""
    w = DECODE.scaled(decode_steps=3)
    inp = device_inputs(w, seed=0)
    tau_d, tau64 = _tau(w.nmodes)
    state = inp["init_state"].clone()
    slices = [(0, 0), (100, 31), (255, 63)]
    refs = {sl: f64(inp["init_state"][sl[0]:sl[0] + 1, sl[1]:sl[1] + 1]) for sl in slices}
    for s in range(w.decode_steps):
        y = frac.decode_step(state, inp["x"][s], inp["dt"][s], inp["Bm"][s], inp["Cm"][s], 0.5, tau_d)
        torch.cuda.synchronize()
        for sl in slices:
            yr, refs[sl] = _oracle_step(inp, s, refs[sl], tau64, sl=sl)
            b, h = sl
            assert_close("y step %d %s" % (s, sl), f64(y[b:b + 1, h:h + 1]), yr, TOL["bf16"])
    for sl in slices:
        b, h = sl
        assert_close("state %s" % (sl,), f64(state[b:b + 1, h:h + 1]), refs[sl], TOL["bf16"])
