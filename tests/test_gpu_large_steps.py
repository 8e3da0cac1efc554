"""Effective steps dt * lambda^(1/alpha) over the paper's whole parameter range,
checked against the float64 oracle: the clipping ranges of the experimental setup
bound dt to [1e-4, 1] and lambda to [0.25, 4] but leave alpha = sigmoid(z) open
below, so steps near 1e19 (alpha 0.03, lambda 3.8) share chunks with steps near
1e-12 (alpha 0.05, lambda 0.3).  Training the layer reaches this state.  The scan
kernels form every decay from per-mode sums of the capped exponents r_m dtt in
float64, and the step-size gradient of every chunk whose total exponent reaches the
cut from its chunk-local form, so the result is held to the usual tolerances there:
y, the final state per mode, and every gradient (dx, ddt, dalpha, dlambda, both
logit gradients, dinit_state, dD, and dB, dC with B/C projections), float32 and
bfloat16, with unit-scale initial states and final-state gradients."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36314_amd as frac
from harness import TOL, assert_close, f64

pytestmark = pytest.mark.gpu

# tokens of the first three chunks (and the ragged tail) that take a huge step
BIG = (3, 40, 41, 43, 64, 90, 127, 129, 150, 151)


def _controls(B, L, H, M, seed):
    """Paper-range controls: alpha ~ U[0.02, 1], lambda ~ U[0.25, 4], dt ~ U[1e-4, 1];
    huge steps (alpha 0.03, lambda 3.8) on the BIG tokens, tiny ones (alpha 0.05,
    lambda 0.3) on the tokens right after them."""
    g = torch.Generator().manual_seed(seed)
    dt = torch.rand(B, L, H, generator=g) * (1.0 - 1e-4) + 1e-4
    alpha = torch.rand(B, L, H, generator=g) * 0.98 + 0.02
    lam = torch.rand(B, L, H, generator=g) * 3.75 + 0.25
    for t in BIG:
        if t < L:
            alpha[:, t], lam[:, t] = 0.03, 3.8
        for u in (t + 1, t + 2):
            if u < L and u not in BIG:
                alpha[:, u], lam[:, u] = 0.05, 0.3
    rl = torch.randn(B, L, H, M, generator=g)
    wl = torch.randn(B, L, H, M, generator=g)
    return g, dt, alpha, lam, rl, wl


def _run_case(io, bc, B, L, H, P, N, M, seed):
    g, dt, alpha, lam, rl, wl = _controls(B, L, H, M, seed)
    iot = torch.float32 if io == "f32" else torch.bfloat16
    x = torch.randn(B, L, H, P, generator=g).to(iot)
    dy = torch.randn(B, L, H, P, generator=g).to(iot)
    if bc:
        Bm = (torch.randn(B, L, 1, N, generator=g) / N ** 0.5).to(iot)
        Cm = (torch.randn(B, L, 1, N, generator=g) / N ** 0.5).to(iot)
    else:
        Bm = Cm = None
    n_st = N if bc else 1
    init = torch.randn(B, H, M, n_st, P, generator=g)
    dfin = torch.randn(B, H, M, n_st, P, generator=g)
    D = torch.randn(H, generator=g)
    t32 = oracle.default_tau(M).astype(np.float32)
    tau = torch.from_numpy(t32).cuda()
    c = lambda t: None if t is None else t.cuda().contiguous()
    kw = dict(lam=c(lam), read_logit=c(rl), write_logit=c(wl), D=c(D), init_state=c(init))
    print("large steps", io, "B/C" if bc else "no B/C", (B, L, H, P, N, M), "seed", seed, flush=True)
    y, fin = frac.scan_fwd(c(x), c(dt), c(Bm), c(Cm), c(alpha), tau, return_final_state=True, **kw)
    gr = frac.scan_bwd(c(x), c(dt), c(Bm), c(Cm), c(alpha), tau, c(dy), d_final_state=c(dfin), all_grads=True, **kw)
    torch.cuda.synchronize()
    if bc:
        Bo, Co = f64(Bm), f64(Cm)
    else:
        Bo = Co = np.ones((B, L, 1, 1))
    okw = dict(lam=f64(lam), read_logit=f64(rl), write_logit=f64(wl), D=f64(D), init_state=f64(init))
    ry, rfin = oracle.forward(f64(x), f64(dt), Bo, Co, f64(alpha), t32.astype(np.float64), **okw)
    rg = oracle.backward(f64(x), f64(dt), Bo, Co, f64(alpha), t32.astype(np.float64), f64(dy),
                         d_final_state=None if dfin is None else f64(dfin), **okw)
    tol = TOL[io]
    assert_close("y", f64(y), ry, tol)
    for m in range(M):
        assert_close("final_state mode %d" % m, f64(fin)[:, :, m], rfin[:, :, m], tol)
    keys = ["dx", "ddt", "dalpha", "dlambda", "dread_logit", "dwrite_logit", "dinit_state", "dD"]
    if bc:
        keys += ["dBm", "dCm"]
    for k in keys:
        assert_close(k, f64(gr[k]), rg[k], tol)


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_paper_form_paper_range_steps_match_the_oracle(io):
    _run_case(io, False, 1, 200, 2, 32, 1, 16, seed=0)


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_paper_form_paper_range_steps_wide_heads(io):
    """Head dim 256: the forward whose weights run ahead of the state (and its
    Gamma tiles with one exponential per pair for the modes past the factorisation
    bound) and the 128-column backward."""
    _run_case(io, False, 1, 200, 2, 256, 1, 16, seed=5)


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_bc_form_paper_range_steps_match_the_oracle(io):
    _run_case(io, True, 1, 160, 2, 32, 16, 8, seed=1)


def test_bc_form_paper_range_full_width_state():
    """The training-size state (N 128, headdim 64, M 8) with two workgroups per head in
    the state and rows sweeps, in bfloat16."""
    _run_case("bf16", True, 1, 140, 2, 64, 128, 8, seed=2)


def test_paper_form_paper_range_bank_of_32():
    _run_case("f32", False, 1, 130, 2, 64, 1, 32, seed=3)


def test_bc_form_paper_range_full_width_state_f32():
    """The same state in float32, with the gradient of the final state."""
    _run_case("f32", True, 1, 140, 2, 64, 128, 8, seed=4)
