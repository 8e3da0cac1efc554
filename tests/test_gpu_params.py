"""GPU parity of the control-branch parameter construction (frac_params_fwd,
frac_params_bwd) against the float64 oracle in oracle/params.py."""
import numpy as np
import pytest
import torch

from oracle import params as op
import paper_2609_36314_amd as frac
from harness import TOL, assert_close, f64

pytestmark = pytest.mark.gpu


def _inputs(B, L, H, M, seed, full=True):
    g = torch.Generator().manual_seed(seed)
    r = lambda *s, sd=1.0, mu=0.0: (torch.randn(*s, generator=g) * sd + mu).float().cuda()
    inp = dict(z_dt=r(B, L, H, sd=2.0, mu=-2.0), z_alpha=r(B, L, H, sd=2.0))
    if full:
        inp.update(dt_bias=r(H), z_lambda=r(B, L, H, sd=2.0), v_read=r(B, L, H, M), v_write=r(B, L, H, M),
                   p_read=r(1), p_write=r(1))
    return inp


def _np(inp):
    return {k: f64(v) for k, v in inp.items()}


CASES = {"all inputs, ragged": (2, 300, 5, 7, True), "step and order only": (1, 77, 3, 4, False),
         "paper shape": (2, 2048, 16, 16, True)}


@pytest.mark.parametrize("name", list(CASES))
def test_params_forward_matches_oracle(name):
    B, L, H, M, full = CASES[name]
    inp = _inputs(B, L, H, M, seed=1, full=full)
    out = frac.params_fwd(**inp)
    torch.cuda.synchronize()
    n = _np(inp)
    ref = op.params_forward(n["z_dt"], n.get("dt_bias", 0.0), n["z_alpha"], n.get("z_lambda"), n.get("v_read"),
                            n.get("v_write"), float(n["p_read"][0]) if full else 0.0,
                            float(n["p_write"][0]) if full else 0.0)
    for k, rk in (("dt", "dt"), ("alpha", "alpha"), ("lam", "lambda"), ("read_logit", "read_logit"),
                  ("write_logit", "write_logit")):
        if ref[rk] is None:
            assert out[k] is None
            continue
        assert_close(k, f64(out[k]), ref[rk], TOL["f32"])
    assert f64(out["dt"]).min() >= np.float32(1e-4) and f64(out["dt"]).max() <= 1.0  # the range in float32
    if full:
        assert f64(out["lam"]).min() >= 0.25 and f64(out["lam"]).max() <= 4.0


@pytest.mark.parametrize("name", list(CASES))
def test_params_backward_matches_oracle(name):
    B, L, H, M, full = CASES[name]
    inp = _inputs(B, L, H, M, seed=2, full=full)
    g = torch.Generator().manual_seed(3)
    cot = dict(ddt=torch.randn(B, L, H, generator=g).cuda(), dalpha=torch.randn(B, L, H, generator=g).cuda())
    if full:
        cot.update(dlambda=torch.randn(B, L, H, generator=g).cuda(),
                   dread_logit=torch.randn(B, L, H, M, generator=g).cuda(),
                   dwrite_logit=torch.randn(B, L, H, M, generator=g).cuda())
    out = frac.params_bwd(**inp, **cot)
    torch.cuda.synchronize()
    n, c = _np(inp), _np(cot)
    ref = op.params_backward(n["z_dt"], n.get("dt_bias", 0.0), n["z_alpha"], n.get("z_lambda"), n.get("v_read"),
                             n.get("v_write"), float(n["p_read"][0]) if full else 0.0,
                             float(n["p_write"][0]) if full else 0.0, ddt=c["ddt"], dalpha=c["dalpha"],
                             dlambda=c.get("dlambda"), dread_logit=c.get("dread_logit"),
                             dwrite_logit=c.get("dwrite_logit"))
    for k in ("dz_dt", "ddt_bias", "dz_alpha", "dz_lambda", "dv_read", "dv_write"):
        if ref[k] is None:
            assert out[k] is None
            continue
        assert_close(k, f64(out[k]), ref[k], TOL["f32"])
    if full:
        for k in ("dp_read", "dp_write"):
            assert abs(float(out[k][0]) - ref[k]) <= 1e-4 * max(1.0, abs(ref[k])), k
    again = frac.params_bwd(**inp, **cot)
    torch.cuda.synchronize()
    for k, v in out.items():
        if v is not None:
            assert torch.equal(v, again[k]), k  # fixed-order sums
