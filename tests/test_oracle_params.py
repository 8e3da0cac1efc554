"""Pins of the parameter-construction oracle (oracle/params.py) against facts that do
not come from it: closed-form values of softplus and sigmoid, the clipping ranges the
paper states for its experiments (dt in [1e-4, 1], lambda in [0.25, 4]), the open
ranges the nonlinearities enforce (0 < alpha < 1, lambda > 0, Sec. 3.3), and central
finite differences of the forward for every gradient."""
import math

import numpy as np

from oracle import params as op


def test_softplus_and_sigmoid_closed_forms():
    assert op.softplus(0.0) == math.log(2.0)
    assert abs(op.softplus(50.0) - 50.0) < 1e-15 * 50
    assert op.softplus(-50.0) > 0 and abs(op.softplus(-50.0) - math.exp(-50.0)) < 1e-30
    assert abs(op.softplus(1.0) - math.log(1.0 + math.e)) < 1e-15
    assert op.sigmoid(0.0) == 0.5
    assert abs(op.sigmoid(2.0) - 1.0 / (1.0 + math.exp(-2.0))) < 1e-15
    x = np.linspace(-30, 30, 61)
    assert np.allclose(op.sigmoid(x) + op.sigmoid(-x), 1.0, atol=1e-15)


def test_ranges_stated_by_the_paper():
    assert op.DT_RANGE == (1e-4, 1.0) and op.LAMBDA_RANGE == (0.25, 4.0)
    rng = np.random.default_rng(0)
    z = rng.normal(0, 6, (4, 50, 3))
    out = op.params_forward(z, np.zeros(3), z, z)
    assert out["dt"].min() == 1e-4 and out["dt"].max() == 1.0
    assert out["lambda"].min() == 0.25 and out["lambda"].max() == 4.0
    assert (out["alpha"] > 0).all() and (out["alpha"] < 1).all()
    inside = (op.softplus(z) > 1e-4) & (op.softplus(z) < 1.0)
    assert np.array_equal(out["dt"][inside], op.softplus(z)[inside])


def test_gated_logits_scale_by_sigmoid_of_the_gate():
    v = np.arange(6.0).reshape(1, 1, 2, 3)
    out = op.params_forward(np.zeros((1, 1, 2)), np.zeros(2), np.zeros((1, 1, 2)), v_read=v, v_write=-v,
                            p_read=0.0, p_write=math.log(3.0))
    assert np.array_equal(out["read_logit"], 0.5 * v)
    assert np.allclose(out["write_logit"], -0.75 * v, rtol=1e-15)


def test_gradients_match_finite_differences():
    rng = np.random.default_rng(1)
    B, L, H, M = 2, 5, 3, 4
    z_dt, z_a, z_l = (rng.normal(0, 2, (B, L, H)) for _ in range(3))
    bias = rng.normal(-1, 1, H)
    vr, vw = rng.normal(size=(B, L, H, M)), rng.normal(size=(B, L, H, M))
    pr, pw = 0.3, -0.7
    cot = {k: rng.normal(size=s) for k, s in (("dt", (B, L, H)), ("alpha", (B, L, H)), ("lambda", (B, L, H)),
                                              ("read_logit", (B, L, H, M)), ("write_logit", (B, L, H, M)))}

    def loss(z_dt, bias, z_a, z_l, vr, vw, pr, pw):
        o = op.params_forward(z_dt, bias, z_a, z_l, vr, vw, pr, pw)
        return sum(float(np.sum(o[k] * cot[k])) for k in cot)

    g = op.params_backward(z_dt, bias, z_a, z_l, vr, vw, pr, pw, ddt=cot["dt"], dalpha=cot["alpha"],
                           dlambda=cot["lambda"], dread_logit=cot["read_logit"], dwrite_logit=cot["write_logit"])
    args = [z_dt, bias, z_a, z_l, vr, vw, pr, pw]
    names = ["dz_dt", "ddt_bias", "dz_alpha", "dz_lambda", "dv_read", "dv_write", "dp_read", "dp_write"]
    h = 1e-6
    for i, name in enumerate(names):
        base = np.asarray(args[i], dtype=np.float64)
        fd = np.zeros(base.shape)
        for idx in np.ndindex(*base.shape):
            up, dn = base.copy(), base.copy()
            up[idx] += h
            dn[idx] -= h
            a_up, a_dn = list(args), list(args)
            a_up[i], a_dn[i] = (up if base.shape else float(up)), (dn if base.shape else float(dn))
            fd[idx] = (loss(*a_up) - loss(*a_dn)) / (2 * h)
        got = np.asarray(g[name], dtype=np.float64)
        # no point lies near a clip boundary, where the derivative jumps
        if name in ("dz_dt", "ddt_bias"):
            s = op.softplus(z_dt + bias)
            near = (np.abs(s - 1e-4) < 1e-5) | (np.abs(s - 1.0) < 1e-5)
            assert not near.any()
        if name == "dz_lambda":
            s = op.softplus(z_l)
            assert not ((np.abs(s - 0.25) < 1e-5) | (np.abs(s - 4.0) < 1e-5)).any()
        assert np.allclose(got, fd, rtol=1e-6, atol=1e-8), name


def test_clipped_entries_pass_no_gradient():
    z = np.array([[[-20.0, 0.0, 20.0]]])
    g = op.params_backward(z, np.zeros(3), z, z, ddt=np.ones_like(z), dlambda=np.ones_like(z))
    assert g["dz_dt"][0, 0, 0] == 0.0 and g["dz_dt"][0, 0, 2] == 0.0 and g["dz_dt"][0, 0, 1] == 0.5
    assert g["dz_lambda"][0, 0, 0] == 0.0 and g["dz_lambda"][0, 0, 2] == 0.0 and g["dz_lambda"][0, 0, 1] == 0.5
