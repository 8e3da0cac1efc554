"""The whole Frac layer (paper_2609_36314_amd.layer.FracLayer) in float32 on the GPU,
forward and backward through autograd, against a float64 chain of the oracles
(oracle.forward / backward for the scan, oracle.params, oracle.conv, oracle.gnorm)
joined by numpy matrix products.  Tolerance: relative L2 1e-3, five float32 stages
each held to 1e-4 in their own tests."""
import numpy as np
import pytest
import torch

import oracle
from oracle import conv as oc, gnorm as og, params as op
from paper_2609_36314_amd.layer import FracLayer
from harness import assert_close, f64

pytestmark = pytest.mark.gpu


def _reference(layer, h, dout):
    H, P, M, C = layer.H, layer.P, layer.M, layer.C
    p = {k: f64(v.detach()) for k, v in layer.named_parameters()}
    tau = f64(layer.tau)
    h, dout = f64(h), f64(dout)
    B, L, _ = h.shape
    zx = h @ p["in_proj"].T
    z, xc, zc = zx[..., :C], zx[..., C:2 * C], zx[..., 2 * C:]
    z_dt, z_a, z_l = zc[..., :H], zc[..., H:2 * H], zc[..., 2 * H:]
    u = oc.conv_forward(xc, p["conv_w"], p["conv_b"])
    vr = (u @ p["w_read"].T).reshape(B, L, H, M)
    vw = (u @ p["w_write"].T).reshape(B, L, H, M)
    pr, pw = float(p["p_read"][0]), float(p["p_write"][0])
    pp = op.params_forward(z_dt, p["dt_bias"], z_a, z_l, vr, vw, pr, pw)
    ones = np.ones((B, L, 1, 1))
    u4 = u.reshape(B, L, H, P)
    kw = dict(lam=pp["lambda"], read_logit=pp["read_logit"], write_logit=pp["write_logit"], D=p["D"])
    y, _ = oracle.forward(u4, pp["dt"], ones, ones, pp["alpha"], tau, **kw)
    y = y.reshape(B, L, C)
    o = og.gnorm_forward(y, z, p["norm_w"], layer.norm_group)
    out = o @ p["out_proj"].T
    # reverse
    g = {"out_proj": np.einsum("blo,blc->oc", dout, o)}
    do = dout @ p["out_proj"]
    gn = og.gnorm_backward(y, z, p["norm_w"], do, layer.norm_group)
    g["norm_w"] = gn["dweight"]
    sb = oracle.backward(u4, pp["dt"], ones, ones, pp["alpha"], tau, gn["dx"].reshape(B, L, H, P), **kw)
    g["D"] = sb["dD"]
    pb = op.params_backward(z_dt, p["dt_bias"], z_a, z_l, vr, vw, pr, pw, ddt=sb["ddt"], dalpha=sb["dalpha"],
                            dlambda=sb["dlambda"], dread_logit=sb["dread_logit"], dwrite_logit=sb["dwrite_logit"])
    g["dt_bias"], g["p_read"], g["p_write"] = pb["ddt_bias"], np.array([pb["dp_read"]]), np.array([pb["dp_write"]])
    dvr, dvw = pb["dv_read"].reshape(B, L, H * M), pb["dv_write"].reshape(B, L, H * M)
    g["w_read"] = np.einsum("blm,blc->mc", dvr, u)
    g["w_write"] = np.einsum("blm,blc->mc", dvw, u)
    du = sb["dx"].reshape(B, L, C) + dvr @ p["w_read"] + dvw @ p["w_write"]
    cb = oc.conv_backward(xc, p["conv_w"], du, p["conv_b"])
    g["conv_w"], g["conv_b"] = cb["dw"], cb["dbias"]
    dzx = np.concatenate([gn["dz"], cb["dx"], pb["dz_dt"], pb["dz_alpha"], pb["dz_lambda"]], axis=-1)
    g["in_proj"] = np.einsum("blk,bld->kd", dzx, h)
    return out, dzx @ p["in_proj"], g


@pytest.mark.parametrize("shape", [(2, 130, 32, 2, 64, 4, None), (1, 70, 48, 3, 32, 16, 32)])
def test_layer_forward_and_backward_match_the_oracle_chain(shape):
    B, L, d_model, H, P, M, grp = shape
    print("layer", shape, flush=True)
    layer = FracLayer(d_model, H, P, M, dtype=torch.float32, seed=5, norm_group=grp)
    with torch.no_grad():  # nonzero gates and conv bias so that every path carries gradient
        layer.p_read.fill_(0.4)
        layer.p_write.fill_(-0.3)
        layer.conv_b.normal_(0, 0.1)
        layer.D.normal_(1.0, 0.3)
    gen = torch.Generator().manual_seed(6)
    h = torch.randn(B, L, d_model, generator=gen).cuda().requires_grad_(True)
    dout = torch.randn(B, L, d_model, generator=gen).cuda()
    out = layer(h)
    out.backward(dout)
    torch.cuda.synchronize()
    ref_out, ref_dh, ref_g = _reference(layer, h.detach(), dout)
    tol = 1e-3
    assert_close("out", f64(out.detach()), ref_out, tol)
    assert_close("dh", f64(h.grad), ref_dh, tol)
    for name, prm in layer.named_parameters():
        assert_close("d" + name, f64(prm.grad), ref_g[name], tol)


def test_bf16_layer_stages_match_the_oracles_on_their_own_inputs():
    """The bfloat16 layer (the paper's shape scaled down: 2 heads of 64, 16 modes),
    forward and backward through autograd, with every call into the library
    recorded: each stage -- convolution, parameter construction, scan, gated
    normalization, forward and backward -- is recomputed by its float64 oracle from
    the inputs the GPU stage actually received (the bfloat16-rounded activations of
    the stages before it), so that each kernel's own error is measured apart from
    the rounding that the chain compounds.  The end-to-end errors against the
    float64 chain are printed beside them."""
    import paper_2609_36314_amd.layer as lay
    calls = {}

    def rec(name, fn):
        def wrapped(*a, **kw):
            out = fn(*a, **kw)
            calls[name] = (a, kw, out)
            return out
        return wrapped

    saved = {n: getattr(lay, n) for n in ("conv_fwd", "conv_bwd", "params_fwd", "params_bwd", "scan_fwd", "scan_bwd",
                                          "gnorm_fwd", "gnorm_bwd")}
    B, L, d_model, H, P, M = 2, 150, 64, 2, 64, 16
    layer = FracLayer(d_model, H, P, M, dtype=torch.bfloat16, seed=7)
    with torch.no_grad():
        layer.p_read.fill_(0.4)
        layer.p_write.fill_(-0.3)
        layer.conv_b.normal_(0, 0.1)
        layer.D.normal_(1.0, 0.3)
    gen = torch.Generator().manual_seed(8)
    h = torch.randn(B, L, d_model, generator=gen).to(torch.bfloat16).cuda().requires_grad_(True)
    dout = torch.randn(B, L, d_model, generator=gen).to(torch.bfloat16).cuda()
    try:
        for n, fn in saved.items():
            setattr(lay, n, rec(n, fn))
        out = layer(h)
        out.backward(dout)
        torch.cuda.synchronize()
    finally:
        for n, fn in saved.items():
            setattr(lay, n, fn)
    tol = 2e-2
    g = lambda t: None if t is None else f64(t)
    # convolution
    (x, w), kw, u = calls["conv_fwd"][0], calls["conv_fwd"][1], calls["conv_fwd"][2]
    assert_close("conv y", f64(u), oc.conv_forward(g(x), g(w), g(kw["bias"])), tol)
    (x, w, dy), kw, cb = calls["conv_bwd"]
    ref = oc.conv_backward(g(x), g(w), g(dy), g(kw["bias"]))
    for k in ("dx", "dw", "dbias"):
        assert_close("conv " + k, f64(cb[k]), ref[k], tol)
    # parameter construction (float32 in and out)
    (z_dt, z_a), kw, po = calls["params_fwd"]
    args = (g(z_dt), g(kw["dt_bias"]), g(z_a), g(kw["z_lambda"]), g(kw["v_read"]), g(kw["v_write"]),
            float(kw["p_read"][0]), float(kw["p_write"][0]))
    ref = op.params_forward(*args)
    for k, rk in (("dt", "dt"), ("alpha", "alpha"), ("lam", "lambda"), ("read_logit", "read_logit"),
                  ("write_logit", "write_logit")):
        assert_close("params " + k, f64(po[k]), ref[rk], 1e-4)
    _, kw, pg = calls["params_bwd"]
    ref = op.params_backward(*args, ddt=g(kw["ddt"]), dalpha=g(kw["dalpha"]), dlambda=g(kw["dlambda"]),
                             dread_logit=g(kw["dread_logit"]), dwrite_logit=g(kw["dwrite_logit"]))
    for k, rk in (("dz_dt", "dz_dt"), ("dz_alpha", "dz_alpha"), ("dz_lambda", "dz_lambda"), ("dv_read", "dv_read"),
                  ("dv_write", "dv_write"), ("ddt_bias", "ddt_bias")):
        assert_close("params " + k, f64(pg[k]), ref[rk], 1e-4)
    # scan without B/C, all gradients
    (x, dt, _, _, alpha, tau), kw, y = calls["scan_fwd"]
    ones = np.ones((B, L, 1, 1))
    okw = dict(lam=g(kw["lam"]), read_logit=g(kw["read_logit"]), write_logit=g(kw["write_logit"]), D=g(kw["D"]))
    ry, _ = oracle.forward(g(x), g(dt), ones, ones, g(alpha), g(tau), **okw)
    assert_close("scan y", f64(y), ry, tol)
    (x, dt, _, _, alpha, tau, dy), kw, sg = calls["scan_bwd"]
    ref = oracle.backward(g(x), g(dt), ones, ones, g(alpha), g(tau), g(dy), **okw)
    for k in ("dx", "ddt", "dalpha", "dlambda", "dread_logit", "dwrite_logit", "dD"):
        assert_close("scan " + k, f64(sg[k]), ref[k], tol)
    # gated normalization
    (x, z, w), kw, o = calls["gnorm_fwd"]
    assert_close("gnorm y", f64(o), og.gnorm_forward(g(x), g(z), g(w), kw["group"]), tol)
    (x, z, w, dy), kw, gg = calls["gnorm_bwd"]
    ref = og.gnorm_backward(g(x), g(z), g(w), g(dy), kw["group"])
    for k, rk in (("dx", "dx"), ("dz", "dz"), ("dweight", "dweight")):
        assert_close("gnorm " + k, f64(gg[k]), ref[rk], tol)
    # the compounded error of the whole bfloat16 chain, for the record
    from harness import rel_l2
    ref_out, ref_dh, ref_g = _reference(layer, h.detach(), dout)
    print("end-to-end bf16 vs float64 chain: out %.2e, dh %.2e" % (rel_l2(f64(out.detach()), ref_out),
                                                                   rel_l2(f64(h.grad), ref_dh)), flush=True)
    for name, prm in layer.named_parameters():
        print("  d%-10s rel-L2 %.2e" % (name, rel_l2(f64(prm.grad), ref_g[name])), flush=True)
