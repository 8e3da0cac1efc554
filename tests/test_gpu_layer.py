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
