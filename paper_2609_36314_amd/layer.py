"""The Frac layer of Sec. 3.3 on this package's kernels.

    h -> input projection -> [z | x | z_dt | z_alpha | z_lambda]
    u = silu(causal depthwise conv(x))                       (frac_conv_fwd, size 4)
    v_read, v_write = W_read u, W_write u                    (projections)
    dt, alpha, lambda, read / write logits                   (frac_params_fwd: softplus / sigmoid,
                                                              clipping, gates sigma(p))
    y = Frac state transition of u (B = C = 1) + D u         (frac_scan_fwd, dstate 1)
    o = gated RMS normalization of y with gate z             (frac_gnorm_fwd)
    out = output projection of o

The projections are plain GEMMs (torch.nn.functional.linear, the platform's BLAS);
every other step and its backward run in the package's HIP kernels, joined by
autograd Functions whose backward calls the library's backward entry points.  The
normalization before the input projection belongs to the residual block around
the layer and is not part of it here.
"""
from __future__ import annotations

import math

import torch
import torch.nn.functional as F

from . import (chunk_states_like, conv_bwd, conv_fwd, default_tau, gnorm_bwd, gnorm_fwd, params_bwd, params_fwd,
               scan_bwd, scan_fwd)


class _Conv(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w, b):
        ctx.save_for_backward(x, w, b)
        return conv_fwd(x, w, bias=b)

    @staticmethod
    def backward(ctx, dy):
        x, w, b = ctx.saved_tensors
        g = conv_bwd(x, w, dy.contiguous(), bias=b)
        return g["dx"], g["dw"], g["dbias"]


class _Params(torch.autograd.Function):
    @staticmethod
    def forward(ctx, z_dt, dt_bias, z_alpha, z_lambda, v_read, v_write, p_read, p_write):
        ctx.save_for_backward(z_dt, dt_bias, z_alpha, z_lambda, v_read, v_write, p_read, p_write)
        o = params_fwd(z_dt, z_alpha, dt_bias=dt_bias, z_lambda=z_lambda, v_read=v_read, v_write=v_write,
                       p_read=p_read, p_write=p_write)
        return o["dt"], o["alpha"], o["lam"], o["read_logit"], o["write_logit"]

    @staticmethod
    def backward(ctx, ddt, dalpha, dlam, drl, dwl):
        z_dt, dt_bias, z_alpha, z_lambda, v_read, v_write, p_read, p_write = ctx.saved_tensors
        c = lambda t: None if t is None else t.contiguous()
        g = params_bwd(z_dt, z_alpha, dt_bias=dt_bias, z_lambda=z_lambda, v_read=v_read, v_write=v_write,
                       p_read=p_read, p_write=p_write, ddt=c(ddt), dalpha=c(dalpha), dlambda=c(dlam),
                       dread_logit=c(drl), dwrite_logit=c(dwl))
        return (g["dz_dt"], g["ddt_bias"], g["dz_alpha"], g["dz_lambda"], g["dv_read"], g["dv_write"],
                g["dp_read"], g["dp_write"])


class _Scan(torch.autograd.Function):
    """The scan keeps the state entering each chunk from its forward (B H M P floats per
    64 tokens) for its backward, which then skips recomputing them."""

    @staticmethod
    def forward(ctx, x, dt, alpha, lam, rl, wl, D, tau):
        cs = chunk_states_like(x, int(tau.shape[0]))
        ctx.save_for_backward(x, dt, alpha, lam, rl, wl, D, tau, cs)
        return scan_fwd(x, dt, None, None, alpha, tau, lam=lam, read_logit=rl, write_logit=wl, D=D, chunk_states=cs)

    @staticmethod
    def backward(ctx, dy):
        x, dt, alpha, lam, rl, wl, D, tau, cs = ctx.saved_tensors
        g = scan_bwd(x, dt, None, None, alpha, tau, dy.contiguous(), lam=lam, read_logit=rl, write_logit=wl, D=D,
                     all_grads=True, chunk_states=cs)
        return g["dx"], g["ddt"], g["dalpha"], g["dlambda"], g["dread_logit"], g["dwrite_logit"], g["dD"], None


class _Gnorm(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, z, w, group):
        ctx.save_for_backward(x, z, w)
        ctx.group = group
        return gnorm_fwd(x, z, w, group=group)

    @staticmethod
    def backward(ctx, dy):
        x, z, w = ctx.saved_tensors
        g = gnorm_bwd(x, z, w, dy.contiguous(), group=ctx.group)
        return g["dx"], g["dz"], g["dweight"], None


class FracLayer(torch.nn.Module):
    """One Frac layer: d_model -> d_model, nheads heads of headdim channels, an
    nmodes-mode bank (the paper: 16 heads of 256, 16 modes, convolution size 4).
    dtype is the activation / projection dtype (bfloat16 or float32); the small
    per-channel parameters are float32.  norm_group: channels per group of the gated
    normalization (all of them by default; group / 8 must be a power of two)."""

    def __init__(self, d_model, nheads, headdim, nmodes=16, d_conv=4, dtype=torch.bfloat16, device="cuda", seed=0,
                 norm_group=None):
        super().__init__()
        H, P, M = nheads, headdim, nmodes
        C = H * P
        self.H, self.P, self.M, self.C = H, P, M, C
        self.norm_group = C if norm_group is None else int(norm_group)
        g = torch.Generator().manual_seed(seed)
        r = lambda *s, sd=1.0: (torch.randn(*s, generator=g) * sd)
        f32 = dict(dtype=torch.float32, device=device)
        P_ = lambda t, **kw: torch.nn.Parameter(t.to(**kw))
        self.in_proj = P_(r(2 * C + 3 * H, d_model, sd=1 / math.sqrt(d_model)), dtype=dtype, device=device)
        self.conv_w = P_(r(C, d_conv, sd=1 / math.sqrt(d_conv)), **f32)
        self.conv_b = P_(torch.zeros(C), **f32)
        # step bias: softplus^{-1} of steps spread log-uniformly over [1e-3, 1e-1]
        dt0 = torch.exp(torch.rand(H, generator=g) * (math.log(0.1) - math.log(1e-3)) + math.log(1e-3))
        self.dt_bias = P_(dt0 + torch.log(-torch.expm1(-dt0)), **f32)
        self.w_read = P_(r(H * M, C, sd=1 / math.sqrt(C)), dtype=dtype, device=device)
        self.w_write = P_(r(H * M, C, sd=1 / math.sqrt(C)), dtype=dtype, device=device)
        self.p_read = P_(torch.zeros(1), **f32)
        self.p_write = P_(torch.zeros(1), **f32)
        self.D = P_(torch.ones(H), **f32)
        self.norm_w = P_(torch.ones(C), **f32)
        self.out_proj = P_(r(d_model, C, sd=1 / math.sqrt(C)), dtype=dtype, device=device)
        self.register_buffer("tau", default_tau(M, device=device))

    def forward(self, h):
        B, L, _ = h.shape
        H, P, M, C = self.H, self.P, self.M, self.C
        zx = F.linear(h, self.in_proj)
        z, xc, zc = zx.split([C, C, 3 * H], dim=-1)
        zc = zc.float()
        z_dt, z_alpha, z_lambda = (zc[..., i * H:(i + 1) * H].contiguous() for i in range(3))
        u = _Conv.apply(xc.contiguous(), self.conv_w, self.conv_b)
        v_read = F.linear(u, self.w_read).float().view(B, L, H, M).contiguous()
        v_write = F.linear(u, self.w_write).float().view(B, L, H, M).contiguous()
        dt, alpha, lam, rl, wl = _Params.apply(z_dt, self.dt_bias, z_alpha, z_lambda, v_read, v_write,
                                               self.p_read, self.p_write)
        y = _Scan.apply(u.view(B, L, H, P), dt, alpha, lam, rl, wl, self.D, self.tau)
        o = _Gnorm.apply(y.view(B, L, C), z.contiguous(), self.norm_w, self.norm_group)
        return F.linear(o, self.out_proj)
