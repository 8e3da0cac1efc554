"""GPU parity of the causal depthwise convolution (frac_conv_fwd, frac_conv_bwd)
against the float64 oracle in oracle/conv.py."""
import pytest
import torch

from oracle import conv as oc
import paper_2609_36314_amd as frac
from harness import TOL, assert_close, f64

pytestmark = pytest.mark.gpu

# name: (B, L, C, K, io, bias, activation)
CASES = {
    "bf16 K4 bias silu ragged": (2, 300, 64, 4, "bf16", True, True),
    "f32 K3 no activation": (1, 77, 24, 3, "f32", False, False),
    "f32 K4 shorter than the kernel": (3, 2, 16, 4, "f32", True, True),
    "bf16 K1": (2, 65, 8, 1, "bf16", True, True),
    "bf16 paper content width C4096 K4": (2, 2048, 4096, 4, "bf16", True, True),
}


def _inputs(B, L, C, K, io, bias, seed):
    g = torch.Generator().manual_seed(seed)
    dt = torch.bfloat16 if io == "bf16" else torch.float32
    x = torch.randn(B, L, C, generator=g).to(dt).cuda()
    w = (torch.randn(C, K, generator=g) / K).cuda()
    b = (0.1 * torch.randn(C, generator=g)).cuda() if bias else None
    dy = torch.randn(B, L, C, generator=g).to(dt).cuda()
    return x, w, b, dy


@pytest.mark.parametrize("name", list(CASES))
def test_conv_forward_and_backward_match_oracle(name):
    B, L, C, K, io, bias, act = CASES[name]
    x, w, b, dy = _inputs(B, L, C, K, io, bias, seed=1)
    print("case", name, flush=True)
    y = frac.conv_fwd(x, w, bias=b, activation=act)
    g = frac.conv_bwd(x, w, dy, bias=b, activation=act)
    torch.cuda.synchronize()
    bb = None if b is None else f64(b)
    tol = TOL[io]
    assert_close("y", f64(y), oc.conv_forward(f64(x), f64(w), bb, act), tol)
    ref = oc.conv_backward(f64(x), f64(w), f64(dy), bb, act)
    assert_close("dx", f64(g["dx"]), ref["dx"], tol)
    assert_close("dw", f64(g["dw"]), ref["dw"], tol)
    if bias:
        assert_close("dbias", f64(g["dbias"]), ref["dbias"], tol)
    g2 = frac.conv_bwd(x, w, dy, bias=b, activation=act)
    torch.cuda.synchronize()
    for k in ("dx", "dw", "dbias"):
        if g[k] is not None:
            assert torch.equal(g[k], g2[k]), k  # fixed-order sums


def test_conv_empty_sequence_gives_zero_sums():
    x = torch.empty(2, 0, 16, dtype=torch.bfloat16, device="cuda")
    w = torch.randn(16, 4).cuda()
    b = torch.randn(16).cuda()
    y = frac.conv_fwd(x, w, bias=b)
    g = frac.conv_bwd(x, w, x.clone(), bias=b)
    torch.cuda.synchronize()
    assert y.shape == x.shape and g["dx"].shape == x.shape
    assert not g["dw"].any() and not g["dbias"].any()
