"""GPU parity of the gated normalization (frac_gnorm_fwd, frac_gnorm_bwd) against
the float64 oracle in oracle/gnorm.py."""
import pytest
import torch

from oracle import gnorm as og
import paper_2609_36314_amd as frac
from harness import TOL, assert_close, f64

pytestmark = pytest.mark.gpu

# name: (B, L, C, group, io)
CASES = {
    "bf16 one group C4096 (paper layer width)": (2, 64, 4096, 4096, "bf16"),
    "bf16 groups of 256 (one head)": (2, 33, 4096, 256, "bf16"),
    "f32 groups of 8": (1, 17, 96, 8, "f32"),
    "f32 groups of 512, C 2560": (2, 9, 2560, 512, "f32"),
    "f32 C 40 in groups of 8": (3, 5, 40, 8, "f32"),
}


@pytest.mark.parametrize("name", list(CASES))
def test_gnorm_forward_and_backward_match_oracle(name):
    B, L, C, grp, io = CASES[name]
    g = torch.Generator().manual_seed(4)
    dt = torch.bfloat16 if io == "bf16" else torch.float32
    x, z, dy = (torch.randn(B, L, C, generator=g).to(dt).cuda() for _ in range(3))
    w = (1.0 + 0.1 * torch.randn(C, generator=g)).cuda()
    print("case", name, flush=True)
    y = frac.gnorm_fwd(x, z, w, group=grp)
    gr = frac.gnorm_bwd(x, z, w, dy, group=grp)
    torch.cuda.synchronize()
    tol = TOL[io]
    assert_close("y", f64(y), og.gnorm_forward(f64(x), f64(z), f64(w), grp), tol)
    ref = og.gnorm_backward(f64(x), f64(z), f64(w), f64(dy), grp)
    for k in ("dx", "dz", "dweight"):
        assert_close(k, f64(gr[k]), ref[k], tol)
    gr2 = frac.gnorm_bwd(x, z, w, dy, group=grp)
    torch.cuda.synchronize()
    for k in gr:
        assert torch.equal(gr[k], gr2[k]), k


def test_gnorm_empty_batch_gives_zero_weight_gradient():
    x = torch.empty(0, 5, 64, dtype=torch.float32, device="cuda")
    w = torch.randn(64).cuda()
    y = frac.gnorm_fwd(x, x.clone(), w)
    g = frac.gnorm_bwd(x, x.clone(), w, x.clone())
    torch.cuda.synchronize()
    assert y.shape == x.shape and not g["dweight"].any()
