"""frac_scan_fwd_noalloc (the forward on the library's static scratch, for callers
that cannot allocate) against frac_scan_fwd with a caller workspace: two calls in a
row on one GPU, the first with a sequence long enough for the two-segment split (the
scratch then holds the C B^T tiles and the boundary state), the second smaller.  The
kernels are the same, so the outputs must agree bit for bit; the second call is also
checked against the float64 oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36314_amd as frac
from paper_2609_36314_amd.workloads import Workload
from harness import TOL, assert_close, device_inputs, f64

pytestmark = pytest.mark.gpu


def _both(w, seed):
    inp = device_inputs(w, seed=seed)
    tau = torch.from_numpy(oracle.default_tau(w.nmodes).astype(np.float32)).cuda()
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state") if k in inp}
    shape = frac._shape(inp["x"], inp["Bm"], w.nmodes, 0)
    need = frac.scan_workspace_size(shape, False)
    assert 0 < need <= frac.scan_fwd_noalloc_limit(), need
    print("no-alloc forward", w, "scratch bytes", need, flush=True)
    y_ref, fin_ref = frac.scan_fwd(inp["x"], inp["dt"], inp["Bm"], inp["Cm"], inp["alpha"], tau,
                                   return_final_state=True, **kw)
    y = torch.empty_like(inp["x"])
    fin = torch.empty_like(fin_ref)
    frac.scan_fwd_noalloc(inp["x"], inp["dt"], inp["Bm"], inp["Cm"], inp["alpha"], tau, y=y, final_state=fin, **kw)
    torch.cuda.synchronize()
    return inp, tau, y, fin, y_ref, fin_ref


def test_noalloc_forward_matches_the_workspace_forward_twice():
    big = Workload("t", 1, 1000, 4, 64, 128, 4, alpha_range=(0.3, 0.8), final_state=True, init_state=True)
    small = Workload("t", 2, 200, 2, 32, 64, 4, extras=True, final_state=True)
    _, _, y, fin, y_ref, fin_ref = _both(big, seed=11)
    assert torch.equal(y, y_ref)
    assert torch.equal(fin, fin_ref)
    inp, tau, y, fin, y_ref, fin_ref = _both(small, seed=12)
    assert torch.equal(y, y_ref)
    assert torch.equal(fin, fin_ref)
    M = small.nmodes
    Bo, Co = f64(inp["Bm"]), f64(inp["Cm"])
    okw = {k: f64(inp[k]) for k in ("lam", "read_logit", "write_logit", "D") if k in inp}
    ry, rfin = oracle.forward(f64(inp["x"]), f64(inp["dt"]), Bo, Co, f64(inp["alpha"]),
                              oracle.default_tau(M).astype(np.float32).astype(np.float64), **okw)
    assert_close("y", f64(y), ry, TOL["bf16"])
    assert_close("final_state", f64(fin), rfin, TOL["bf16"])
