"""The forward that allocates nothing (frac_scan_fwd_noalloc) inside a captured graph:
replayed several times, with new inputs written eagerly and the device synchronized
between replays, every replay gives the bits of the same call made eagerly."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36314_amd as frac
from paper_2609_36314_amd.workloads import Workload
from harness import device_inputs

pytestmark = pytest.mark.gpu

CASES = {
    # two sequence segments: the state-only pass, the boundary states and the output pass
    "bc split": Workload("t", 1, 700, 4, 64, 128, 4, extras=True, init_state=True, final_state=True),
    "paper": Workload("t", 2, 300, 2, 256, 1, 16, bc=False, extras=True, init_state=True, final_state=True),
}


@pytest.mark.parametrize("name", list(CASES))
def test_noalloc_forward_replays_in_a_graph(name):
    w = CASES[name]
    inp = device_inputs(w, seed=41)
    tau = torch.from_numpy(oracle.default_tau(w.nmodes).astype(np.float32)).cuda()
    x = inp["x"].clone()
    Bm, Cm = inp.get("Bm"), inp.get("Cm")
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state")}
    st = inp["init_state"]
    y_g, fin_g = torch.empty_like(x), torch.empty_like(st)
    y_e, fin_e = torch.empty_like(x), torch.empty_like(st)

    def call(y, fin):
        frac.scan_fwd_noalloc(x, inp["dt"], Bm, Cm, inp["alpha"], tau, y=y, final_state=fin, **kw)

    print("graph", name, flush=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # first call outside the capture: the scratch address is looked up
        call(y_g, fin_g)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(y_g, fin_g)
    gen = torch.Generator(device="cpu").manual_seed(5)
    for rep in range(3):
        x.copy_(torch.randn(x.shape, generator=gen).to(x.dtype))  # eager work between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        call(y_e, fin_e)
        torch.cuda.synchronize()
        assert torch.equal(y_g, y_e), rep
        assert torch.equal(fin_g, fin_e), rep
        assert torch.isfinite(y_e.float()).all()


@pytest.mark.parametrize("name", list(CASES))
def test_backward_with_a_caller_workspace_replays_in_a_graph(name):
    """The backward with every gradient, its workspace and outputs allocated before the
    capture: each replay gives the bits of an eager call on the same inputs."""
    w = CASES[name].scaled(backward=True)
    inp = device_inputs(w, seed=42)
    tau = torch.from_numpy(oracle.default_tau(w.nmodes).astype(np.float32)).cuda()
    dy = inp["dy"].clone()
    Bm, Cm = inp.get("Bm"), inp.get("Cm")
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state")}
    shape = frac._shape(inp["x"], Bm, w.nmodes, 0)
    ws = torch.empty(max(1, frac.scan_workspace_size(shape, True)), dtype=torch.uint8, device="cuda")

    def call():
        return frac.scan_bwd(inp["x"], inp["dt"], Bm, Cm, inp["alpha"], tau, dy, all_grads=True, workspace=ws,
                             d_final_state=inp.get("d_final_state"), **kw)

    print("graph bwd", name, flush=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out_g = call()
    gen = torch.Generator(device="cpu").manual_seed(6)
    for rep in range(3):
        dy.copy_(torch.randn(dy.shape, generator=gen).to(dy.dtype))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        out_e = call()
        torch.cuda.synchronize()
        for k, v in out_e.items():
            if v is not None:
                assert torch.equal(out_g[k], v), (rep, k)
