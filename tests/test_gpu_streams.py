"""The library runs on the caller's stream: results on a second stream, and from two
host threads on two streams at once, are the bits of the same calls on the default
stream (every reduction is in a fixed order)."""
import threading

import numpy as np
import pytest
import torch

import oracle
import paper_2609_36314_amd as frac
from paper_2609_36314_amd.workloads import Workload
from harness import device_inputs

pytestmark = pytest.mark.gpu

CASES = {
    "bc": Workload("t", 2, 300, 4, 64, 128, 8, extras=True, init_state=True, backward=True, final_state=True),
    "paper": Workload("t", 2, 300, 2, 256, 1, 16, bc=False, extras=True, init_state=True, backward=True,
                      final_state=True),
}


def _calls(w, inp):
    """Forward, backward with every gradient and one decode step on the final state."""
    tau = torch.from_numpy(oracle.default_tau(w.nmodes).astype(np.float32)).cuda()
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state")}
    Bm, Cm = inp.get("Bm"), inp.get("Cm")
    y, fin = frac.scan_fwd(inp["x"], inp["dt"], Bm, Cm, inp["alpha"], tau, return_final_state=True, **kw)
    g = frac.scan_bwd(inp["x"], inp["dt"], Bm, Cm, inp["alpha"], tau, inp["dy"],
                      d_final_state=inp.get("d_final_state"), all_grads=True, **kw)
    st = fin.clone()
    x1 = inp["x"][:, -1].contiguous()
    dt1 = inp["dt"][:, -1].contiguous()
    al1 = inp["alpha"][:, -1].contiguous()
    B1 = None if Bm is None else Bm[:, -1].contiguous()
    C1 = None if Cm is None else Cm[:, -1].contiguous()
    y1 = frac.decode_step(st, x1, dt1, B1, C1, al1, tau)
    out = {"y": y, "final_state": fin, "state": st, "y1": y1}
    out.update({k: v for k, v in g.items() if v is not None})
    return out


def _same(a, b):
    assert a.keys() == b.keys()
    for k in a:
        assert torch.equal(a[k], b[k]), k


@pytest.mark.parametrize("name", list(CASES))
def test_a_second_stream_gives_the_default_streams_bits(name):
    w = CASES[name]
    inp = device_inputs(w, seed=31)
    print("stream", name, flush=True)
    ref = _calls(w, inp)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()  # default priority
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        got = _calls(w, inp)
    s.synchronize()
    _same(ref, got)


def test_two_host_threads_on_two_streams():
    """Both forms at once from two threads, each on its own stream and workspaces."""
    inps = {n: device_inputs(w, seed=32) for n, w in CASES.items()}
    ref = {n: _calls(CASES[n], inps[n]) for n in CASES}
    torch.cuda.synchronize()
    got, errors = {}, []
    streams = {n: torch.cuda.Stream() for n in CASES}
    for s in streams.values():
        s.wait_stream(torch.cuda.current_stream())

    def work(n):
        try:
            with torch.cuda.stream(streams[n]):
                for _ in range(3):
                    got[n] = _calls(CASES[n], inps[n])
            streams[n].synchronize()
        except Exception as e:  # surfaced below
            errors.append(e)

    ts = [threading.Thread(target=work, args=(n,)) for n in CASES]
    for t in ts:
        t.start()
    for t in ts:
        t.join(timeout=120)
    assert not errors, errors
    for n in CASES:
        _same(ref[n], got[n])
