"""GPU parity of the chunked forward scan (frac_scan_fwd) against the float64 oracle.

Small cases run the oracle on every output; the full-size benchmark workloads are
launched exactly as the benchmark launches them and checked on sampled
(batch, head) slices, which the oracle computes independently of the rest.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36314_amd as frac
from paper_2609_36314_amd.workloads import LAYER_FWD, LONG_PREFILL, TINY_F32, Workload
from harness import TOL, assert_close, device_inputs, f64

pytestmark = pytest.mark.gpu


def _tau(M, device="cuda"):
    t32 = oracle.default_tau(M).astype(np.float32)
    return torch.from_numpy(t32).to(device), t32.astype(np.float64)


def _run(w, inp, tau_d, chunk=0):
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state") if k in inp}
    alpha = inp["alpha"]
    return frac.scan_fwd(inp["x"], inp["dt"], inp["Bm"], inp["Cm"], alpha, tau_d, return_final_state=True,
                         chunk=chunk, **kw)


def _oracle(inp, tau64, sl=None):
    """Oracle forward on the device inputs (optionally a (b, h) slice)."""
    def g(k):
        v = inp.get(k)
        if v is None:
            return None
        return f64(v)
    x, dt, Bm, Cm = g("x"), g("dt"), g("Bm"), g("Cm")
    kw = dict(lam=g("lam"), read_logit=g("read_logit"), write_logit=g("write_logit"), D=g("D"),
              init_state=g("init_state"))
    H = x.shape[2]
    a = inp["alpha"]
    if isinstance(a, torch.Tensor) and a.dim() == 1:  # one alpha per head
        alpha = np.broadcast_to(f64(a)[None, None, :], dt.shape)
    else:
        alpha = np.broadcast_to(f64(a), dt.shape)
    if sl is not None:
        b, h = sl
        G = Bm.shape[2]
        gidx = h * G // H
        x, dt, alpha = x[b:b + 1, :, h:h + 1], dt[b:b + 1, :, h:h + 1], alpha[b:b + 1, :, h:h + 1]
        Bm, Cm = Bm[b:b + 1, :, gidx:gidx + 1], Cm[b:b + 1, :, gidx:gidx + 1]
        for k in ("lam",):
            if kw[k] is not None:
                kw[k] = kw[k][b:b + 1, :, h:h + 1]
        for k in ("read_logit", "write_logit"):
            if kw[k] is not None:
                kw[k] = kw[k][b:b + 1, :, h:h + 1]
        if kw["D"] is not None:
            kw["D"] = kw["D"][h:h + 1]
        if kw["init_state"] is not None:
            kw["init_state"] = kw["init_state"][b:b + 1, h:h + 1]
    return oracle.forward(x, dt, Bm, Cm, alpha, tau64, **kw)


def _check_state(fs_gpu, fs_ref, tol, M):
    for m in range(M):
        assert_close("final_state mode %d" % m, fs_gpu[:, :, m], fs_ref[:, :, m], tol)


SMALL = {
    "tiny-f32 (full)": TINY_F32,
    "f32 ragged groups extras": Workload("t", 2, 200, 4, 32, 32, 3, ngroups=2, io_dtype="f32", extras=True,
                                         init_state=True, final_state=True),
    "bf16 ragged": Workload("t", 2, 200, 4, 64, 128, 4, final_state=True),
    "bf16 M8": Workload("t", 1, 130, 2, 64, 128, 8, final_state=True),
    "bf16 G=H extras": Workload("t", 1, 100, 4, 64, 64, 4, ngroups=4, extras=True, init_state=True,
                                final_state=True),
    "bf16 M1 N16 P16": Workload("t", 2, 70, 3, 16, 16, 1, final_state=True),
    "bf16 M2 N32 P48": Workload("t", 1, 64, 2, 48, 32, 2, final_state=True),
    "f32 P64 N16": Workload("t", 1, 90, 2, 64, 16, 4, io_dtype="f32", final_state=True),
    "bf16 L1 init": Workload("t", 2, 1, 2, 64, 128, 4, final_state=True, init_state=True),
    "bf16 per-head alpha": LONG_PREFILL.scaled(seqlen=300, nheads=4),
    "f32 M8 N128": Workload("t", 1, 150, 2, 64, 128, 8, io_dtype="f32", final_state=True, extras=True),
    # 8 modes split P over two workgroups: a partly filled second half, an empty one
    "bf16 M8 P48 groups": Workload("t", 2, 190, 4, 48, 64, 8, ngroups=2, final_state=True, init_state=True),
    "bf16 M6 P16 N32": Workload("t", 1, 129, 2, 16, 32, 6, final_state=True, extras=True),
    # few heads and a long sequence: cut at a chunk boundary, a state-only pass to the
    # boundary state, then both parts at once
    "bf16 split M4 extras": Workload("t", 1, 700, 2, 64, 128, 4, extras=True, init_state=True, final_state=True),
    "bf16 split M8": Workload("t", 1, 520, 2, 64, 64, 8, final_state=True),
    "f32 split M2 ragged": Workload("t", 1, 777, 1, 32, 32, 2, io_dtype="f32", final_state=True, init_state=True),
    # more modes than one launch holds: blocks of eight, weights normalised over all
    # modes, outputs summed across the blocks (the paper's bank of 16, its ablation's 32)
    "bf16 M16 extras": Workload("t", 2, 200, 2, 64, 128, 16, extras=True, init_state=True, final_state=True),
    "f32 M12 N64 extras": Workload("t", 1, 150, 2, 32, 64, 12, io_dtype="f32", extras=True, init_state=True,
                                   final_state=True),
    "bf16 M32": Workload("t", 1, 130, 2, 64, 128, 32, final_state=True),
    "bf16 split M16": Workload("t", 1, 600, 2, 64, 128, 16, init_state=True, final_state=True),
    # longer sequences: up to 16 segments, a state-only pass per segment, the boundary
    # states chained, then every segment at once
    "bf16 split8 M4 extras": Workload("t", 1, 2000, 2, 64, 128, 4, extras=True, init_state=True, final_state=True),
    "f32 split6 M3 ragged": Workload("t", 1, 1500, 1, 32, 32, 3, io_dtype="f32", init_state=True, final_state=True),
    "bf16 split4 M16": Workload("t", 1, 1100, 2, 64, 128, 16, extras=True, init_state=True, final_state=True),
    # headdim above 64: groups of 64 columns (the last one partial)
    "bf16 P128 extras": Workload("t", 2, 150, 2, 128, 128, 4, extras=True, init_state=True, final_state=True),
    "f32 P96 M8": Workload("t", 1, 130, 2, 96, 64, 8, io_dtype="f32", init_state=True, final_state=True),
    "bf16 P128 M16 split": Workload("t", 1, 1300, 2, 128, 128, 16, init_state=True, final_state=True),
    # the largest sizes built: 32 modes, state 128, headdim 128 (four mode blocks x two column groups)
    "bf16 max M32 N128 P128": Workload("t", 1, 100, 2, 128, 128, 32, extras=True, init_state=True,
                                       final_state=True),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_fwd_parity_small(name):
    w = SMALL[name]
    inp = device_inputs(w, seed=1)
    tau_d, tau64 = _tau(w.nmodes)
    print("case", name, w, flush=True)
    y, fs = _run(w, inp, tau_d)
    torch.cuda.synchronize()
    yr, fsr = _oracle(inp, tau64)
    tol = TOL[w.io_dtype]
    assert_close("y", f64(y), yr, tol)
    _check_state(f64(fs), fsr, tol, w.nmodes)


@pytest.mark.parametrize("M,mode", [(4, 0), (4, 1), (4, 2), (4, 3), (16, 0), (16, 7), (16, 8), (16, 15)])
def test_fwd_mode_isolation(M, mode):
    """One-hot read/write logits (+-30) route everything through one mode, so the
    slow modes, invisible under the prior weights, are checked in y as well; with 16
    modes, the first and last mode of each block of eight."""
    w = Workload("t", 1, 200, 2, 64, 128, M, final_state=True)
    inp = device_inputs(w, seed=2)
    lg = torch.full((1, 200, 2, M), -30.0, device="cuda")
    lg[..., mode] = 30.0
    inp["read_logit"] = lg.contiguous()
    inp["write_logit"] = lg.clone()
    tau_d, tau64 = _tau(M)
    y, fs = _run(w, inp, tau_d)
    torch.cuda.synchronize()
    yr, fsr = _oracle(inp, tau64)
    assert_close("y", f64(y), yr, TOL["bf16"])
    assert_close("state of mode %d" % mode, f64(fs)[:, :, mode], fsr[:, :, mode], TOL["bf16"])


@pytest.mark.parametrize("io,M,N", [("f32", 4, 32), ("bf16", 4, 32), ("bf16", 8, 64), ("bf16", 8, 128)])
def test_fwd_large_steps_use_direct_decay(io, M, N):
    """Steps large enough that r A_Q exceeds the factorisation bound for the fast
    modes (the per-pair exponential path) and the state scale is folded back into
    the accumulators every chunk."""
    w = Workload("t", 1, 140, 2, 32, N, M, io_dtype=io, final_state=True)
    inp = device_inputs(w, seed=3)
    inp["dt"] = (inp["dt"] * 8.0).contiguous()
    tau_d, tau64 = _tau(M)
    print("case", io, M, N, flush=True)
    y, fs = _run(w, inp, tau_d)
    torch.cuda.synchronize()
    yr, fsr = _oracle(inp, tau64)
    assert_close("y", f64(y), yr, TOL[io])
    _check_state(f64(fs), fsr, TOL[io], M)


def test_fwd_chunk_split_invariance():
    """Prefill of L tokens == prefill of 128 then L-128 more from the returned state."""
    w = Workload("t", 2, 300, 4, 64, 128, 4, final_state=True)
    inp = device_inputs(w, seed=3)
    tau_d, _ = _tau(4)
    y, fs = _run(w, inp, tau_d)
    a = {k: (v[:, :128].contiguous() if k in ("x", "dt", "Bm", "Cm") else v) for k, v in inp.items()}
    b = {k: (v[:, 128:].contiguous() if k in ("x", "dt", "Bm", "Cm") else v) for k, v in inp.items()}
    y1, fs1 = _run(w, a, tau_d)
    b["init_state"] = fs1
    y2, fs2 = _run(w, b, tau_d)
    torch.cuda.synchronize()
    assert_close("y split", f64(torch.cat([y1, y2], 1)), f64(y), TOL["bf16"])
    assert_close("state split", f64(fs2), f64(fs), TOL["bf16"])


def test_fwd_deterministic():
    w = Workload("t", 2, 256, 8, 64, 128, 4, final_state=True)
    inp = device_inputs(w, seed=4)
    tau_d, _ = _tau(4)
    y1, f1 = _run(w, inp, tau_d)
    y2, f2 = _run(w, inp, tau_d)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2) and torch.equal(f1, f2)


def test_fwd_empty_sequence_returns_init_state():
    w = Workload("t", 2, 1, 2, 64, 128, 4, init_state=True)
    inp = device_inputs(w, seed=5)
    tau_d, _ = _tau(4)
    x0 = inp["x"][:, :0].contiguous()
    y, fs = frac.scan_fwd(x0, inp["dt"][:, :0].contiguous(), inp["Bm"][:, :0].contiguous(),
                          inp["Cm"][:, :0].contiguous(), 0.5, tau_d, init_state=inp["init_state"],
                          return_final_state=True)
    torch.cuda.synchronize()
    assert y.numel() == 0 and torch.equal(fs, inp["init_state"])


@pytest.mark.parametrize("w,slices", [
    (LAYER_FWD, [(0, 0), (3, 17), (7, 63)]),
    (LONG_PREFILL, [(0, 0), (0, 41), (0, 63)]),
    (LAYER_FWD.scaled(nmodes=16), [(0, 0), (7, 63)]),
])
def test_fwd_full_size_sampled(w, slices):
    """Benchmark workloads at full size, launched as the benchmark launches them;
    the oracle recomputes sampled (batch, head) slices end to end."""
    inp = device_inputs(w, seed=0)
    tau_d, tau64 = _tau(w.nmodes)
    print("full-size", w.name, flush=True)
    y, fs = _run(w, inp, tau_d)
    torch.cuda.synchronize()
    assert torch.isfinite(y.float()).all()
    for (b, h) in slices:
        yr, fsr = _oracle(inp, tau64, sl=(b, h))
        assert_close("y[%d,:,%d]" % (b, h), f64(y[b:b + 1, :, h:h + 1]), yr, TOL[w.io_dtype])
        _check_state(f64(fs[b:b + 1, h:h + 1]), fsr, TOL[w.io_dtype], w.nmodes)
