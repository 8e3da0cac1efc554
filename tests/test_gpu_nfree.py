"""GPU parity of the paper's own layer form -- no B/C projections (dstate 1,
B = C = 1), an M x d_h state per head -- against the float64 oracle run with
B = C = 1: the forward scan (frac_scan_fwd with Bm = Cm = NULL), its backward
(frac_scan_bwd with dBm = dCm = NULL) and the decode step (frac_decode_step
with Bm = Cm = NULL)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36314_amd as frac
from paper_2609_36314_amd.workloads import PAPER_NFREE, PAPER_NFREE_TRAIN, Workload
from harness import TOL, assert_close, device_inputs, f64

pytestmark = pytest.mark.gpu


def _tau(M):
    t32 = oracle.default_tau(M).astype(np.float32)
    return torch.from_numpy(t32).cuda(), t32.astype(np.float64)


def _oracle_fwd(inp, tau64, sl=None):
    x, dt = f64(inp["x"]), f64(inp["dt"])
    g = lambda k: None if inp.get(k) is None else f64(inp[k])
    kw = dict(lam=g("lam"), read_logit=g("read_logit"), write_logit=g("write_logit"), D=g("D"),
              init_state=g("init_state"))
    a = inp["alpha"]
    alpha = np.broadcast_to(f64(a) if not isinstance(a, torch.Tensor) or a.dim() != 1 else f64(a)[None, None, :],
                            dt.shape)
    if sl is not None:
        b, h = sl
        x, dt, alpha = x[b:b + 1, :, h:h + 1], dt[b:b + 1, :, h:h + 1], alpha[b:b + 1, :, h:h + 1]
        for k in ("lam", "read_logit", "write_logit"):
            if kw[k] is not None:
                kw[k] = kw[k][b:b + 1, :, h:h + 1]
        if kw["D"] is not None:
            kw["D"] = kw["D"][h:h + 1]
        if kw["init_state"] is not None:
            kw["init_state"] = kw["init_state"][b:b + 1, h:h + 1]
    ones = np.ones(x.shape[:2] + (1, 1))
    return oracle.forward(x, dt, ones, ones, alpha, tau64, **kw)


def _run(inp, tau_d):
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state") if k in inp}
    return frac.scan_fwd(inp["x"], inp["dt"], None, None, inp["alpha"], tau_d, return_final_state=True, **kw)


SMALL = {
    "bf16 paper shape M16 P256 extras": Workload("t", 2, 300, 3, 256, 1, 16, bc=False, extras=True, init_state=True,
                                                 final_state=True),
    "f32 M4 P64": Workload("t", 1, 200, 2, 64, 1, 4, bc=False, io_dtype="f32", final_state=True),
    "bf16 M32 P128": Workload("t", 1, 130, 2, 128, 1, 32, bc=False, final_state=True, init_state=True),
    "bf16 M8 P40 ragged": Workload("t", 2, 70, 2, 40, 1, 8, bc=False, final_state=True, extras=True),
    "f32 M11 P96 extras": Workload("t", 1, 129, 2, 96, 1, 11, bc=False, io_dtype="f32", extras=True,
                                   init_state=True, final_state=True),
    "bf16 M16 L1": Workload("t", 2, 1, 2, 256, 1, 16, bc=False, final_state=True, init_state=True),
    # 128-column workgroups (head dims above 128): a half-filled second group, 4 and 32 modes, float32
    "bf16 M4 P192 ragged extras": Workload("t", 1, 201, 2, 192, 1, 4, bc=False, extras=True, init_state=True,
                                           final_state=True),
    "bf16 M32 P256": Workload("t", 1, 150, 2, 256, 1, 32, bc=False, final_state=True, init_state=True),
    "f32 M16 P256 extras": Workload("t", 1, 130, 2, 256, 1, 16, bc=False, io_dtype="f32", extras=True,
                                    final_state=True),
    # the forward whose weights run ahead of the state: one chunk, two, and a ragged
    # last group of columns (a single 16-column group with outputs)
    "bf16 M16 P256 L64 extras": Workload("t", 2, 64, 2, 256, 1, 16, bc=False, extras=True, init_state=True,
                                         final_state=True),
    "bf16 M8 P256 L65": Workload("t", 1, 65, 2, 256, 1, 8, bc=False, init_state=True, final_state=True),
    "f32 M4 P136 ragged extras": Workload("t", 1, 129, 2, 136, 1, 4, bc=False, io_dtype="f32", extras=True,
                                          init_state=True, final_state=True),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_nfree_fwd_parity(name):
    w = SMALL[name]
    inp = device_inputs(w, seed=11)
    tau_d, tau64 = _tau(w.nmodes)
    print("case", name, w, flush=True)
    y, fs = _run(inp, tau_d)
    torch.cuda.synchronize()
    yr, fsr = _oracle_fwd(inp, tau64)
    tol = TOL[w.io_dtype]
    assert_close("y", f64(y), yr, tol)
    for m in range(w.nmodes):
        assert_close("final_state mode %d" % m, f64(fs)[:, :, m], fsr[:, :, m], tol)


@pytest.mark.parametrize("P", [64, 256])
def test_nfree_large_steps_use_direct_decay(P):
    """Steps large enough that the fast modes pass the factorisation bound."""
    w = Workload("t", 1, 140, 2, P, 1, 16, bc=False, final_state=True)
    inp = device_inputs(w, seed=12)
    inp["dt"] = (inp["dt"] * 8.0).contiguous()
    tau_d, tau64 = _tau(16)
    y, fs = _run(inp, tau_d)
    torch.cuda.synchronize()
    yr, fsr = _oracle_fwd(inp, tau64)
    assert_close("y", f64(y), yr, TOL["bf16"])
    for m in range(16):
        assert_close("final_state mode %d" % m, f64(fs)[:, :, m], fsr[:, :, m], TOL["bf16"])


def test_nfree_full_size_sampled():
    """The paper-shape workload at full size; the oracle recomputes sampled (batch, head) slices."""
    w = PAPER_NFREE
    inp = device_inputs(w, seed=0)
    tau_d, tau64 = _tau(w.nmodes)
    print("full-size", w.name, flush=True)
    y = frac.scan_fwd(inp["x"], inp["dt"], None, None, inp["alpha"], tau_d)
    torch.cuda.synchronize()
    assert torch.isfinite(y.float()).all()
    for (b, h) in [(0, 0), (7, 15), (3, 9)]:
        yr, _ = _oracle_fwd(inp, tau64, sl=(b, h))
        assert_close("y[%d,:,%d]" % (b, h), f64(y[b:b + 1, :, h:h + 1]), yr, TOL["bf16"])


def test_nfree_decode_matches_oracle_steps():
    """Decode steps without B/C from a random state equal the oracle's recurrence."""
    w = Workload("t", 2, 1, 3, 256, 1, 16, bc=False, decode_steps=4, init_state=True, extras=True)
    a = device_inputs(w, seed=13)
    tau_d, tau64 = _tau(16)
    state = a["init_state"].clone()
    ref = f64(state)
    alpha = a["alpha"]  # [S, B, H] per step with extras
    for s in range(w.decode_steps):
        y = frac.decode_step(state, a["x"][s].contiguous(), a["dt"][s].contiguous(), None, None,
                             alpha[s].contiguous(), tau_d, lam=a["lam"][s].contiguous(),
                             read_logit=a["read_logit"][s].contiguous(), write_logit=a["write_logit"][s].contiguous(),
                             D=a["D"])
        torch.cuda.synchronize()
        ones = np.ones((w.batch, 1, 1))
        yr, ref = oracle.decode_step(ref, f64(a["x"][s]), f64(a["dt"][s]), ones, ones, f64(alpha[s]), tau64,
                                     lam=f64(a["lam"][s]), read_logit=f64(a["read_logit"][s]),
                                     write_logit=f64(a["write_logit"][s]), D=f64(a["D"]))
        assert_close("decode y step %d" % s, f64(y), yr, TOL["bf16"])
        assert_close("decode state step %d" % s, f64(state), ref, TOL["bf16"])


def _oracle_bwd(inp, tau64, dfs=None):
    x, dt, dy = f64(inp["x"]), f64(inp["dt"]), f64(inp["dy"])
    a = inp["alpha"]
    alpha = np.broadcast_to(f64(a) if not isinstance(a, torch.Tensor) or a.dim() != 1 else f64(a)[None, None, :],
                            dt.shape)
    kw = {k: f64(inp[k]) for k in ("lam", "read_logit", "write_logit", "D", "init_state") if k in inp}
    ones = np.ones(x.shape[:2] + (1, 1))
    return oracle.backward(x, dt, ones, ones, alpha, tau64, dy, d_final_state=None if dfs is None else f64(dfs), **kw)


BWD = {
    "bf16 paper shape M16 P256 extras dfinal": Workload("t", 2, 300, 2, 256, 1, 16, bc=False, extras=True,
                                                        init_state=True, backward=True, final_state=True),
    "f32 M4 P64": Workload("t", 1, 200, 2, 64, 1, 4, bc=False, io_dtype="f32", backward=True),
    "bf16 M32 P128 init": Workload("t", 1, 130, 2, 128, 1, 32, bc=False, backward=True, init_state=True),
    "bf16 M8 P40 ragged extras": Workload("t", 2, 70, 2, 40, 1, 8, bc=False, backward=True, extras=True),
    "f32 M11 P96 extras dfinal": Workload("t", 1, 129, 2, 96, 1, 11, bc=False, io_dtype="f32", extras=True,
                                          init_state=True, backward=True, final_state=True),
    "bf16 M16 L1": Workload("t", 2, 1, 2, 256, 1, 16, bc=False, backward=True, init_state=True, final_state=True),
    # 128-column workgroups (head dims above 128): a half-filled second group, 4 and 32 modes, float32
    # (with 32 modes the float32 backward keeps 64-column workgroups)
    "bf16 M4 P192 ragged extras dfinal": Workload("t", 1, 201, 2, 192, 1, 4, bc=False, extras=True,
                                                  init_state=True, backward=True, final_state=True),
    "bf16 M32 P256 init": Workload("t", 1, 150, 2, 256, 1, 32, bc=False, backward=True, init_state=True),
    "f32 M16 P256 extras": Workload("t", 1, 130, 2, 256, 1, 16, bc=False, io_dtype="f32", extras=True,
                                    backward=True),
    "f32 M32 P256 extras": Workload("t", 1, 90, 2, 256, 1, 32, bc=False, io_dtype="f32", extras=True,
                                    backward=True),
}


@pytest.mark.parametrize("name", list(BWD))
def test_nfree_bwd_parity(name):
    w = BWD[name]
    inp = device_inputs(w, seed=15)
    tau_d, tau64 = _tau(w.nmodes)
    dfs = inp.get("d_final_state")
    print("case", name, w, flush=True)
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state") if k in inp}
    g = frac.scan_bwd(inp["x"], inp["dt"], None, None, inp["alpha"], tau_d, inp["dy"], d_final_state=dfs,
                      all_grads=True, **kw)
    torch.cuda.synchronize()
    ref = _oracle_bwd(inp, tau64, dfs)
    tol = TOL[w.io_dtype]
    assert g["dBm"] is None and g["dCm"] is None
    assert_close("dx", f64(g["dx"]), ref["dx"], tol)
    assert_close("ddt", f64(g["ddt"]), ref["ddt"], tol)
    if "D" in inp:
        assert_close("dD", f64(g["dD"]), ref["dD"], tol)
    _check_further_grads(g, ref, tol, "lam" in inp)


def _check_further_grads(g, ref, tol, has_lambda):
    """Gradients of alpha, lambda, the logits (the oracle's, also at zero logits) and
    the initial state."""
    assert_close("dalpha", f64(g["dalpha"]), ref["dalpha"], tol)
    if has_lambda:
        assert_close("dlambda", f64(g["dlambda"]), ref["dlambda"], tol)
    else:
        assert not g["dlambda"].any()
    assert_close("dread_logit", f64(g["dread_logit"]), ref["dread_logit"], tol)
    assert_close("dwrite_logit", f64(g["dwrite_logit"]), ref["dwrite_logit"], tol)
    for m in range(ref["dinit_state"].shape[2]):
        assert_close("dinit_state mode %d" % m, f64(g["dinit_state"])[:, :, m], ref["dinit_state"][:, :, m], tol)


def test_nfree_bwd_large_steps_use_direct_decay():
    w = Workload("t", 1, 140, 2, 64, 1, 16, bc=False, backward=True)
    inp = device_inputs(w, seed=16)
    inp["dt"] = (inp["dt"] * 8.0).contiguous()
    tau_d, tau64 = _tau(16)
    g = frac.scan_bwd(inp["x"], inp["dt"], None, None, inp["alpha"], tau_d, inp["dy"], all_grads=True)
    torch.cuda.synchronize()
    ref = _oracle_bwd(inp, tau64)
    assert_close("dx", f64(g["dx"]), ref["dx"], TOL["bf16"])
    assert_close("ddt", f64(g["ddt"]), ref["ddt"], TOL["bf16"])
    _check_further_grads(g, ref, TOL["bf16"], False)


def test_nfree_bwd_all_grads_leave_the_other_outputs_unchanged():
    """Asking for the further gradients takes another kernel variant: dx, ddt and dD
    must not change bit for bit."""
    w = Workload("t", 1, 150, 2, 128, 1, 16, bc=False, backward=True, extras=True)
    inp = device_inputs(w, seed=18)
    tau_d, _ = _tau(16)
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D") if k in inp}
    g1 = frac.scan_bwd(inp["x"], inp["dt"], None, None, inp["alpha"], tau_d, inp["dy"], **kw)
    g2 = frac.scan_bwd(inp["x"], inp["dt"], None, None, inp["alpha"], tau_d, inp["dy"], all_grads=True, **kw)
    torch.cuda.synchronize()
    for k in ("dx", "ddt", "dD"):
        assert torch.equal(g1[k], g2[k]), k


def test_nfree_bwd_deterministic():
    w = Workload("t", 2, 192, 2, 256, 1, 16, bc=False, backward=True)
    inp = device_inputs(w, seed=17)
    tau_d, _ = _tau(16)
    g1 = frac.scan_bwd(inp["x"], inp["dt"], None, None, inp["alpha"], tau_d, inp["dy"])
    g2 = frac.scan_bwd(inp["x"], inp["dt"], None, None, inp["alpha"], tau_d, inp["dy"])
    torch.cuda.synchronize()
    assert torch.equal(g1["dx"], g2["dx"]) and torch.equal(g1["ddt"], g2["ddt"])


def test_nfree_bwd_shared_logits_all_grads():
    """One tensor passed as both read and write logits (the write weights then equal
    the read weights); both logit gradients still match the oracle's."""
    w = Workload("t", 1, 100, 2, 64, 1, 8, bc=False, backward=True, extras=True)
    inp = device_inputs(w, seed=19)
    inp["write_logit"] = inp["read_logit"]
    tau_d, tau64 = _tau(8)
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D") if k in inp}
    g = frac.scan_bwd(inp["x"], inp["dt"], None, None, inp["alpha"], tau_d, inp["dy"], all_grads=True, **kw)
    torch.cuda.synchronize()
    ref = _oracle_bwd(inp, tau64)
    tol = TOL["bf16"]
    for k in ("dx", "ddt", "dalpha", "dlambda", "dread_logit", "dwrite_logit"):
        assert_close(k, f64(g[k]), ref[k], tol)


def test_nfree_bwd_full_size_all_grads_sampled():
    """The paper-shape training workload at full size (batch 8, L 2048, 16 heads of
    256, 16 modes), with lambda, both logits, D, an initial state and a final-state
    gradient drawn over the paper's ranges, all gradients: every gradient of sampled
    (batch, head) slices, the first and the last, recomputed by the oracle; dD of the
    sampled heads over all batch elements."""
    w = PAPER_NFREE_TRAIN.scaled(extras=True, init_state=True, final_state=True)
    inp = device_inputs(w, seed=20)
    tau_d, tau64 = _tau(w.nmodes)
    dfs = inp["d_final_state"]
    print("full-size", w.name, "all gradients", flush=True)
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state")}
    g = frac.scan_bwd(inp["x"], inp["dt"], None, None, inp["alpha"], tau_d, inp["dy"], d_final_state=dfs,
                      all_grads=True, **kw)
    torch.cuda.synchronize()
    tol = TOL["bf16"]
    for (b, h) in [(0, 0), (3, 9), (7, 15)]:
        sl = {k: inp[k][b:b + 1, :, h:h + 1] for k in ("x", "dt", "dy", "alpha", "lam", "read_logit", "write_logit")}
        sl["D"] = inp["D"][h:h + 1]
        sl["init_state"] = inp["init_state"][b:b + 1, h:h + 1]
        ref = _oracle_bwd(sl, tau64, dfs[b:b + 1, h:h + 1])
        sg = {k: g[k][b:b + 1, :, h:h + 1] for k in ("dx", "ddt", "dalpha", "dlambda", "dread_logit", "dwrite_logit")}
        sg["dinit_state"] = g["dinit_state"][b:b + 1, h:h + 1]
        print("slice", b, h, flush=True)
        assert_close("dx", f64(sg["dx"]), ref["dx"], tol)
        assert_close("ddt", f64(sg["ddt"]), ref["ddt"], tol)
        _check_further_grads(sg, ref, tol, True)
    for h in (0, 15):
        sl = {k: inp[k][:, :, h:h + 1] for k in ("x", "dt", "dy", "alpha", "lam", "read_logit", "write_logit")}
        sl["D"] = inp["D"][h:h + 1]
        sl["init_state"] = inp["init_state"][:, h:h + 1]
        ref = _oracle_bwd(sl, tau64, dfs[:, h:h + 1])
        assert_close("dD[%d]" % h, f64(g["dD"][h:h + 1]), ref["dD"], tol)


def test_nfree_custom_tau_bank():
    """The paper's form with an unsorted bank of the caller's own timescales, modes faster
    than one step among them: forward, final state and every gradient."""
    M = 8
    w = Workload("t", 1, 150, 2, 128, 1, M, bc=False, extras=True, init_state=True, backward=True, final_state=True)
    inp = device_inputs(w, seed=22)
    t32 = np.array([2.0, 0.3, 9000.0, 50.0, 0.8, 131072.0, 7.0, 1.0], dtype=np.float32)
    tau_d, tau64 = torch.from_numpy(t32).cuda(), t32.astype(np.float64)
    dfs = inp["d_final_state"]
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state")}
    y, fin = frac.scan_fwd(inp["x"], inp["dt"], None, None, inp["alpha"], tau_d, return_final_state=True, **kw)
    g = frac.scan_bwd(inp["x"], inp["dt"], None, None, inp["alpha"], tau_d, inp["dy"], d_final_state=dfs,
                      all_grads=True, **kw)
    torch.cuda.synchronize()
    yr, fr = _oracle_fwd(inp, tau64)
    ref = _oracle_bwd(inp, tau64, dfs)
    tol = TOL["bf16"]
    assert_close("y", f64(y), yr, tol)
    assert_close("final_state", f64(fin), fr, tol)
    assert_close("dx", f64(g["dx"]), ref["dx"], tol)
    assert_close("ddt", f64(g["ddt"]), ref["ddt"], tol)
    assert_close("dD", f64(g["dD"]), ref["dD"], tol)
    _check_further_grads(g, ref, tol, True)


@pytest.mark.parametrize("P,M,io", [(256, 16, "bf16"), (192, 8, "bf16"), (64, 4, "f32"), (256, 16, "f32")])
def test_chunk_states_from_the_forward_feed_the_backward(P, M, io):
    """The chunk states the forward keeps: slot 0 is the initial state, slot k the state
    after the first 64 k tokens (against the oracle's final state on that prefix), the last
    slot the final state; y and final_state are those of a forward that keeps none, and the
    backward that reads them returns the gradients of the one that recomputes them."""
    L = 200
    w = Workload("t", 2, L, 2, P, 1, M, bc=False, io_dtype=io, extras=True, init_state=True, backward=True,
                 final_state=True)
    inp = device_inputs(w, seed=23)
    tau_d, tau64 = _tau(M)
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state")}
    args = (inp["x"], inp["dt"], None, None, inp["alpha"], tau_d)
    print("chunk states", P, M, io, flush=True)
    y0, f0 = frac.scan_fwd(*args, return_final_state=True, **kw)
    cs = frac.chunk_states_like(inp["x"], M)
    y1, f1 = frac.scan_fwd(*args, return_final_state=True, chunk_states=cs, **kw)
    g0 = frac.scan_bwd(*args, inp["dy"], d_final_state=inp.get("d_final_state"), all_grads=True, **kw)
    g1 = frac.scan_bwd(*args, inp["dy"], d_final_state=inp.get("d_final_state"), all_grads=True, chunk_states=cs, **kw)
    torch.cuda.synchronize()
    assert torch.equal(y0, y1) and torch.equal(f0, f1)
    nch = (L + 63) // 64
    slots = cs.view(2, 2, nch + 1, M, P)
    assert torch.equal(slots[:, :, nch], f1[:, :, :, 0, :])
    assert torch.equal(slots[:, :, 0], inp["init_state"][:, :, :, 0, :])
    for k in (1, 3):
        pre = {key: (v[:, :64 * k].contiguous() if isinstance(v, torch.Tensor) and v.dim() >= 2 and v.shape[1] == L
                     else v) for key, v in inp.items()}
        _, ref = _oracle_fwd(pre, tau64)
        assert_close("chunk state %d" % k, f64(slots[:, :, k]), ref[:, :, :, 0, :], TOL[io])
    # the kept states come from the forward kernel, the recomputed ones from the
    # checkpoint pass: float32 states may differ in their last bit, which the telescoping
    # step-size sums carry into dlambda and dalpha at about 1e-6 of their largest value
    bound = 1e-5 if io == "f32" else 1e-6
    for name, v in g0.items():
        if v is None:
            continue
        ref, got = f64(v), f64(g1[name])
        scale = max(float(np.abs(ref).max()), 1e-30)
        assert float(np.abs(got - ref).max()) <= bound * scale, name


@pytest.mark.parametrize("L", [0, 1, 64, 65])
def test_chunk_states_at_chunk_boundaries(L):
    """Sequences of no token, one token, exactly one chunk and one token past it: the kept
    states hold ceil(L / 64) + 1 slots, the first the initial state and the last the final
    state, and a backward that reads them matches one that recomputes them."""
    w = Workload("t", 1, L, 2, 256, 1, 16, bc=False, extras=True, init_state=True, backward=True, final_state=True)
    inp = device_inputs(w, seed=24)
    tau_d, _ = _tau(16)
    kw = {k: inp[k] for k in ("lam", "read_logit", "write_logit", "D", "init_state")}
    args = (inp["x"], inp["dt"], None, None, inp["alpha"], tau_d)
    print("chunk states L", L, flush=True)
    cs = frac.chunk_states_like(inp["x"], 16)
    nch = (L + 63) // 64
    assert cs.numel() == 1 * 2 * (nch + 1) * 16 * 256
    _, fin = frac.scan_fwd(*args, return_final_state=True, chunk_states=cs, **kw)
    torch.cuda.synchronize()
    slots = cs.view(1, 2, nch + 1, 16, 256)
    assert torch.equal(slots[:, :, 0], inp["init_state"][:, :, :, 0, :])
    assert torch.equal(slots[:, :, nch], fin[:, :, :, 0, :])
    if L == 0:
        return
    g0 = frac.scan_bwd(*args, inp["dy"], d_final_state=inp.get("d_final_state"), all_grads=True, **kw)
    g1 = frac.scan_bwd(*args, inp["dy"], d_final_state=inp.get("d_final_state"), all_grads=True, chunk_states=cs,
                       **kw)
    torch.cuda.synchronize()
    for name, v in g0.items():
        if v is None:
            continue
        ref, got = f64(v), f64(g1[name])
        scale = max(float(np.abs(ref).max()), 1e-30)
        assert float(np.abs(got - ref).max()) <= 1e-6 * scale, name
