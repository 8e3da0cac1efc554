"""Shared helpers of the GPU parity tests: seeded inputs on the device, the exact
(rounded) values handed to the oracle, and the error metrics."""
from __future__ import annotations

import numpy as np
import torch

from paper_2609_36314_amd.workloads import Workload, generate

# relative L2 error bound per io dtype (float32 end to end; bfloat16 inputs with float32 accumulation)
TOL = {"f32": 1e-4, "bf16": 2e-2}


def io_torch_dtype(w: Workload):
    return torch.bfloat16 if w.io_dtype == "bf16" else torch.float32


def device_inputs(w: Workload, seed: int = 0, device="cuda") -> dict:
    """Seeded inputs on the device: x, Bm, Cm, dy in the io dtype, the rest float32."""
    a = generate(w, seed)
    io = io_torch_dtype(w)
    out = {}
    for k, v in a.items():
        t = torch.as_tensor(np.asarray(v))
        if k in ("x", "Bm", "Cm", "dy"):
            t = t.to(io)
        out[k] = t.to(device).contiguous() if t.dim() else t.item()
    return out


def f64(t) -> np.ndarray:
    """The exact values a device tensor holds, as float64 on the host."""
    if isinstance(t, (float, int)):
        return np.float64(t)
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel_l2(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref.ravel())
    num = np.linalg.norm((got - ref).ravel())
    return float(num / den) if den > 0 else float(num)


def max_rel(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.abs(ref).max()
    return float(np.abs(got - ref).max() / den) if den > 0 else float(np.abs(got - ref).max())


def assert_close(name, got, ref, tol):
    """Relative L2 error within tol, and the largest element error relative to the
    largest reference magnitude within 2 tol (an error confined to a few elements, one
    head or one chunk fails the second)."""
    e = rel_l2(got, ref)
    mr = max_rel(got, ref)
    assert np.all(np.isfinite(np.asarray(got, np.float64))), "%s: non-finite values" % name
    assert e <= tol, "%s: relative L2 error %.3e > %.1e (max-rel %.3e)" % (name, e, tol, mr)
    assert mr <= 2 * tol, "%s: max|err| / max|ref| = %.3e > %.1e (relative L2 %.3e)" % (name, mr, 2 * tol, e)
    print("  %-24s rel-L2 %.2e  max-rel %.2e" % (name, e, mr), flush=True)
    return e
