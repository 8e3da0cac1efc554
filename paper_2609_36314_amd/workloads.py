"""Seeded synthetic inputs for the Frac scan, shared by the tests and the benchmark.

Distributions only -- none of the scan's arithmetic lives here.  Every workload
draws float32 values from numpy.random.default_rng(seed) in a fixed order:
x, B, C, z (for dt), then alpha (per-head configs), dy (training), the initial
state (decode), and for decode the per-step tokens step by step.

  x ~ N(0, 1);  B, C ~ N(0, 1/N);  dt = softplus(z - 2), z ~ N(0, 1) (not clipped)
  alpha: a constant, or one value per head drawn from U[lo, hi]
  tau: the paper's geometric bank on [1, 2^17] (built by the library, not here)
  lambda, read/write logits and D are absent unless a test asks for them (then
  lambda ~ U[0.25, 4], alpha ~ U[0.02, 1] per token, logits and D ~ N(0, 1)).
  Without B/C projections (bc False, dstate 1): B = C = 1, nothing drawn for them.

The named workloads are the five benchmark configurations of the Frac layer at
the 1.3B-model layer shape (H = 64 heads, head dim 64, state 128, one B/C group),
and the paper's own layer form (no B/C, 16 heads of 256, 16 modes).
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional, Tuple

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    seqlen: int
    nheads: int
    headdim: int
    dstate: int
    nmodes: int
    ngroups: int = 1
    io_dtype: str = "bf16"            # "bf16" or "f32"
    alpha: float = 0.5                 # used when alpha_range is None
    alpha_range: Optional[Tuple[float, float]] = None   # per-head U[lo, hi]
    chunk: int = 64
    backward: bool = False
    final_state: bool = False
    decode_steps: int = 0              # > 0: decode workload (seqlen is 1 per step)
    init_state: bool = False
    extras: bool = False               # also draw lambda, logits and D (tests only)
    bc: bool = True                    # False: the form without B/C (dstate 1, B = C = 1)

    def scaled(self, **kw) -> "Workload":
        return replace(self, **kw)


TINY_F32 = Workload("tiny-f32", 1, 256, 2, 16, 16, 4, io_dtype="f32")
LAYER_FWD = Workload("layer-fwd-b8-l2048", 8, 2048, 64, 64, 128, 4)
LONG_PREFILL = Workload("prefill-b1-l16384", 1, 16384, 64, 64, 128, 4, alpha_range=(0.3, 0.8), final_state=True)
TRAIN = Workload("train-b4-l4096-m8", 4, 4096, 64, 64, 128, 8, backward=True)
# the same step with the paper's bank of 16 modes (two blocks of eight)
TRAIN_M16 = Workload("train-b4-l4096-m16", 4, 4096, 64, 64, 128, 16, backward=True)
DECODE = Workload("decode-b256-128steps", 256, 1, 64, 64, 128, 4, decode_steps=128, init_state=True)
# the paper's layer (state H x M x d_h, no B/C), forward at batch 8 x 2048 tokens
PAPER_NFREE = Workload("paper-nfree-b8-l2048", 8, 2048, 16, 256, 1, 16, bc=False)
PAPER_NFREE_TRAIN = Workload("paper-nfree-train-b8-l2048", 8, 2048, 16, 256, 1, 16, bc=False, backward=True)
# decode of the paper's form: 2048 sequences, a 537 MB float32 state (larger than the on-chip caches)
PAPER_NFREE_DECODE = Workload("paper-nfree-decode-b2048-128steps", 2048, 1, 16, 256, 1, 16, bc=False,
                              decode_steps=128, init_state=True)

WORKLOADS = {w.name: w for w in (TINY_F32, LAYER_FWD, LONG_PREFILL, TRAIN, TRAIN_M16, DECODE, PAPER_NFREE,
                                  PAPER_NFREE_TRAIN, PAPER_NFREE_DECODE)}


def _softplus(v: np.ndarray) -> np.ndarray:
    return np.logaddexp(0.0, v).astype(np.float32)


def generate(w: Workload, seed: int = 0) -> dict:
    """float32 numpy arrays for workload `w` (dt already passed through softplus)."""
    rng = np.random.default_rng(seed)
    Bsz, H, P, N, G, M = w.batch, w.nheads, w.headdim, w.dstate, w.ngroups, w.nmodes
    f32 = np.float32
    out = {}
    if w.decode_steps:
        S = w.decode_steps
        out["x"] = rng.standard_normal((S, Bsz, H, P), dtype=f32)
        if w.bc:
            out["Bm"] = (rng.standard_normal((S, Bsz, G, N), dtype=f32) / np.sqrt(N)).astype(f32)
            out["Cm"] = (rng.standard_normal((S, Bsz, G, N), dtype=f32) / np.sqrt(N)).astype(f32)
        out["dt"] = _softplus(rng.standard_normal((S, Bsz, H), dtype=f32) - 2.0)
    else:
        L = w.seqlen
        out["x"] = rng.standard_normal((Bsz, L, H, P), dtype=f32)
        if w.bc:
            out["Bm"] = (rng.standard_normal((Bsz, L, G, N), dtype=f32) / np.sqrt(N)).astype(f32)
            out["Cm"] = (rng.standard_normal((Bsz, L, G, N), dtype=f32) / np.sqrt(N)).astype(f32)
        out["dt"] = _softplus(rng.standard_normal((Bsz, L, H), dtype=f32) - 2.0)
    if w.alpha_range is not None:
        out["alpha"] = rng.uniform(w.alpha_range[0], w.alpha_range[1], H).astype(f32)
    else:
        out["alpha"] = f32(w.alpha)
    if w.backward:
        out["dy"] = rng.standard_normal(out["x"].shape, dtype=f32)
        if w.final_state:
            out["d_final_state"] = rng.standard_normal((Bsz, H, M, N, P), dtype=f32)
    if w.init_state:
        out["init_state"] = rng.standard_normal((Bsz, H, M, N, P), dtype=f32)
    if w.extras:
        lead = out["dt"].shape
        # the paper's ranges: lambda clipped to [0.25, 4], alpha = sigmoid(.) in (0, 1)
        # (here down to 0.02, where lambda^{1/alpha} reaches 2^100)
        out["lam"] = rng.uniform(0.25, 4.0, lead).astype(f32)
        out["read_logit"] = rng.standard_normal(lead + (M,), dtype=f32)
        out["write_logit"] = rng.standard_normal(lead + (M,), dtype=f32)
        out["D"] = rng.standard_normal(H, dtype=f32)
        out["alpha"] = rng.uniform(0.02, 1.0, lead).astype(f32)
    return out
