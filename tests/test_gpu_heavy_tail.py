"""A short training run of the heavy-tail probe (Sec. 4.1, Appendix E.1) through the
whole layer on the package's kernels: 400 Adam steps at length 512 must bring the
training loss well below chance (ln 2) and the accuracy on fresh length-512
sequences above 70%, and the logits at length 8192 must stay finite."""
import math

import numpy as np
import pytest
import torch

from paper_2609_36314_amd import heavy_tail as ht

pytestmark = pytest.mark.gpu


def test_short_training_learns_the_task():
    print("heavy-tail training, 400 steps", flush=True)
    model = ht.HeavyTailModel(seed=0)
    losses = ht.train(model, steps=400, batch=64, L=512, lr=3e-3, seed=0)
    assert all(math.isfinite(v) for v in losses)
    final, acc = float(np.mean(losses[-20:])), ht.evaluate(model, 512, n=256)
    print(f"final loss {final:.4f}, accuracy at 512 {acc:.3f}", flush=True)
    assert final < 0.55
    assert acc > 0.7
    with torch.no_grad():
        tok, _ = ht._batch(4, 8192, 123, "cuda")
        assert bool(torch.isfinite(model(tok)).all())
