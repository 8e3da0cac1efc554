"""Pins of the gated normalization oracle (oracle/gnorm.py): the output of each group
has root-mean-square 1 before the weight (up to eps); scale invariance in x; the gate
is SiLU (z = 0 zeroes the output, large z passes x through); finite differences."""
import numpy as np

from oracle import gnorm as og


def test_unit_rms_per_group_and_scale_invariance():
    rng = np.random.default_rng(0)
    x, z = rng.normal(size=(2, 5, 12)), rng.normal(size=(2, 5, 12))
    y = og.gnorm_forward(x, z, np.ones(12), group=4, eps=0.0)
    rms = np.sqrt(np.mean(y.reshape(2, 5, 3, 4) ** 2, axis=-1))
    assert np.allclose(rms, 1.0, rtol=1e-13)
    assert np.allclose(og.gnorm_forward(7.5 * x, z, np.ones(12), 4, eps=0.0), y, rtol=1e-12)


def test_gate_is_silu():
    rng = np.random.default_rng(1)
    x = rng.normal(size=(1, 3, 8))
    w = rng.normal(size=8)
    assert np.all(og.gnorm_forward(x, np.zeros_like(x), w, 8) == 0.0)
    big = og.gnorm_forward(x, np.full_like(x, 60.0), w, 8, eps=0.0)
    ref = x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) * w
    assert np.allclose(big, ref, rtol=1e-12)


def test_gradients_match_finite_differences():
    rng = np.random.default_rng(2)
    B, L, C, grp = 2, 3, 8, 4
    x, z, w, dy = rng.normal(size=(B, L, C)), rng.normal(size=(B, L, C)), rng.normal(size=C), rng.normal(size=(B, L, C))
    g = og.gnorm_backward(x, z, w, dy, grp)
    loss = lambda x, z, w: float(np.sum(og.gnorm_forward(x, z, w, grp) * dy))
    h = 1e-6
    for name, arr, mk in (("dx", x, lambda a: (a, z, w)), ("dz", z, lambda a: (x, a, w)),
                          ("dweight", w, lambda a: (x, z, a))):
        fd = np.zeros(arr.shape)
        for i in np.ndindex(*arr.shape):
            up, dn = arr.copy(), arr.copy()
            up[i] += h
            dn[i] -= h
            fd[i] = (loss(*mk(up)) - loss(*mk(dn))) / (2 * h)
        assert np.allclose(g[name], fd, rtol=1e-6, atol=1e-8), name
