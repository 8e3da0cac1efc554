"""Pins of the causal depthwise convolution oracle (oracle/conv.py): each channel is
an FIR filter, so without the activation it equals scipy.signal.lfilter with the
reversed taps; causality (an output never depends on later tokens); the impulse
response is the taps; SiLU closed forms; finite differences for every gradient."""
import numpy as np
from scipy.signal import lfilter

from oracle import conv as oc


def test_each_channel_is_an_fir_filter():
    rng = np.random.default_rng(0)
    x, w, b = rng.normal(size=(2, 40, 5)), rng.normal(size=(5, 4)), rng.normal(size=5)
    y = oc.conv_forward(x, w, b, activation=False)
    for bb in range(2):
        for c in range(5):
            ref = lfilter(w[c, ::-1], [1.0], x[bb, :, c]) + b[c]
            assert np.allclose(y[bb, :, c], ref, rtol=1e-13, atol=1e-13)


def test_causal_and_impulse_response():
    rng = np.random.default_rng(1)
    w = rng.normal(size=(3, 4))
    x = np.zeros((1, 10, 3))
    x[0, 2, :] = 1.0
    y = oc.conv_forward(x, w, activation=False)
    assert np.all(y[0, :2] == 0.0)
    for k in range(4):  # the token k steps after the impulse sees tap K-1-k
        assert np.array_equal(y[0, 2 + k], w[:, 3 - k])
    assert np.all(y[0, 6:] == 0.0)
    x2 = rng.normal(size=(1, 10, 3))
    x3 = x2.copy()
    x3[0, 7:] += 5.0
    assert np.array_equal(oc.conv_forward(x2, w)[0, :7], oc.conv_forward(x3, w)[0, :7])


def test_silu_closed_forms():
    x = np.array([[[0.0], [0.0]]])
    w = np.zeros((1, 4))
    assert np.all(oc.conv_forward(x, w, np.array([0.0])) == 0.0)
    y = oc.conv_forward(x, w, np.array([2.0]))
    assert np.allclose(y, 2.0 / (1.0 + np.exp(-2.0)), rtol=1e-15)


def test_gradients_match_finite_differences():
    rng = np.random.default_rng(2)
    B, L, C, K = 2, 7, 3, 4
    x, w, b, dy = rng.normal(size=(B, L, C)), rng.normal(size=(C, K)), rng.normal(size=C), rng.normal(size=(B, L, C))
    for act in (True, False):
        g = oc.conv_backward(x, w, dy, b, act)
        loss = lambda x, w, b: float(np.sum(oc.conv_forward(x, w, b, act) * dy))
        h = 1e-6
        for name, arr, idx_fn in (("dx", x, lambda a: (a, w, b)), ("dw", w, lambda a: (x, a, b)),
                                  ("dbias", b, lambda a: (x, w, a))):
            fd = np.zeros(arr.shape)
            for i in np.ndindex(*arr.shape):
                up, dn = arr.copy(), arr.copy()
                up[i] += h
                dn[i] -= h
                fd[i] = (loss(*idx_fn(up)) - loss(*idx_fn(dn))) / (2 * h)
            assert np.allclose(g[name], fd, rtol=1e-6, atol=1e-8), (name, act)


def test_sequence_shorter_than_the_kernel():
    rng = np.random.default_rng(3)
    x, w = rng.normal(size=(1, 2, 2)), rng.normal(size=(2, 4))
    y = oc.conv_forward(x, w, activation=False)
    assert np.allclose(y[0, 0], w[:, 3] * x[0, 0])
    assert np.allclose(y[0, 1], w[:, 3] * x[0, 1] + w[:, 2] * x[0, 0])
