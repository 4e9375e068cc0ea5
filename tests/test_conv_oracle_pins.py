"""Pins for the short-convolution oracle (CPU only).

The oracle is checked against numpy's own correlate on single channels, the
identity and shift kernels, the closed forms of SiLU and its derivative,
central finite differences of the loss sum <dy, y> + <dtail_out, tail_out>,
and the exact segment composition that carrying the tail must give (Sec. 3.1:
a segment's boundary state may include short-convolution states).  A reversed
tap order, an off-by-one in the tail, a dropped tail-gradient term or a wrong
dw index fails at least one of them.
"""
import numpy as np
import pytest

import oracle
from oracle import conv as oc


def rand(rng, B, L, C, W):
    x = rng.standard_normal((B, L, C))
    w = rng.standard_normal((C, W))
    tail = rng.standard_normal((B, W - 1, C))
    dy = rng.standard_normal((B, L, C))
    dtail = rng.standard_normal((B, W - 1, C))
    return x, w, tail, dy, dtail


@pytest.mark.parametrize("W", [1, 2, 3, 4])
def test_matches_numpy_correlate(W):
    rng = np.random.default_rng(10 + W)
    B, L, C = 2, 37, 5
    x, w, tail, _, _ = rand(rng, B, L, C, W)
    u, tail_out = oracle.conv_forward(x, w, tail, act="none")
    for b in range(B):
        for c in range(C):
            xh = np.concatenate([tail[b, :, c], x[b, :, c]])
            ref = np.correlate(xh, w[c], mode="valid")  # sum_j xh[t+j] w[j]
            np.testing.assert_allclose(u[b, :, c], ref, rtol=1e-13, atol=1e-13)
            np.testing.assert_array_equal(tail_out[b, :, c], xh[len(xh) - (W - 1):] if W > 1 else xh[:0])


def test_identity_and_shift_kernels():
    rng = np.random.default_rng(3)
    B, L, C, W = 2, 20, 4, 4
    x, _, tail, _, _ = rand(rng, B, L, C, W)
    ident = np.zeros((C, W))
    ident[:, W - 1] = 1.0
    y, _ = oracle.conv_forward(x, ident, tail, act="silu")
    np.testing.assert_allclose(y, x / (1.0 + np.exp(-x)), rtol=1e-15)
    shift = np.zeros((C, W))
    shift[:, 0] = 1.0  # y_t = xh_{t-W+1}
    u, _ = oracle.conv_forward(x, shift, tail, act="none")
    np.testing.assert_array_equal(u[:, W - 1:], x[:, :L - (W - 1)])
    np.testing.assert_array_equal(u[:, :W - 1], tail)


def test_silu_closed_forms():
    # sigmoid(log 3) = 3/4 exactly, so silu(log 3) = 0.75 log 3 and
    # silu'(log 3) = 3/4 (1 + log 3 / 4)
    u = np.array([0.0, np.log(3.0), 60.0, -60.0])
    np.testing.assert_allclose(oc.silu(u)[:2], [0.0, 0.75 * np.log(3.0)], rtol=1e-15, atol=0)
    np.testing.assert_allclose(oc.silu(u)[2], 60.0, rtol=1e-15)
    assert abs(oc.silu(u)[3]) < 1e-24
    np.testing.assert_allclose(oc.silu_grad(u)[:2], [0.5, 0.75 * (1.0 + np.log(3.0) / 4.0)], rtol=1e-15)
    np.testing.assert_allclose(oc.silu_grad(u)[2:], [1.0, 0.0], atol=1e-20)


@pytest.mark.parametrize("W", [2, 4])
@pytest.mark.parametrize("act", ["none", "silu"])
def test_gradients_finite_differences(W, act):
    rng = np.random.default_rng(100 + W)
    B, L, C = 2, 9, 3
    x, w, tail, dy, dtail = rand(rng, B, L, C, W)

    def loss(x_, w_, t_):
        y, to = oracle.conv_forward(x_, w_, t_, act=act)
        return float((dy * y).sum() + (dtail * to).sum())

    dx, dw, dti = oracle.conv_backward(x, w, tail, dy, dtail, act=act)
    h = 1e-6
    for arr, grad, idx_list in ((x, dx, [(0, 0, 0), (1, 4, 2), (0, L - 1, 1), (1, L - 2, 0)]),
                                (w, dw, [(0, 0), (2, W - 1), (1, 1)]),
                                (tail, dti, [(0, 0, 0), (1, W - 2, 2)])):
        for idx in idx_list:
            p, m = arr.copy(), arr.copy()
            p[idx] += h
            m[idx] -= h
            args_p = [p if arr is a else a for a in (x, w, tail)]
            args_m = [m if arr is a else a for a in (x, w, tail)]
            fd = (loss(*args_p) - loss(*args_m)) / (2 * h)
            assert abs(fd - grad[idx]) <= 1e-6 * max(1.0, abs(fd)), (idx, fd, grad[idx])


@pytest.mark.parametrize("W", [1, 3, 4])
def test_segment_composition(W):
    """Two segments chained through the tail equal one call over both, in the
    forward (y, tail_out) and the backward (dx, dw, dtail_in); the second
    segment is shorter than the tail."""
    rng = np.random.default_rng(7 + W)
    B, C = 2, 3
    for L1, L2 in ((13, 2), (5, 11), (1, 1)):
        x, w, tail, dy, dtail = rand(rng, B, L1 + L2, C, W)
        y, to = oracle.conv_forward(x, w, tail)
        y1, t1 = oracle.conv_forward(x[:, :L1], w, tail)
        y2, t2 = oracle.conv_forward(x[:, L1:], w, t1)
        np.testing.assert_allclose(np.concatenate([y1, y2], axis=1), y, rtol=1e-14, atol=1e-14)
        np.testing.assert_array_equal(t2, to)
        dx, dw, dti = oracle.conv_backward(x, w, tail, dy, dtail)
        dx2, dw2, dti2 = oracle.conv_backward(x[:, L1:], w, t1, dy[:, L1:], dtail)
        dx1, dw1, dti1 = oracle.conv_backward(x[:, :L1], w, tail, dy[:, :L1], dti2)
        np.testing.assert_allclose(np.concatenate([dx1, dx2], axis=1), dx, rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(dw1 + dw2, dw, rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(dti1, dti, rtol=1e-13, atol=1e-13)


def test_short_and_empty_segments():
    rng = np.random.default_rng(5)
    B, C, W = 1, 2, 4
    x, w, tail, dy, dtail = rand(rng, B, 2, C, W)
    _, to = oracle.conv_forward(x, w, tail)
    # L = 2 < W - 1 = 3: the tail keeps the newest tail_in entry, then x
    np.testing.assert_array_equal(to[:, 0], tail[:, 2])
    np.testing.assert_array_equal(to[:, 1:], x)
    x0 = np.zeros((B, 0, C))
    y0, t0 = oracle.conv_forward(x0, w, tail)
    assert y0.shape == (B, 0, C)
    np.testing.assert_array_equal(t0, tail)
    dx0, dw0, dti0 = oracle.conv_backward(x0, w, tail, x0, dtail)
    np.testing.assert_array_equal(dti0, dtail)
    np.testing.assert_array_equal(dw0, np.zeros((C, W)))
