"""fp64 oracle of the short convolution with a boundary tail.

TEST INFRASTRUCTURE ONLY: tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may use it; the product path never does.

Sec. 3.1 lets the boundary state of a segment include short-convolution
states next to S.  The operation (its form is a reading: the paper names it
only) is a causal depthwise convolution of W taps over the tokens, per batch
b and channel c,

    u_t[c] = sum_{j=0}^{W-1} w[c][j] * xh_{t-W+1+j}[c],     y_t[c] = act(u_t[c]),

with xh the segment input preceded by the tail of the previous segment
(xh_s = tail_in[W-1+s] for s < 0).  The tail handed on is the last W-1
entries of xh.  act is the identity or SiLU, u * sigmoid(u).

The backward is the reverse-mode derivative of the loss
    sum_t <dy_t, y_t> + <dtail_out, tail_out>
written out by hand: du = dy * act'(u); each tap j sends w[c][j] du_t back to
xh_{t-W+1+j}; tail_out sends dtail_out back to the last W-1 entries of xh; and
dw[c][j] = sum over batch and tokens of du_t[c] xh_{t-W+1+j}[c].

Pinned by tests/test_oracle_pins.py: numpy's correlate on single channels,
identity and shift kernels, segment composition, finite differences and the
SiLU closed forms.
"""
import numpy as np


def _f64(x):
    if x is None:
        return None
    if hasattr(x, "detach"):
        x = x.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def silu(u):
    with np.errstate(over="ignore"):
        return u / (1.0 + np.exp(-u))


def silu_grad(u):
    with np.errstate(over="ignore"):
        s = 1.0 / (1.0 + np.exp(-u))
    return s * (1.0 + u * (1.0 - s))


def _extended(x, W, tail_in):
    B, L, C = x.shape
    tail = np.zeros((B, W - 1, C)) if tail_in is None or W == 1 else _f64(tail_in)
    return np.concatenate([tail, x], axis=1)  # xh[:, W-1+s] = x_s


def _pre(xh, w, L):
    W = w.shape[1]
    u = np.zeros((xh.shape[0], L, xh.shape[2]))
    for j in range(W):
        u += w[:, j] * xh[:, j:j + L, :]
    return u


def conv_forward(x, w, tail_in=None, act="silu"):
    """Returns (y, tail_out) in float64.  x: [B, L, C]; w: [C, W];
    tail_in: [B, W-1, C] or None (zeros)."""
    x, w = _f64(x), _f64(w)
    B, L, C = x.shape
    W = w.shape[1]
    xh = _extended(x, W, tail_in)
    u = _pre(xh, w, L)
    y = silu(u) if act == "silu" else u
    return y, xh[:, L:L + W - 1, :].copy()


def conv_backward(x, w, tail_in, dy, dtail_out=None, act="silu"):
    """Returns (dx, dw, dtail_in) in float64."""
    x, w, dy = _f64(x), _f64(w), _f64(dy)
    B, L, C = x.shape
    W = w.shape[1]
    xh = _extended(x, W, tail_in)
    u = _pre(xh, w, L)
    du = dy * silu_grad(u) if act == "silu" else dy
    dxh = np.zeros_like(xh)
    for j in range(W):
        dxh[:, j:j + L, :] += w[:, j] * du
    if dtail_out is not None and W > 1:
        dxh[:, L:L + W - 1, :] += _f64(dtail_out)
    dw = np.zeros((C, W))
    for j in range(W):
        dw[:, j] = (du * xh[:, j:j + L, :]).sum(axis=(0, 1))
    return dxh[:, W - 1:, :], dw, dxh[:, :W - 1, :]
