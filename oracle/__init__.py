"""fp64 CPU oracle for the segmented gated linear recurrence.

TEST INFRASTRUCTURE ONLY: tests/, __graft_entry__.smoke() and the cpu_baseline
leg of bench.py may import it; the product path (paper_2608_06838_amd) never
does, and the two share no code.

`forward` / `backward` run the plain token-by-token definition (paper Sec. 2.1,
Eq. 1: S_t = a_t o S_{t-1} + k_t v_t^T, o_t = S_t^T q_t, a_t = exp(g_t)) and its
hand-written reverse-mode derivative (Sec. 3.1, "Backward Computation": dS_out in,
dS_in out), in C (sf_oracle.c) with OpenMP over (batch, head).  Because the
paper's sequence chunking is exact (Sec. 4.1 states it introduces no
approximation), a chained run over segments equals one run over the whole
sequence; `forward(..., snap_pos=...)` returns the boundary states a chain
produces.

Every function here is pinned by tests/test_oracle_pins.py against brute force,
closed forms, finite differences, an autograd route and composition identities.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_build.LIB):
        _build.build()
    lib = ctypes.CDLL(_build.LIB)
    dp = ctypes.POINTER(ctypes.c_double)
    lp = ctypes.POINTER(ctypes.c_long)
    lib.sfo_forward.argtypes = [ctypes.c_int] * 4 + [ctypes.c_long, ctypes.c_int] + [dp] * 7 + [
        ctypes.c_int, lp, dp, ctypes.c_int]
    lib.sfo_forward.restype = ctypes.c_int
    lib.sfo_backward.argtypes = [ctypes.c_int] * 4 + [ctypes.c_long, ctypes.c_int] + [dp] * 12 + [
        ctypes.c_int]
    lib.sfo_backward.restype = ctypes.c_int
    _lib = lib
    return lib


def _f64(x):
    """Exact upcast to a C-contiguous float64 numpy array (accepts torch tensors)."""
    if x is None:
        return None
    if hasattr(x, "detach"):  # torch tensor: exact upcast on the CPU
        x = x.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _dims(q, v, g):
    B, L, H, Dk = q.shape
    Dv = v.shape[3]
    if g.ndim == 4:
        vec = 1
        assert g.shape == (B, L, H, Dk)
    else:
        vec = 0
        assert g.shape == (B, L, H)
    return B, L, H, Dk, Dv, vec


def forward(q, k, v, g, S_in=None, snap_pos=None, threads=0):
    """Returns (o, S_out, snaps) in float64.

    q, k: [B, L, H, Dk]; v: [B, L, H, Dv]; g: [B, L, H] (scalar gate) or
    [B, L, H, Dk] (vector gate), natural-log decay; S_in: [B, H, Dk, Dv] or None.
    snaps[p] is the state after snap_pos[p] tokens.
    """
    q, k, v, g, S_in = (_f64(x) for x in (q, k, v, g, S_in))
    B, L, H, Dk, Dv, vec = _dims(q, v, g)
    o = np.zeros((B, L, H, Dv))
    S_out = np.zeros((B, H, Dk, Dv))
    pos = np.ascontiguousarray(np.asarray(snap_pos if snap_pos is not None else [], dtype=np.int64))
    snaps = np.zeros((max(len(pos), 1), B, H, Dk, Dv))
    rc = _load().sfo_forward(B, H, Dk, Dv, L, vec, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(S_in),
                             _ptr(o), _ptr(S_out), len(pos),
                             pos.ctypes.data_as(ctypes.POINTER(ctypes.c_long)), _ptr(snaps),
                             int(threads))
    if rc != 0:
        raise RuntimeError(f"sfo_forward failed ({rc})")
    return o, S_out, snaps[: len(pos)]


def backward(q, k, v, g, S_in, dO, dS_out=None, threads=0):
    """Returns (dq, dk, dv, dg, dS_in) in float64 for
    Loss = sum_t <dO_t, o_t> + <dS_out, S_out>."""
    q, k, v, g, S_in, dO, dS_out = (_f64(x) for x in (q, k, v, g, S_in, dO, dS_out))
    B, L, H, Dk, Dv, vec = _dims(q, v, g)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    dg = np.zeros_like(g)
    dS_in = np.zeros((B, H, Dk, Dv))
    rc = _load().sfo_backward(B, H, Dk, Dv, L, vec, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(S_in),
                              _ptr(dO), _ptr(dS_out), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dg),
                              _ptr(dS_in), int(threads))
    if rc != 0:
        raise RuntimeError(f"sfo_backward failed ({rc})")
    return dq, dk, dv, dg, dS_in

from .conv import conv_backward, conv_forward  # noqa: E402,F401
