"""fp64 oracle of the gated delta rule (Gated DeltaNet), the paper's main
evaluated operator (Sec. 2.1: scalar-plus-low-rank transition).

TEST INFRASTRUCTURE ONLY.  Token-by-token forward and hand-written backward
in gdn_oracle.c (see its header for the equations); pinned by
tests/test_gdn_oracle_pins.py.
"""
import ctypes

import numpy as np

from . import _f64, _load, _ptr

_ready = False


def _lib():
    global _ready
    lib = _load()
    if not _ready:
        dp = ctypes.POINTER(ctypes.c_double)
        lib.gdo_forward.argtypes = [ctypes.c_int] * 4 + [ctypes.c_long] + [dp] * 9 + [ctypes.c_int]
        lib.gdo_forward.restype = ctypes.c_int
        lib.gdo_backward.argtypes = [ctypes.c_int] * 4 + [ctypes.c_long] + [dp] * 14 + [ctypes.c_int]
        lib.gdo_backward.restype = ctypes.c_int
        _ready = True
    return lib


def _dims(q, v, g, beta):
    B, L, H, Dk = q.shape
    assert g.shape == (B, L, H) and beta.shape == (B, L, H)
    return B, L, H, Dk, v.shape[3]


def forward(q, k, v, g, beta, S_in=None, threads=0, with_u=False):
    """Returns (o, S_out) in float64, and u (the corrected values V^new,
    [B, L, H, Dv]) after them when with_u.  q, k: [B, L, H, Dk];
    v: [B, L, H, Dv]; g (natural-log decay), beta: [B, L, H];
    S_in: [B, H, Dk, Dv] or None."""
    q, k, v, g, beta, S_in = (_f64(x) for x in (q, k, v, g, beta, S_in))
    B, L, H, Dk, Dv = _dims(q, v, g, beta)
    o = np.zeros((B, L, H, Dv))
    S_out = np.zeros((B, H, Dk, Dv))
    u = np.zeros((B, L, H, Dv)) if with_u else None
    rc = _lib().gdo_forward(B, H, Dk, Dv, L, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S_in), _ptr(o),
                            _ptr(S_out), _ptr(u), int(threads))
    if rc != 0:
        raise RuntimeError(f"gdo_forward failed ({rc})")
    return (o, S_out, u) if with_u else (o, S_out)


def backward(q, k, v, g, beta, S_in, dO, dS_out=None, threads=0):
    """Returns (dq, dk, dv, dg, dbeta, dS_in) in float64 for
    Loss = sum_t <dO_t, o_t> + <dS_out, S_out>."""
    q, k, v, g, beta, S_in, dO, dS_out = (_f64(x) for x in (q, k, v, g, beta, S_in, dO, dS_out))
    B, L, H, Dk, Dv = _dims(q, v, g, beta)
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    dg, dbeta = np.zeros_like(g), np.zeros_like(beta)
    dS_in = np.zeros((B, H, Dk, Dv))
    rc = _lib().gdo_backward(B, H, Dk, Dv, L, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S_in), _ptr(dO),
                             _ptr(dS_out), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dg), _ptr(dbeta), _ptr(dS_in),
                             int(threads))
    if rc != 0:
        raise RuntimeError(f"gdo_backward failed ({rc})")
    return dq, dk, dv, dg, dbeta, dS_in
