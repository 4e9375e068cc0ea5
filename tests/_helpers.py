"""Shared helpers for the parity tests: error metrics and oracle runs on
selected (batch, head) pairs."""
import os

import numpy as np
import torch

import oracle

# Tolerances:
#  fp32 I/O: elementwise relative error floored by the tensor RMS <= 1e-4.
#  bf16 I/O: the same mixed metric <= 2e-2, and the normwise error <= 1e-2.
TOL = {"f32": dict(mixed=1e-4, l2=1e-5), "bf16": dict(mixed=2e-2, l2=1e-2)}


def cores():
    return max(1, min(16, len(os.sched_getaffinity(0))))


def to64(t):
    return t.detach().to("cpu").double().numpy()


def err(X, R, floor=0.0):
    X = np.asarray(X, dtype=np.float64)
    R = np.asarray(R, dtype=np.float64)
    rms = float(np.sqrt(np.mean(R * R))) if R.size else 0.0
    rms = max(rms, floor, 1e-30)
    d = np.abs(X - R)
    return dict(mixed=float(np.max(d / np.maximum(np.abs(R), rms))) if d.size else 0.0,
                max_over_rms=float(d.max() / rms) if d.size else 0.0,
                l2=float(np.linalg.norm(d) / max(np.linalg.norm(R), floor * np.sqrt(R.size), 1e-30))
                if d.size else 0.0)


def assert_close(name, X, R, io, floor=0.0):
    """floor: an extra lower bound on the error scale (used for dg, see dg_floor)."""
    e = err(X, R, floor)
    tol = TOL[io]
    print(f"  {name:7s} mixed={e['mixed']:.3e} max/rms={e['max_over_rms']:.3e} l2={e['l2']:.3e}",
          flush=True)
    assert np.all(np.isfinite(np.asarray(X, dtype=np.float64))), f"{name}: non-finite values"
    assert e["mixed"] <= tol["mixed"] and e["l2"] <= tol["l2"], f"{name}: {e} exceeds {tol}"
    return e


def select(x, pairs):
    """Stack (b, h) slices of a [B, L, H, ...] tensor into [1, L, P, ...]."""
    return torch.stack([x[b, :, h] for b, h in pairs], dim=1).unsqueeze(0)


def select_state(s, pairs):
    if s is None:
        return None
    return torch.stack([s[b, h] for b, h in pairs], dim=0).unsqueeze(0)


def oracle_run(inp, pairs=None, snap_pos=None):
    """Oracle forward + backward on the given (b, h) pairs (all by default).

    Returns dict of float64 arrays with a leading [1, L, P] (or [1, P]) layout."""
    q, k, v, g, dO = inp["q"], inp["k"], inp["v"], inp["g"], inp["dO"]
    B, L, H, D = q.shape
    if pairs is None:
        pairs = [(b, h) for b in range(B) for h in range(H)]
    sq, sk, sv, sg, sdo = (to64(select(x, pairs)) for x in (q, k, v, g, dO))
    S_in = select_state(inp.get("S_in"), pairs)
    dS = select_state(inp.get("dS_out"), pairs)
    S_in = to64(S_in) if S_in is not None else None
    dS = to64(dS) if dS is not None else None
    o, S_out, snaps = oracle.forward(sq, sk, sv, sg, S_in, snap_pos=snap_pos, threads=cores())
    dq, dk, dv, dg, dS_in = oracle.backward(sq, sk, sv, sg, S_in, sdo, dS, threads=cores())
    return dict(o=o, S_out=S_out, snaps=snaps, dq=dq, dk=dk, dv=dv, dg=dg, dS_in=dS_in, pairs=pairs)


def dg_floor(ref, q, k):
    """Scale of the per-token terms q_t.dq_t and k_t.dk_t (per channel for the
    vector gate) whose telescoping sum
    gives the decay gradient (dg_t = sum_{t'>=t} (q.dq - k.dk)_{t'} plus the
    carry from later superchunks).  The kernels evaluate dg through that sum,
    so its absolute error is relative to this scale; when the gate is so
    strong that dg itself is many orders smaller (a_t ~ 0), this floor keeps
    the metric meaningful."""
    if ref["dg"].ndim == q.ndim:  # per-key-channel gate: dg per channel
        qd, kd = q * ref["dq"], k * ref["dk"]
    else:
        qd = np.sum(q * ref["dq"], axis=-1)
        kd = np.sum(k * ref["dk"], axis=-1)
    return float(np.sqrt(np.mean(qd * qd + kd * kd)))
