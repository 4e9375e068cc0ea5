"""libstateflow for MI355X: the segmented gated linear recurrence of StateFlow
(arXiv 2608.06838) as hand-written gfx950 HIP kernels behind a C ABI.

Python surface (torch tensors in, torch tensors out; PyTorch supplies device
memory and streams only, every arithmetic step runs in libstateflow.so):

    o, S_out                 = segment_fwd(q, k, v, g, S_in)
    dq, dk, dv, dg, dS_in    = segment_bwd(q, k, v, g, S_in, dO, dS_out)
    o, S_bnd                 = chain_fwd(q, k, v, g, seg_lens, S_init)
    dq, dk, dv, dg, dS_init  = chain_bwd(q, k, v, g, seg_lens, S_bnd, dO, dS_final)

Shapes: q, k, v, dO: [B, L, H, D] (bf16 or fp32, channel dim contiguous, all
with the same strides); g: [B, L, H] fp32 natural-log decay; states:
[B, H, D, D] fp32 (S stored as Dk x Dv).  See include/stateflow.h.

The short convolution whose tail is the auxiliary boundary state of a segment:

    y, tail_out              = conv_fwd(x, w, tail_in, act="silu")
    dx, dw, dtail_in         = conv_bwd(x, w, tail_in, dy, dtail_out, act="silu")

x, y: [B, L, C] (bf16 or fp32, channels contiguous); w: [C, W] fp32;
tails: [B, W-1, C] fp32.
"""
import ctypes

import torch

from . import _lib
from ._lib import KERNELS, StateflowError  # noqa: F401
from . import tuned
from .timing import KernelTimer  # noqa: F401

__all__ = ["segment_fwd", "segment_fwd_noalloc", "segment_bwd", "chain_ckpt_bytes", "chain_fwd", "chain_bwd", "fwd_workspace_bytes",
           "bwd_workspace_bytes", "chain_workspace_bytes", "conv_fwd", "conv_bwd", "conv_bwd_workspace_bytes",
           "gdn_fwd", "gdn_fwd_workspace_bytes", "gdn_bwd", "gdn_chain_ckpt_bytes", "gdn_chain_fwd", "gdn_chain_bwd", "partition_hybrid", "KernelTimer", "StateflowError", "abi_version"]

_IO = {torch.bfloat16: _lib.SF_BF16, torch.float32: _lib.SF_F32}
_aux_streams = {}


def abi_version():
    return _lib.lib().sf_abi_version()


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream_handle(s):
    return ctypes.c_void_p(s.cuda_stream)


def _overlap_mode(overlap):
    """False / True select modes 0 / 1; the integers 0, 1, 2 pass through
    (2: the preparation kernels on the aux stream as well, see sf_tuning)."""
    if isinstance(overlap, bool):
        return int(overlap)
    m = int(overlap)
    if m not in (0, 1, 2):
        raise ValueError(f"overlap must be a bool or 0, 1 or 2, got {overlap!r}")
    return m


def _tuning(ts=0, overlap=True, timing=None):
    """timing: a timing.KernelTimer whose record the call's launches use."""
    t = _lib.SfTuning()
    t.ts = int(ts)
    t.overlap = _overlap_mode(overlap)
    if timing is not None:
        t.timing = ctypes.pointer(timing.rec)
    return t


def _shape(q, g):
    if q.dim() != 4:
        raise ValueError("q must be [B, L, H, D]")
    if q.dtype not in _IO:
        raise TypeError(f"unsupported I/O dtype {q.dtype}")
    if g.dtype != torch.float32:
        raise TypeError("g must be float32")
    B, L, H, D = q.shape
    vec = g.dim() == 4
    if (vec and tuple(g.shape) != (B, L, H, D)) or (not vec and tuple(g.shape) != (B, L, H)):
        raise ValueError(f"g has shape {tuple(g.shape)}, expected {(B, L, H)} or {(B, L, H, D)}")
    if q.stride(3) != 1 or (vec and g.stride(3) != 1):
        raise ValueError("the channel dim must be contiguous")
    sh = _lib.SfShape()
    sh.B, sh.H, sh.Dk, sh.Dv, sh.L = B, H, D, D, L
    sh.chunk = 64
    sh.io_dtype = _IO[q.dtype]
    sh.gate = _lib.SF_GATE_VECTOR if vec else _lib.SF_GATE_SCALAR
    sh.reserved = 0
    sh.sx_b, sh.sx_l, sh.sx_h = q.stride(0), q.stride(1), q.stride(2)
    sh.sg_b, sh.sg_l, sh.sg_h = g.stride(0), g.stride(1), g.stride(2)
    return sh


def _same_layout(ref, *ts):
    for t in ts:
        if t is None:
            continue
        if t.shape != ref.shape or t.stride() != ref.stride() or t.dtype != ref.dtype:
            raise ValueError("q, k, v, dO must share shape, strides and dtype")
        if t.device != ref.device:
            raise ValueError("all tensors must be on one device")


def _state(t, B, H, D, name, n=None):
    if t is None:
        return None
    want = (B, H, D, D) if n is None else (n, B, H, D, D)
    if tuple(t.shape) != want or t.dtype != torch.float32 or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous float32 tensor of shape {want}")
    return t


def _like(x):
    return torch.empty_strided(x.size(), x.stride(), dtype=x.dtype, device=x.device)


def _ws(nbytes, device):
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def fwd_workspace_bytes(q, g, ts=0):
    return _lib.lib().sf_fwd_workspace_bytes(ctypes.byref(_shape(q, g)), ctypes.byref(_tuning(ts)))


def bwd_workspace_bytes(q, g, ts=0):
    return _lib.lib().sf_bwd_workspace_bytes(ctypes.byref(_shape(q, g)), ctypes.byref(_tuning(ts)))


def gdn_fwd_workspace_bytes(q, g, ts=0):
    return _lib.lib().sf_gdn_fwd_workspace_bytes(ctypes.byref(_shape(q, g)), ctypes.byref(_tuning(ts)))


def chain_workspace_bytes(q, g, seg_lens, ts=0):
    sl = (ctypes.c_int64 * len(seg_lens))(*[int(x) for x in seg_lens])
    return _lib.lib().sf_chain_workspace_bytes(ctypes.byref(_shape(q, g)), len(seg_lens), sl,
                                               ctypes.byref(_tuning(ts)))


def segment_fwd(q, k, v, g, S_in=None, *, ts=0, stream=None, timing=None):
    """(o, S_out) = Fwd(q, k, v, g; S_in) for one segment."""
    _same_layout(q, k, v)
    sh = _shape(q, g)
    B, L, H, D = q.shape
    _state(S_in, B, H, D, "S_in")
    stream = stream or torch.cuda.current_stream(q.device)
    L_ = _lib.lib()
    tun = _tuning(ts, timing=timing)
    with torch.cuda.stream(stream):
        o = _like(q)
        S_out = torch.empty((B, H, D, D), dtype=torch.float32, device=q.device)
        nbytes = L_.sf_fwd_workspace_bytes(ctypes.byref(sh), ctypes.byref(tun))
        ws = _ws(nbytes, q.device)
    rc = L_.sf_segment_fwd(ctypes.byref(sh), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(S_in), _ptr(o),
                           _ptr(S_out), _ptr(ws), ws.numel(), ctypes.byref(tun), _stream_handle(stream))
    _lib.check("sf_segment_fwd", rc)
    return o, S_out


def segment_fwd_noalloc(q, k, v, g, S_in, o, S_out, *, ts=0, stream=None, timing=None):
    """segment_fwd into caller-supplied o and S_out through the library's
    allocation-free entry point (no workspace; nothing is allocated here
    either).  o: like q; S_out: float32 [B, H, D, D] contiguous."""
    _same_layout(q, k, v, o)
    sh = _shape(q, g)
    B, L, H, D = q.shape
    _state(S_in, B, H, D, "S_in")
    _state(S_out, B, H, D, "S_out")
    stream = stream or torch.cuda.current_stream(q.device)
    rc = _lib.lib().sf_segment_fwd_noalloc(ctypes.byref(sh), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(S_in),
                                           _ptr(o), _ptr(S_out), ctypes.byref(_tuning(ts, timing=timing)),
                                           _stream_handle(stream))
    _lib.check("sf_segment_fwd_noalloc", rc)
    return o, S_out


def segment_bwd(q, k, v, g, S_in, dO, dS_out=None, *, ts=0, stream=None, timing=None):
    """(dq, dk, dv, dg, dS_in) = Bwd(q, k, v, g, S_in; dO, dS_out) for one segment."""
    _same_layout(q, k, v, dO)
    sh = _shape(q, g)
    B, L, H, D = q.shape
    _state(S_in, B, H, D, "S_in")
    _state(dS_out, B, H, D, "dS_out")
    stream = stream or torch.cuda.current_stream(q.device)
    L_ = _lib.lib()
    tun = _tuning(ts, timing=timing)
    with torch.cuda.stream(stream):
        dq, dk, dv = _like(q), _like(q), _like(q)
        dg = _like(g)
        dS_in = torch.empty((B, H, D, D), dtype=torch.float32, device=q.device)
        nbytes = L_.sf_bwd_workspace_bytes(ctypes.byref(sh), ctypes.byref(tun))
        ws = _ws(nbytes, q.device)
    rc = L_.sf_segment_bwd(ctypes.byref(sh), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(S_in), _ptr(dO),
                           _ptr(dS_out), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dg), _ptr(dS_in), _ptr(ws),
                           ws.numel(), ctypes.byref(tun), _stream_handle(stream))
    _lib.check("sf_segment_bwd", rc)
    return dq, dk, dv, dg, dS_in


def _aux_for(device, aux_stream, overlap):
    if not overlap:
        return None
    if aux_stream is not None:
        return aux_stream
    key = torch.device(device).index
    if key not in _aux_streams:
        _aux_streams[key] = torch.cuda.Stream(device=device)  # default priority
    return _aux_streams[key]


def _pick(q, g, seg_lens, ts, overlap):
    """ts / overlap left as None take the profiled per-shape setting."""
    if ts is not None and overlap is not None:
        return int(ts), _overlap_mode(overlap)
    B, L, H, D = q.shape
    t = tuned.lookup(B, H, D, "bf16" if q.dtype == torch.bfloat16 else "f32",
                     "vector" if g.dim() == 4 else "scalar", seg_lens)
    return (t["ts"] if ts is None else int(ts)), _overlap_mode(t["overlap"] if overlap is None else overlap)


def chain_ckpt_bytes(q, g, seg_lens, ts=None, overlap=None):
    """Bytes of the superchunk states chain_fwd(keep_states=True) keeps."""
    sh = _shape(q, g)
    n = len(seg_lens)
    ts, overlap = _pick(q, g, seg_lens, ts, overlap)
    tun = _tuning(ts, overlap)
    sl = (ctypes.c_int64 * n)(*[int(x) for x in seg_lens])
    L_ = _lib.lib()
    nb = L_.sf_chain_ckpt_bytes(ctypes.byref(sh), n, sl, ctypes.byref(tun))
    if nb == 0 and L_.sf_last_error():
        raise StateflowError("sf_chain_ckpt_bytes: " + L_.sf_last_error().decode())
    return nb


def chain_fwd(q, k, v, g, seg_lens, S_init=None, *, ts=None, overlap=None, stream=None, aux_stream=None,
              out=None, timing=None, keep_states=False):
    """Forward over consecutive segments with S_in(i+1) = S_out(i).

    Returns (o, S_bnd) with S_bnd[i] the state entering segment i
    (S_bnd[0] = S_init or zero, S_bnd[-1] the final state).  `out` may supply
    preallocated (o, S_bnd, workspace) buffers.  keep_states=True also returns
    the superchunk states (a uint8 device tensor of chain_ckpt_bytes bytes, or
    a caller's buffer given as out[3]) for chain_bwd(ckpt=...), which then
    skips replaying them; the results are the same.  overlap: None takes the
    profiled per-shape setting; False / 0 serialises on `stream`; True / 1
    runs the state scans on the aux stream; 2 runs each segment's
    preparation kernel there as well, ahead of its scan.  ts and overlap do
    not change the results.
    """
    _same_layout(q, k, v)
    sh = _shape(q, g)
    B, L, H, D = q.shape
    n = len(seg_lens)
    _state(S_init, B, H, D, "S_init")
    ts, overlap = _pick(q, g, seg_lens, ts, overlap)
    stream = stream or torch.cuda.current_stream(q.device)
    aux = _aux_for(q.device, aux_stream, overlap)
    L_ = _lib.lib()
    tun = _tuning(ts, overlap, timing)
    sl = (ctypes.c_int64 * n)(*[int(x) for x in seg_lens])
    ck = None
    with torch.cuda.stream(stream):
        if out is None:
            o = _like(q)
            S_bnd = torch.empty((n + 1, B, H, D, D), dtype=torch.float32, device=q.device)
            ws = _ws(L_.sf_chain_workspace_bytes(ctypes.byref(sh), n, sl, ctypes.byref(tun)), q.device)
        else:
            o, S_bnd, ws = out[:3]
            ck = out[3] if len(out) > 3 else None
        if keep_states and ck is None:
            ck = _ws(L_.sf_chain_ckpt_bytes(ctypes.byref(sh), n, sl, ctypes.byref(tun)), q.device)
        if S_init is None:
            S_bnd[0].zero_()
        else:
            S_bnd[0].copy_(S_init)
    if not keep_states:
        ck = None
    rc = L_.sf_chain_fwd(ctypes.byref(sh), n, sl, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(o), _ptr(S_bnd),
                         _ptr(ck), ck.numel() if ck is not None else 0, _ptr(ws), ws.numel(),
                         ctypes.byref(tun), _stream_handle(stream), _stream_handle(aux) if aux is not None else None)
    _lib.check("sf_chain_fwd", rc)
    return (o, S_bnd, ck) if keep_states else (o, S_bnd)


def chain_bwd(q, k, v, g, seg_lens, S_bnd, dO, dS_final=None, *, ts=None, overlap=None, stream=None,
              aux_stream=None, out=None, timing=None, ckpt=None):
    """Backward over the segments in reverse with dS_out(i) = dS_in(i+1).

    Returns (dq, dk, dv, dg, dS_init).  `out` may supply preallocated
    (dq, dk, dv, dg, dS_init, workspace) buffers.  ckpt: the superchunk states
    of chain_fwd(keep_states=True) for the same inputs, segments and settings.
    """
    _same_layout(q, k, v, dO)
    sh = _shape(q, g)
    B, L, H, D = q.shape
    n = len(seg_lens)
    if (S_bnd.dim() != 5 or S_bnd.shape[0] < n or tuple(S_bnd.shape[1:]) != (B, H, D, D)
            or S_bnd.dtype != torch.float32 or not S_bnd.is_contiguous()):
        raise ValueError("S_bnd must be a contiguous float32 [n_seg(+1), B, H, D, D] tensor")
    _state(dS_final, B, H, D, "dS_final")
    ts, overlap = _pick(q, g, seg_lens, ts, overlap)
    stream = stream or torch.cuda.current_stream(q.device)
    aux = _aux_for(q.device, aux_stream, overlap)
    L_ = _lib.lib()
    tun = _tuning(ts, overlap, timing)
    sl = (ctypes.c_int64 * n)(*[int(x) for x in seg_lens])
    with torch.cuda.stream(stream):
        if out is None:
            dq, dk, dv = _like(q), _like(q), _like(q)
            dg = _like(g)
            dS_init = torch.empty((B, H, D, D), dtype=torch.float32, device=q.device)
            ws = _ws(L_.sf_chain_workspace_bytes(ctypes.byref(sh), n, sl, ctypes.byref(tun)), q.device)
        else:
            dq, dk, dv, dg, dS_init, ws = out
    if ckpt is not None and (ckpt.device != q.device or not ckpt.is_contiguous()):
        raise ValueError("ckpt must be a contiguous buffer on the inputs' device")
    rc = L_.sf_chain_bwd(ctypes.byref(sh), n, sl, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(S_bnd), _ptr(ckpt),
                         ckpt.numel() * ckpt.element_size() if ckpt is not None else 0, _ptr(dO),
                         _ptr(dS_final), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dg), _ptr(dS_init), _ptr(ws),
                         ws.numel(), ctypes.byref(tun), _stream_handle(stream),
                         _stream_handle(aux) if aux is not None else None)
    _lib.check("sf_chain_bwd", rc)
    return dq, dk, dv, dg, dS_init


_ACT = {"none": _lib.SF_ACT_NONE, "silu": _lib.SF_ACT_SILU}


def _conv_shape(x, w, act):
    if x.dim() != 3:
        raise ValueError("x must be [B, L, C]")
    if x.dtype not in _IO:
        raise TypeError(f"unsupported I/O dtype {x.dtype}")
    if w.dim() != 2 or w.dtype != torch.float32 or not w.is_contiguous():
        raise ValueError("w must be a contiguous float32 [C, W] tensor")
    B, L, C = x.shape
    if w.shape[0] != C:
        raise ValueError(f"w has {w.shape[0]} channels, x has {C}")
    if x.stride(2) != 1:
        raise ValueError("x must have a contiguous channel dim")
    sh = _lib.SfConvShape()
    sh.B, sh.C, sh.L, sh.W = B, C, L, w.shape[1]
    sh.io_dtype = _IO[x.dtype]
    sh.act = _ACT[act]
    sh.sx_b, sh.sx_l = x.stride(0), x.stride(1)
    return sh


def _tail(t, B, W, C, name):
    if t is None or W == 1:
        return None
    if t.dtype != torch.float32 or tuple(t.shape) != (B, W - 1, C) or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous float32 [{B}, {W - 1}, {C}] tensor")
    return t


def conv_bwd_workspace_bytes(x, w, act="silu"):
    return _lib.lib().sf_conv_bwd_workspace_bytes(ctypes.byref(_conv_shape(x, w, act)))


def _out_like(t, ref, name):
    if tuple(t.shape) != tuple(ref.shape) or t.stride() != ref.stride() or t.dtype != ref.dtype:
        raise ValueError(f"{name} must match x in shape, strides and dtype")
    return t


def conv_fwd(x, w, tail_in=None, act="silu", *, stream=None, out=None, timing=None):
    """(y, tail_out) of the short convolution over one segment; tail_out is
    None for W = 1.  out=(y, tail_out) supplies the outputs (no allocation)."""
    sh = _conv_shape(x, w, act)
    B, L, C = x.shape
    W = w.shape[1]
    tail_in = _tail(tail_in, B, W, C, "tail_in")
    stream = stream or torch.cuda.current_stream(x.device)
    if out is not None:
        y, tail_out = _out_like(out[0], x, "y"), _tail(out[1], B, W, C, "tail_out")
    else:
        with torch.cuda.stream(stream):
            y = _like(x)
            tail_out = torch.empty((B, W - 1, C), dtype=torch.float32, device=x.device) if W > 1 else None
    rc = _lib.lib().sf_conv_fwd(ctypes.byref(sh), _ptr(x), _ptr(w), _ptr(tail_in), _ptr(y), _ptr(tail_out),
                                ctypes.byref(_tuning(timing=timing)), _stream_handle(stream))
    _lib.check("sf_conv_fwd", rc)
    return y, tail_out


def conv_bwd(x, w, tail_in, dy, dtail_out=None, act="silu", *, stream=None, out=None, timing=None):
    """(dx, dw, dtail_in) for the loss sum <dy, y> + <dtail_out, tail_out>;
    dtail_in is None for W = 1.  out=(dx, dw, dtail_in, workspace) supplies
    the outputs and a workspace of conv_bwd_workspace_bytes() (no allocation)."""
    sh = _conv_shape(x, w, act)
    B, L, C = x.shape
    W = w.shape[1]
    if tuple(dy.shape) != tuple(x.shape) or dy.stride() != x.stride() or dy.dtype != x.dtype:
        raise ValueError("dy must match x in shape, strides and dtype")
    tail_in = _tail(tail_in, B, W, C, "tail_in")
    dtail_out = _tail(dtail_out, B, W, C, "dtail_out")
    stream = stream or torch.cuda.current_stream(x.device)
    L_ = _lib.lib()
    if out is not None:
        dx, dw, dtail_in, ws = out
        _out_like(dx, x, "dx")
        dtail_in = _tail(dtail_in, B, W, C, "dtail_in")
        if tuple(dw.shape) != (C, W) or dw.dtype != torch.float32 or not dw.is_contiguous():
            raise ValueError("dw must be a contiguous float32 [C, W] tensor")
    else:
        with torch.cuda.stream(stream):
            dx = _like(x)
            dw = torch.empty((C, W), dtype=torch.float32, device=x.device)
            dtail_in = torch.empty((B, W - 1, C), dtype=torch.float32, device=x.device) if W > 1 else None
            ws = _ws(L_.sf_conv_bwd_workspace_bytes(ctypes.byref(sh)), x.device)
    rc = L_.sf_conv_bwd(ctypes.byref(sh), _ptr(x), _ptr(w), _ptr(tail_in), _ptr(dy), _ptr(dtail_out), _ptr(dx),
                        _ptr(dw), _ptr(dtail_in), _ptr(ws), ws.numel(), ctypes.byref(_tuning(timing=timing)),
                        _stream_handle(stream))
    _lib.check("sf_conv_bwd", rc)
    return dx, dw, dtail_in


def gdn_fwd(q, k, v, g, beta, S_in=None, *, ts=0, with_v_new=False, stream=None, timing=None):
    """(o, S_out) of the gated delta rule over one segment: q, k, v [B, L, H, D]
    bf16; g (natural-log decay) and beta float32 [B, L, H] with the same
    strides; S_in [B, H, D, D] float32 or None.  ts: superchunk length in
    tokens (a multiple of 64; 0 chooses).  with_v_new: also return the
    corrected values (V^new, laid out like v) as a third result."""
    _same_layout(q, k, v)
    sh = _shape(q, g)
    if tuple(beta.shape) != tuple(g.shape) or beta.stride() != g.stride() or beta.dtype != torch.float32:
        raise ValueError("beta must match g in shape, strides and dtype (float32)")
    B, L, H, D = q.shape
    _state(S_in, B, H, D, "S_in")
    stream = stream or torch.cuda.current_stream(q.device)
    L_ = _lib.lib()
    tun = _tuning(ts, timing=timing)
    with torch.cuda.stream(stream):
        o = _like(q)
        vn = _like(q) if with_v_new else None
        S_out = torch.empty((B, H, D, D), dtype=torch.float32, device=q.device)
        ws = _ws(L_.sf_gdn_fwd_workspace_bytes(ctypes.byref(sh), ctypes.byref(tun)), q.device)
    rc = L_.sf_gdn_fwd(ctypes.byref(sh), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S_in), _ptr(o),
                       _ptr(S_out), _ptr(vn), _ptr(ws), ws.numel(), ctypes.byref(tun), _stream_handle(stream))
    _lib.check("sf_gdn_fwd", rc)
    return (o, S_out, vn) if with_v_new else (o, S_out)


def gdn_bwd(q, k, v, g, beta, S_in, dO, dS_out=None, *, ts=0, stream=None, timing=None):
    """(dq, dk, dv, dg, dbeta, dS_in) of the gated delta rule over one segment
    for Loss = sum <dO, o> + <dS_out, S_out>; arguments as for gdn_fwd."""
    _same_layout(q, k, v, dO)
    sh = _shape(q, g)
    if tuple(beta.shape) != tuple(g.shape) or beta.stride() != g.stride() or beta.dtype != torch.float32:
        raise ValueError("beta must match g in shape, strides and dtype (float32)")
    B, L, H, D = q.shape
    _state(S_in, B, H, D, "S_in")
    _state(dS_out, B, H, D, "dS_out")
    stream = stream or torch.cuda.current_stream(q.device)
    L_ = _lib.lib()
    tun = _tuning(ts, timing=timing)
    with torch.cuda.stream(stream):
        dq, dk, dv = _like(q), _like(k), _like(v)
        dg, dbeta = _like(g), _like(beta)
        dS_in = torch.empty((B, H, D, D), dtype=torch.float32, device=q.device)
        ws = _ws(L_.sf_gdn_bwd_workspace_bytes(ctypes.byref(sh), ctypes.byref(tun)), q.device)
    rc = L_.sf_gdn_bwd(ctypes.byref(sh), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S_in), _ptr(dO),
                       _ptr(dS_out), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dg), _ptr(dbeta), _ptr(dS_in), _ptr(ws),
                       ws.numel(), ctypes.byref(tun), _stream_handle(stream))
    _lib.check("sf_gdn_bwd", rc)
    return dq, dk, dv, dg, dbeta, dS_in


def gdn_chain_ckpt_bytes(q, g, seg_lens, ts=0, overlap=True):
    """Bytes of the superchunk states and maps gdn_chain_fwd(keep_states=True) keeps."""
    sh = _shape(q, g)
    n = len(seg_lens)
    tun = _tuning(ts, overlap)
    sl = (ctypes.c_int64 * n)(*[int(x) for x in seg_lens])
    L_ = _lib.lib()
    nb = L_.sf_gdn_chain_ckpt_bytes(ctypes.byref(sh), n, sl, ctypes.byref(tun))
    if nb == 0 and L_.sf_last_error():
        raise StateflowError("sf_gdn_chain_ckpt_bytes: " + L_.sf_last_error().decode())
    return nb


def gdn_chain_fwd(q, k, v, g, beta, seg_lens, S_init=None, *, ts=0, overlap=True, with_v_new=False, stream=None,
                  aux_stream=None, timing=None, keep_states=False):
    """Gated-delta-rule forward over consecutive segments with
    S_in(i+1) = S_out(i), the state scans overlapped on an aux stream.

    Returns (o, S_bnd) (and V^new after them when with_v_new) with S_bnd[i] the
    state entering segment i and S_bnd[-1] the final state.  keep_states=True
    appends the kept superchunk states and maps (a uint8 device tensor) for
    gdn_chain_bwd(ckpt=...), which then skips replaying them."""
    _same_layout(q, k, v)
    sh = _shape(q, g)
    if tuple(beta.shape) != tuple(g.shape) or beta.stride() != g.stride() or beta.dtype != torch.float32:
        raise ValueError("beta must match g in shape, strides and dtype (float32)")
    B, L, H, D = q.shape
    n = len(seg_lens)
    _state(S_init, B, H, D, "S_init")
    stream = stream or torch.cuda.current_stream(q.device)
    aux = _aux_for(q.device, aux_stream, overlap)
    L_ = _lib.lib()
    tun = _tuning(ts, overlap, timing)
    sl = (ctypes.c_int64 * n)(*[int(x) for x in seg_lens])
    with torch.cuda.stream(stream):
        o = _like(q)
        vn = _like(q) if with_v_new else None
        S_bnd = torch.empty((n + 1, B, H, D, D), dtype=torch.float32, device=q.device)
        ws = _ws(L_.sf_gdn_chain_workspace_bytes(ctypes.byref(sh), n, sl, ctypes.byref(tun)), q.device)
        ck = _ws(L_.sf_gdn_chain_ckpt_bytes(ctypes.byref(sh), n, sl, ctypes.byref(tun)), q.device) \
            if keep_states else None
        if S_init is None:
            S_bnd[0].zero_()
        else:
            S_bnd[0].copy_(S_init)
    rc = L_.sf_gdn_chain_fwd(ctypes.byref(sh), n, sl, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(o),
                             _ptr(S_bnd), _ptr(ck), ck.numel() if ck is not None else 0, _ptr(vn), _ptr(ws),
                             ws.numel(), ctypes.byref(tun), _stream_handle(stream),
                             _stream_handle(aux) if aux is not None else None)
    _lib.check("sf_gdn_chain_fwd", rc)
    out = (o, S_bnd, vn) if with_v_new else (o, S_bnd)
    return out + (ck,) if keep_states else out


def gdn_chain_bwd(q, k, v, g, beta, seg_lens, S_bnd, dO, dS_final=None, *, ts=0, overlap=True, stream=None,
                  aux_stream=None, timing=None, ckpt=None):
    """Gated-delta-rule backward over the segments in reverse with
    dS_out(i) = dS_in(i+1); S_bnd from gdn_chain_fwd, ckpt its kept states
    (same inputs, segments and settings) or None.  Returns
    (dq, dk, dv, dg, dbeta, dS_init)."""
    _same_layout(q, k, v, dO)
    sh = _shape(q, g)
    if tuple(beta.shape) != tuple(g.shape) or beta.stride() != g.stride() or beta.dtype != torch.float32:
        raise ValueError("beta must match g in shape, strides and dtype (float32)")
    B, L, H, D = q.shape
    n = len(seg_lens)
    if tuple(S_bnd.shape) != (n + 1, B, H, D, D) or S_bnd.dtype != torch.float32 or not S_bnd.is_contiguous():
        raise ValueError("S_bnd must be a contiguous float32 [n_seg + 1, B, H, D, D] tensor")
    _state(dS_final, B, H, D, "dS_final")
    stream = stream or torch.cuda.current_stream(q.device)
    aux = _aux_for(q.device, aux_stream, overlap)
    L_ = _lib.lib()
    tun = _tuning(ts, overlap, timing)
    sl = (ctypes.c_int64 * n)(*[int(x) for x in seg_lens])
    with torch.cuda.stream(stream):
        dq, dk, dv = _like(q), _like(k), _like(v)
        dg, dbeta = _like(g), _like(beta)
        dS_init = torch.empty((B, H, D, D), dtype=torch.float32, device=q.device)
        ws = _ws(L_.sf_gdn_chain_workspace_bytes(ctypes.byref(sh), n, sl, ctypes.byref(tun)), q.device)
    if ckpt is not None and (ckpt.device != q.device or not ckpt.is_contiguous()):
        raise ValueError("ckpt must be a contiguous buffer on the inputs' device")
    rc = L_.sf_gdn_chain_bwd(ctypes.byref(sh), n, sl, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S_bnd),
                             _ptr(ckpt), ckpt.numel() * ckpt.element_size() if ckpt is not None else 0,
                             _ptr(dO), _ptr(dS_final), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dg), _ptr(dbeta),
                             _ptr(dS_init), _ptr(ws), ws.numel(), ctypes.byref(tun), _stream_handle(stream),
                             _stream_handle(aux) if aux is not None else None)
    _lib.check("sf_gdn_chain_bwd", rc)
    return dq, dk, dv, dg, dbeta, dS_init


def partition_hybrid(T, N, alpha, w_tok, w_soft, round_to=128):
    """Segment lengths of the hybrid-aware chunking (host-only, no GPU): N
    segments of a T-token sequence whose boundaries interpolate, by alpha,
    between equal lengths and the partition that equalises the per-segment
    cost w_tok * s + w_soft * (c * s + s^2 / 2)."""
    out = (ctypes.c_int64 * int(N))()
    _lib.check("sf_partition_hybrid", _lib.lib().sf_partition_hybrid(int(T), int(N), float(alpha), float(w_tok),
                                                                      float(w_soft), int(round_to), out))
    return [int(x) for x in out]
