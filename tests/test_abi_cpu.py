"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, sizes workspaces, and rejects bad arguments before any launch."""
import ctypes
import os
import re

import pytest

from paper_2608_06838_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "stateflow.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sf_[a-z_]+)\s*\(", text)))


def shape(**kw):
    s = _lib.SfShape()
    s.B, s.H, s.Dk, s.Dv, s.L = 1, 2, 128, 128, 1024
    s.chunk, s.io_dtype, s.gate, s.reserved = 64, _lib.SF_BF16, _lib.SF_GATE_SCALAR, 0
    for k, v in kw.items():
        setattr(s, k, v)
    return s


def test_exports_every_declared_symbol():
    L = _lib.lib()
    declared = header_functions()
    assert set(declared) == set(_lib.EXPORTS), (declared, _lib.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name
    assert L.sf_abi_version() == 3
    assert L.sf_status_str(_lib.SF_E_ALIAS) == b"SF_E_ALIAS"


def test_workspace_sizes():
    L = _lib.lib()
    t = _lib.SfTuning()
    t.ts = 256
    s = shape(L=1024)
    n = 1024 // 256
    fwd = L.sf_fwd_workspace_bytes(ctypes.byref(s), ctypes.byref(t))
    bwd = L.sf_bwd_workspace_bytes(ctypes.byref(s), ctypes.byref(t))
    state = 2 * n * 128 * 128 * 4
    assert fwd >= state + 2 * n * 4
    assert bwd >= 2 * state + 2 * n * 4 + 2 * n * 64 * 4
    t.ts = 1024  # one superchunk: the walkers start from S_in directly
    assert L.sf_fwd_workspace_bytes(ctypes.byref(s), ctypes.byref(t)) == 0
    assert 0 < L.sf_bwd_workspace_bytes(ctypes.byref(s), ctypes.byref(t)) <= 4096
    # invalid shapes size to 0
    assert L.sf_fwd_workspace_bytes(ctypes.byref(shape(L=100)), None) == 0
    assert L.sf_fwd_workspace_bytes(None, None) == 0
    segs = (ctypes.c_int64 * 3)(512, 256, 256)
    assert L.sf_chain_workspace_bytes(ctypes.byref(s), 3, segs, None) > 0
    bad = (ctypes.c_int64 * 3)(512, 256, 128)
    assert L.sf_chain_workspace_bytes(ctypes.byref(s), 3, bad, None) == 0


FAKE = 0x7F0000000000  # never dereferenced: every case below fails validation first


def p(i):
    return ctypes.c_void_p(FAKE + i * (1 << 32))


def _tuning(ts=0):
    t = _lib.SfTuning()
    t.ts = ts
    return t


def fwd(s, q=1, k=2, v=3, g=4, S_in=None, o=5, S_out=6, ws=7, ws_bytes=1 << 30, tun=None):
    L = _lib.lib()
    args = [p(x) if x is not None else None for x in (q, k, v, g, S_in, o, S_out, ws)]
    return L.sf_segment_fwd(ctypes.byref(s) if s is not None else None, *args, ws_bytes,
                            ctypes.byref(tun) if tun is not None else None, None)


@pytest.mark.parametrize("kw,status", [
    (dict(L=100), _lib.SF_E_SHAPE),
    (dict(B=0), _lib.SF_E_SHAPE),
    (dict(Dk=96, Dv=96), _lib.SF_E_UNSUPPORTED),
    (dict(Dk=128, Dv=64), _lib.SF_E_UNSUPPORTED),
    (dict(chunk=32), _lib.SF_E_UNSUPPORTED),
    (dict(io_dtype=7), _lib.SF_E_DTYPE),
    (dict(gate=5), _lib.SF_E_DTYPE),
    (dict(io_dtype=_lib.SF_F32, Dk=128, Dv=128, gate=_lib.SF_GATE_VECTOR), _lib.SF_E_UNSUPPORTED),
    (dict(reserved=1), _lib.SF_E_SHAPE),
    (dict(sx_b=1024 * 2 * 128, sx_l=100, sx_h=128), _lib.SF_E_SHAPE),   # rows overlap
    (dict(sx_b=1024 * 2 * 136, sx_l=2 * 136, sx_h=132), _lib.SF_E_ALIGN),  # 264-byte head stride
    # a 64-token chunk spanning >= 2 GiB (the kernels address chunks with 32-bit offsets)
    (dict(sx_b=1024 * (1 << 25), sx_l=1 << 25, sx_h=128), _lib.SF_E_SHAPE),
])
def test_shape_validation(kw, status):
    assert fwd(shape(**kw)) == status
    assert _lib.lib().sf_last_error() != b""


def test_fp32_d128_scalar_gate_accepted():
    """fp32 I/O at d = 128 takes the scalar gate: validation passes up to the
    workspace check (no launch: a too-small workspace is reported)."""
    t = _lib.SfTuning()
    t.ts = 128
    s = shape(io_dtype=_lib.SF_F32, Dk=128, Dv=128)
    assert fwd(s, ws_bytes=16, tun=t) == _lib.SF_E_WORKSPACE
    assert _lib.lib().sf_fwd_workspace_bytes(ctypes.byref(s), ctypes.byref(t)) > 0


def test_pointer_validation():
    s = shape()
    assert fwd(None) == _lib.SF_E_NULL
    assert fwd(s, q=None) == _lib.SF_E_NULL
    assert fwd(s, S_out=None) == _lib.SF_E_NULL
    # misaligned pointer
    L = _lib.lib()
    rc = L.sf_segment_fwd(ctypes.byref(s), ctypes.c_void_p(FAKE + 2), p(2), p(3), p(4), None, p(5), p(6),
                          p(7), 1 << 30, None, None)
    assert rc == _lib.SF_E_ALIGN
    # output overlapping an input
    assert fwd(s, o=1) == _lib.SF_E_ALIAS
    assert fwd(s, S_out=5) == _lib.SF_E_ALIAS  # S_out inside o
    # workspace too small
    t = _lib.SfTuning()
    t.ts = 128
    assert fwd(s, ws_bytes=16, tun=t) == _lib.SF_E_WORKSPACE
    assert fwd(s, ws=None, tun=t) == _lib.SF_E_NULL
    t.ts = 100
    assert fwd(s, tun=t) == _lib.SF_E_SHAPE


def test_workspace_alias():
    """The workspace is an output: it may overlap no input and no other output
    (segment and chain calls, both directions)."""
    L = _lib.lib()
    t = _tuning(ts=128)  # several superchunks: the calls need a workspace
    s = shape()
    assert fwd(s, ws=5, tun=t) == _lib.SF_E_ALIAS   # over o
    assert fwd(s, ws=1, tun=t) == _lib.SF_E_ALIAS   # over q
    assert fwd(s, ws=6, tun=t) == _lib.SF_E_ALIAS   # over S_out

    def bwd(ws, dq=8):
        args = [p(i) for i in (1, 2, 3, 4)] + [None, p(6), None] + [p(i) for i in (dq, 9, 10, 11, 12, ws)]
        return L.sf_segment_bwd(ctypes.byref(s), *args, 1 << 30, ctypes.byref(t), None)

    assert bwd(ws=8) == _lib.SF_E_ALIAS      # over dq
    assert bwd(ws=6) == _lib.SF_E_ALIAS      # over dO
    assert bwd(ws=12) == _lib.SF_E_ALIAS     # over dS_in
    segs = (ctypes.c_int64 * 2)(512, 512)
    rc = L.sf_chain_fwd(ctypes.byref(s), 2, segs, p(1), p(2), p(3), p(4), p(5), p(6), None, 0, p(5), 1 << 30, None,
                        None, None)
    assert rc == _lib.SF_E_ALIAS             # workspace over o
    rc = L.sf_chain_fwd(ctypes.byref(s), 2, segs, p(1), p(2), p(3), p(4), p(5), p(6), None, 0, p(6), 1 << 30, None,
                        None, None)
    assert rc == _lib.SF_E_ALIAS             # workspace over S_bnd
    rc = L.sf_chain_bwd(ctypes.byref(s), 2, segs, p(1), p(2), p(3), p(4), p(5), None, 0, p(6), None, p(8), p(9),
                        p(10), p(11), p(12), p(8), 1 << 30, None, None, None)
    assert rc == _lib.SF_E_ALIAS             # workspace over dq
    rc = L.sf_chain_bwd(ctypes.byref(s), 2, segs, p(1), p(2), p(3), p(4), p(5), None, 0, p(6), None, p(8), p(9),
                        p(10), p(11), p(12), p(5), 1 << 30, None, None, None)
    assert rc == _lib.SF_E_ALIAS             # workspace over S_bnd (an input of the backward)


def test_chain_ckpt():
    """Kept superchunk states: sizing, and the buffer is an output of the
    forward and an input of the backward (alias and size checks)."""
    L = _lib.lib()
    t = _tuning(ts=128)
    s = shape(L=1024)
    segs = (ctypes.c_int64 * 3)(512, 384, 128)  # 4, 3 and 1 superchunks
    SS, bh = 128 * 128 * 4, 2

    def al(x):
        return (x + 255) // 256 * 256

    def seg(n):
        return al(bh * n * SS) + al(bh * n * 4) + al(bh * SS) if n > 1 else 0

    need = L.sf_chain_ckpt_bytes(ctypes.byref(s), 3, segs, ctypes.byref(t))
    assert need == seg(4) + seg(3) + seg(1)
    one = (ctypes.c_int64 * 1)(1024)
    t1 = _tuning(ts=1024)
    assert L.sf_chain_ckpt_bytes(ctypes.byref(s), 1, one, ctypes.byref(t1)) == 0
    vs = shape(L=1024, gate=_lib.SF_GATE_VECTOR)
    assert L.sf_chain_ckpt_bytes(ctypes.byref(vs), 3, segs, ctypes.byref(t)) == \
        sum(al(bh * n * SS) + al(bh * n * 128 * 4) + al(bh * SS) for n in (4, 3))
    bad = (ctypes.c_int64 * 3)(512, 384, 64)
    assert L.sf_chain_ckpt_bytes(ctypes.byref(s), 3, bad, ctypes.byref(t)) == 0
    assert L.sf_last_error()
    tp = ctypes.byref(t)

    def fwd(ck, nb=1 << 30, ws=7):
        return L.sf_chain_fwd(ctypes.byref(s), 3, segs, p(1), p(2), p(3), p(4), p(5), p(6), ck, nb, p(ws), 1 << 30,
                              tp, None, None)

    assert fwd(p(5)) == _lib.SF_E_ALIAS             # over o
    assert fwd(p(6)) == _lib.SF_E_ALIAS             # over S_bnd
    assert fwd(p(7)) == _lib.SF_E_ALIAS             # over the workspace
    assert fwd(p(1)) == _lib.SF_E_ALIAS             # over q
    assert fwd(p(8), nb=need - 1) == _lib.SF_E_WORKSPACE
    assert fwd(ctypes.c_void_p(p(8).value + 4)) == _lib.SF_E_ALIGN

    def bwd(ck, nb=1 << 30, dq=8):
        return L.sf_chain_bwd(ctypes.byref(s), 3, segs, p(1), p(2), p(3), p(4), p(5), ck, nb, p(6), None,
                              p(dq), p(9), p(10), p(11), p(12), p(13), 1 << 30, tp, None, None)

    assert bwd(p(8)) == _lib.SF_E_ALIAS             # over dq
    assert bwd(p(13)) == _lib.SF_E_ALIAS            # over the workspace
    assert bwd(p(14), nb=need - 256) == _lib.SF_E_WORKSPACE


def test_chain_validation():
    L = _lib.lib()
    s = shape(L=1024)
    segs = (ctypes.c_int64 * 2)(512, 448)   # sums to 960
    rc = L.sf_chain_fwd(ctypes.byref(s), 2, segs, p(1), p(2), p(3), p(4), p(5), p(6), None, 0, p(7), 1 << 30, None,
                        None, None)
    assert rc == _lib.SF_E_SHAPE
    segs = (ctypes.c_int64 * 2)(512, 512)
    rc = L.sf_chain_fwd(ctypes.byref(s), 0, segs, p(1), p(2), p(3), p(4), p(5), p(6), None, 0, p(7), 1 << 30, None,
                        None, None)
    assert rc == _lib.SF_E_SHAPE
    rc = L.sf_chain_bwd(ctypes.byref(s), 2, segs, p(1), p(2), p(3), p(4), p(5), None, 0, p(6), None, p(8), p(9),
                        p(10), p(11), None, p(13), 1 << 30, None, None, None)
    assert rc == _lib.SF_E_NULL  # dS_init missing


def test_overlap_mode_validation():
    """tuning.overlap takes 0, 1 or 2; anything else is rejected before any launch."""
    L = _lib.lib()
    s = shape()
    segs = (ctypes.c_int64 * 2)(512, 512)
    for bad in (-1, 3):
        t = _tuning()
        t.overlap = bad
        assert fwd(s, tun=t) == _lib.SF_E_SHAPE
        rc = L.sf_chain_fwd(ctypes.byref(s), 2, segs, p(1), p(2), p(3), p(4), p(5), p(6), None, 0, p(7), 1 << 30,
                            ctypes.byref(t), None, None)
        assert rc == _lib.SF_E_SHAPE
    import paper_2608_06838_amd as sf
    assert sf._overlap_mode(True) == 1 and sf._overlap_mode(False) == 0 and sf._overlap_mode(2) == 2
    with pytest.raises(ValueError):
        sf._overlap_mode(3)


def test_timing_validation():
    """A caller's timing record is checked before any launch."""
    tm = _lib.SfTiming()
    t = _tuning()
    t.timing = ctypes.pointer(tm)
    s = shape()
    tm.capacity, tm.count = 4, 5
    assert fwd(s, tun=t) == _lib.SF_E_SHAPE      # count beyond capacity
    tm.capacity, tm.count = -1, 0
    assert fwd(s, tun=t) == _lib.SF_E_SHAPE
    tm.capacity, tm.count = 4, 0
    assert fwd(s, tun=t) == _lib.SF_E_NULL       # no event arrays
    assert conv_fwd(conv_shape(), tun=t) == _lib.SF_E_NULL


# ------------------------------------------------------------ short convolution
def conv_shape(**kw):
    s = _lib.SfConvShape()
    s.B, s.C, s.L, s.W, s.io_dtype, s.act, s.reserved = 2, 64, 1000, 4, _lib.SF_BF16, _lib.SF_ACT_SILU, 0
    for k, v in kw.items():
        setattr(s, k, v)
    return s


def conv_fwd(s, x=1, w=2, tail_in=3, y=4, tail_out=5, tun=None):
    args = [p(i) if i is not None else None for i in (x, w, tail_in, y, tail_out)]
    return _lib.lib().sf_conv_fwd(ctypes.byref(s) if s is not None else None, *args,
                                  ctypes.byref(tun) if tun is not None else None, None)


def conv_bwd(s, x=1, w=2, tail_in=3, dy=4, dtail_out=5, dx=6, dw=7, dtail_in=8, ws=9, ws_bytes=1 << 30):
    args = [p(i) if i is not None else None for i in (x, w, tail_in, dy, dtail_out, dx, dw, dtail_in, ws)]
    return _lib.lib().sf_conv_bwd(ctypes.byref(s), *args, ws_bytes, None, None)


def test_conv_workspace_bytes():
    L = _lib.lib()
    # 1000 tokens: blocks of 256, 4 partials per batch of C * W floats
    assert L.sf_conv_bwd_workspace_bytes(ctypes.byref(conv_shape())) == 2 * 4 * 64 * 4 * 4
    # 262144 tokens: the block grows to 1024 so that 256 partials per batch remain
    assert L.sf_conv_bwd_workspace_bytes(ctypes.byref(conv_shape(B=1, L=262144, C=5120))) == 256 * 5120 * 4 * 4
    assert L.sf_conv_bwd_workspace_bytes(ctypes.byref(conv_shape(L=0))) == 0
    assert L.sf_conv_bwd_workspace_bytes(ctypes.byref(conv_shape(C=12))) == 0
    assert L.sf_conv_bwd_workspace_bytes(None) == 0


@pytest.mark.parametrize("kw,status", [
    (dict(B=0), _lib.SF_E_SHAPE),
    (dict(L=-1), _lib.SF_E_SHAPE),
    (dict(C=12), _lib.SF_E_UNSUPPORTED),
    (dict(W=5), _lib.SF_E_UNSUPPORTED),
    (dict(W=0), _lib.SF_E_UNSUPPORTED),
    (dict(io_dtype=7), _lib.SF_E_DTYPE),
    (dict(act=3), _lib.SF_E_DTYPE),
    (dict(reserved=1), _lib.SF_E_SHAPE),
    (dict(sx_b=1000 * 64, sx_l=32), _lib.SF_E_SHAPE),          # rows overlap
    (dict(sx_b=1000 * 68, sx_l=68), _lib.SF_E_ALIGN),          # 136-byte rows
])
def test_conv_shape_validation(kw, status):
    assert conv_fwd(conv_shape(**kw)) == status
    assert _lib.lib().sf_last_error() != b""


def test_conv_pointer_validation():
    s = conv_shape()
    assert conv_fwd(None) == _lib.SF_E_NULL
    assert conv_fwd(s, x=None) == _lib.SF_E_NULL
    assert conv_fwd(s, w=None) == _lib.SF_E_NULL
    rc = _lib.lib().sf_conv_fwd(ctypes.byref(s), ctypes.c_void_p(FAKE + 8), p(2), p(3), p(4), p(5), None, None)
    assert rc == _lib.SF_E_ALIGN
    assert conv_fwd(s, y=1) == _lib.SF_E_ALIAS          # y over x
    assert conv_fwd(s, tail_out=2) == _lib.SF_E_ALIAS   # tail_out over w
    assert conv_bwd(s, dw=None) == _lib.SF_E_NULL
    assert conv_bwd(s, ws_bytes=16) == _lib.SF_E_WORKSPACE
    assert conv_bwd(s, ws=None) == _lib.SF_E_WORKSPACE
    assert conv_bwd(s, dx=4) == _lib.SF_E_ALIAS         # dx over dy
    assert conv_bwd(s, dtail_in=9) == _lib.SF_E_ALIAS   # dtail_in inside the workspace


# ------------------------------------------------------------ gated delta rule
def test_gdn_validation():
    L = _lib.lib()

    def call(s, q=1, k=2, v=3, g=4, beta=5, S_in=None, o=6, S_out=7, v_new=None, ws=8, ws_bytes=1 << 30, tun=None):
        args = [p(i) if i is not None else None for i in (q, k, v, g, beta, S_in, o, S_out, v_new, ws)]
        return L.sf_gdn_fwd(ctypes.byref(s) if s is not None else None, *args, ws_bytes,
                            ctypes.byref(tun) if tun is not None else None, None)

    assert call(None) == _lib.SF_E_NULL
    assert call(shape(io_dtype=_lib.SF_F32, Dk=64, Dv=64)) == _lib.SF_E_UNSUPPORTED
    assert call(shape(gate=_lib.SF_GATE_VECTOR)) == _lib.SF_E_UNSUPPORTED
    assert call(shape(L=100)) == _lib.SF_E_SHAPE
    assert call(shape(), beta=None) == _lib.SF_E_NULL
    assert call(shape(), S_out=None) == _lib.SF_E_NULL
    assert call(shape(), o=1) == _lib.SF_E_ALIAS
    assert call(shape(), S_out=5) == _lib.SF_E_ALIAS   # S_out over beta
    assert call(shape(), ws=6) == _lib.SF_E_ALIAS      # workspace over o
    assert call(shape(), v_new=3) == _lib.SF_E_ALIAS   # V^new over v
    assert call(shape(), v_new=6) == _lib.SF_E_ALIAS   # V^new over o
    rc = L.sf_gdn_fwd(ctypes.byref(shape()), ctypes.c_void_p(FAKE + 2), p(2), p(3), p(4), p(5), None, p(6), p(7),
                      None, p(8), 1 << 30, None, None)
    assert rc == _lib.SF_E_ALIGN
    # superchunks: ts must be a positive multiple of 64; the workspace holds
    # S_J for every superchunk and (M_J, N_J) for all but the last
    assert call(shape(), tun=_tuning(ts=100)) == _lib.SF_E_SHAPE
    s = shape(L=1024)
    need = L.sf_gdn_fwd_workspace_bytes(ctypes.byref(s), ctypes.byref(_tuning(ts=256)))
    assert need == 2 * 4 * 128 * 128 * 4 + 2 * (2 * 3 * 128 * 128 * 4)
    assert L.sf_gdn_fwd_workspace_bytes(ctypes.byref(s), ctypes.byref(_tuning(ts=1024))) == 0
    assert L.sf_gdn_fwd_workspace_bytes(ctypes.byref(s), ctypes.byref(_tuning(ts=4096))) == 0
    assert call(s, tun=_tuning(ts=256), ws=None) == _lib.SF_E_NULL
    assert call(s, tun=_tuning(ts=256), ws_bytes=need - 1) == _lib.SF_E_WORKSPACE
    assert call(s, tun=_tuning(ts=1024), ws=None, ws_bytes=0, S_out=1) == _lib.SF_E_ALIAS  # passes the workspace checks


def test_gdn_bwd_validation():
    L = _lib.lib()

    def call(s, q=1, k=2, v=3, g=4, beta=5, S_in=None, dO=6, dS_out=None, dq=7, dk=8, dv=9, dg=10, dbeta=11,
             dS_in=12, ws=13, ws_bytes=1 << 40, tun=None):
        args = [p(i) if i is not None else None
                for i in (q, k, v, g, beta, S_in, dO, dS_out, dq, dk, dv, dg, dbeta, dS_in, ws)]
        return L.sf_gdn_bwd(ctypes.byref(s) if s is not None else None, *args, ws_bytes,
                            ctypes.byref(tun) if tun is not None else None, None)

    assert call(None) == _lib.SF_E_NULL
    assert call(shape(io_dtype=_lib.SF_F32, Dk=64, Dv=64)) == _lib.SF_E_UNSUPPORTED
    assert call(shape(gate=_lib.SF_GATE_VECTOR)) == _lib.SF_E_UNSUPPORTED
    assert call(shape(L=100)) == _lib.SF_E_SHAPE
    assert call(shape(), dO=None) == _lib.SF_E_NULL
    assert call(shape(), dS_in=None) == _lib.SF_E_NULL
    assert call(shape(), dbeta=None) == _lib.SF_E_NULL
    assert call(shape(), dq=1) == _lib.SF_E_ALIAS       # dq over q
    assert call(shape(), dk=6) == _lib.SF_E_ALIAS       # dk over dO
    assert call(shape(), ws=7) == _lib.SF_E_ALIAS       # workspace over dq
    assert call(shape(), ws=None) == _lib.SF_E_NULL
    assert call(shape(), tun=_tuning(ts=96)) == _lib.SF_E_SHAPE
    # workspace: states and state gradients of every chunk, the maps of every
    # superchunk, E_J (all but the first) and dS_end(J)
    s, n, nc, SS = shape(L=1024), 4, 16, 128 * 128 * 4
    need = L.sf_gdn_bwd_workspace_bytes(ctypes.byref(s), ctypes.byref(_tuning(ts=256)))
    assert need == 2 * SS * (4 * n + (n - 1)) + 2 * (2 * nc * SS)
    assert call(s, tun=_tuning(ts=256), ws_bytes=need - 1) == _lib.SF_E_WORKSPACE


def test_gdn_chain_validation():
    L = _lib.lib()
    segs = (ctypes.c_int64 * 3)(256, 512, 256)

    def fwd(s, n=3, sl=segs, q=1, k=2, v=3, g=4, beta=5, o=6, S_bnd=7, v_new=None, ws=8, ws_bytes=1 << 40,
            ck=None, ck_bytes=1 << 40, tun=None):
        a1 = [p(i) if i is not None else None for i in (q, k, v, g, beta, o, S_bnd)]
        a2 = [p(i) if i is not None else None for i in (v_new, ws)]
        return L.sf_gdn_chain_fwd(ctypes.byref(s), n, sl, *a1, p(ck) if ck else None, ck_bytes, *a2, ws_bytes,
                                  tun, None, None)

    def bwd(s, n=3, sl=segs, dq=9, dS_init=14, ws=15, ck=None, ck_bytes=1 << 40, tun=None):
        a1 = [p(i) for i in (1, 2, 3, 4, 5, 7)]
        a2 = [p(i) if i is not None else None for i in (6, None, dq, 10, 11, 12, 13, dS_init, ws)]
        return L.sf_gdn_chain_bwd(ctypes.byref(s), n, sl, *a1, p(ck) if ck else None, ck_bytes, *a2, 1 << 40,
                                  tun, None, None)

    s = shape(L=1024)
    assert fwd(s, n=0) == _lib.SF_E_SHAPE
    assert fwd(shape(L=1000)) == _lib.SF_E_SHAPE
    assert fwd(s, sl=(ctypes.c_int64 * 3)(256, 500, 268)) == _lib.SF_E_SHAPE   # not multiples of 64
    assert fwd(s, sl=(ctypes.c_int64 * 3)(256, 512, 128)) == _lib.SF_E_SHAPE   # sum != L
    assert fwd(s, beta=None) == _lib.SF_E_NULL
    assert fwd(s, o=1) == _lib.SF_E_ALIAS
    assert fwd(s, ws_bytes=16) == _lib.SF_E_WORKSPACE
    assert fwd(shape(L=1024, gate=_lib.SF_GATE_VECTOR)) == _lib.SF_E_UNSUPPORTED
    assert bwd(s, dq=2) == _lib.SF_E_ALIAS
    assert bwd(s, dS_init=None) == _lib.SF_E_NULL
    need = L.sf_gdn_chain_workspace_bytes(ctypes.byref(s), 3, segs, None)
    assert need > 0
    assert L.sf_gdn_chain_workspace_bytes(ctypes.byref(s), 3, (ctypes.c_int64 * 3)(256, 512, 128), None) == 0
    # kept states: S_J and M_J of each segment of more than one superchunk
    t = _tuning(ts=128)
    SS, bh = 128 * 128 * 4, 2
    kneed = L.sf_gdn_chain_ckpt_bytes(ctypes.byref(s), 3, segs, ctypes.byref(t))
    assert kneed == sum(2 * ((bh * n * SS + 255) // 256 * 256) for n in (2, 4, 2))
    # one superchunk per segment: nothing to keep
    assert L.sf_gdn_chain_ckpt_bytes(ctypes.byref(s), 3, segs, ctypes.byref(_tuning(ts=512))) == 0
    assert L.sf_gdn_chain_ckpt_bytes(ctypes.byref(s), 3, (ctypes.c_int64 * 3)(256, 512, 128), ctypes.byref(t)) == 0
    tp = ctypes.byref(t)
    assert fwd(s, ck=6, tun=tp) == _lib.SF_E_ALIAS        # over o
    assert fwd(s, ck=8, tun=tp) == _lib.SF_E_ALIAS        # over the workspace
    assert fwd(s, ck=16, ck_bytes=kneed - 1, tun=tp) == _lib.SF_E_WORKSPACE
    assert bwd(s, ck=9, tun=tp) == _lib.SF_E_ALIAS        # over dq
    assert bwd(s, ck=16, ck_bytes=kneed - 256, tun=tp) == _lib.SF_E_WORKSPACE
