"""ctypes binding of libstateflow (include/stateflow.h).

Argument marshalling only: every step of the recurrence runs in the HIP
kernels of libstateflow.so.  Importing this module fails loudly when the
library has not been built; there is no fallback path.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libstateflow.so")

SF_OK, SF_E_NULL, SF_E_SHAPE, SF_E_DTYPE, SF_E_ALIGN, SF_E_ALIAS, SF_E_WORKSPACE, \
    SF_E_UNSUPPORTED, SF_E_HIP = range(9)
SF_F32, SF_BF16 = 0, 1
SF_GATE_SCALAR, SF_GATE_VECTOR = 0, 1
# sf_kernel_id: the kernel kinds a timing record can select
KERNELS = {"fwd_prep": 0, "scan": 1, "fwd_out": 2, "bwd_prep": 3, "bwd_dq": 4, "bwd_dkv": 5,
           "conv_fwd": 6, "conv_bwd": 7, "gdn_prep": 8, "gdn_scan": 9, "gdn_out": 10, "gdn_store": 11,
           "gdn_dprep": 12, "gdn_dscan": 13, "gdn_dwalk": 14, "gdn_dchunk": 15}
SF_ACT_NONE, SF_ACT_SILU = 0, 1
NOALLOC_SCRATCH_BYTES = 64 << 20  # SF_NOALLOC_SCRATCH_BYTES

# every symbol include/stateflow.h declares
EXPORTS = ["sf_abi_version", "sf_status_str", "sf_last_error", "sf_fwd_workspace_bytes",
           "sf_bwd_workspace_bytes", "sf_segment_fwd", "sf_segment_fwd_noalloc", "sf_segment_bwd", "sf_chain_workspace_bytes",
           "sf_chain_ckpt_bytes", "sf_chain_fwd", "sf_chain_bwd", "sf_conv_bwd_workspace_bytes", "sf_conv_fwd", "sf_conv_bwd",
           "sf_gdn_fwd_workspace_bytes", "sf_gdn_fwd", "sf_gdn_bwd_workspace_bytes", "sf_gdn_bwd",
           "sf_gdn_chain_workspace_bytes", "sf_gdn_chain_ckpt_bytes", "sf_gdn_chain_fwd", "sf_gdn_chain_bwd",
           "sf_partition_hybrid"]


class SfShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("H", ctypes.c_int32), ("Dk", ctypes.c_int32),
                ("Dv", ctypes.c_int32), ("L", ctypes.c_int64), ("chunk", ctypes.c_int32),
                ("io_dtype", ctypes.c_int32), ("gate", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("sx_b", ctypes.c_int64), ("sx_l", ctypes.c_int64), ("sx_h", ctypes.c_int64),
                ("sg_b", ctypes.c_int64), ("sg_l", ctypes.c_int64), ("sg_h", ctypes.c_int64)]


class SfConvShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("C", ctypes.c_int32), ("L", ctypes.c_int64), ("W", ctypes.c_int32),
                ("io_dtype", ctypes.c_int32), ("act", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("sx_b", ctypes.c_int64), ("sx_l", ctypes.c_int64)]


class SfTiming(ctypes.Structure):
    _fields_ = [("mask", ctypes.c_uint32), ("capacity", ctypes.c_int32), ("count", ctypes.c_int32),
                ("dropped", ctypes.c_int32), ("start", ctypes.POINTER(ctypes.c_void_p)),
                ("stop", ctypes.POINTER(ctypes.c_void_p)), ("kind", ctypes.POINTER(ctypes.c_int32))]


class SfTuning(ctypes.Structure):
    _fields_ = [("ts", ctypes.c_int32), ("overlap", ctypes.c_int32),
                ("reserved", ctypes.c_int32 * 4), ("timing", ctypes.POINTER(SfTiming))]


class StateflowError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn} failed: {STATUS.get(status, status)}: {msg}")
        self.status = status


STATUS = {SF_OK: "SF_OK", SF_E_NULL: "SF_E_NULL", SF_E_SHAPE: "SF_E_SHAPE",
          SF_E_DTYPE: "SF_E_DTYPE", SF_E_ALIGN: "SF_E_ALIGN", SF_E_ALIAS: "SF_E_ALIAS",
          SF_E_WORKSPACE: "SF_E_WORKSPACE", SF_E_UNSUPPORTED: "SF_E_UNSUPPORTED",
          SF_E_HIP: "SF_E_HIP"}

_lib = None


def lib():
    """Load libstateflow.so (raises if it was not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2608_06838_amd/build.py "
                          "(or __graft_entry__.build()); there is no non-HIP fallback")
    L = ctypes.CDLL(LIB_PATH)
    vp, sp, tp = ctypes.c_void_p, ctypes.POINTER(SfShape), ctypes.POINTER(SfTuning)
    i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    i64p = ctypes.POINTER(ctypes.c_int64)
    L.sf_abi_version.restype = ctypes.c_int
    L.sf_abi_version.argtypes = []
    L.sf_status_str.restype = ctypes.c_char_p
    L.sf_status_str.argtypes = [ctypes.c_int]
    L.sf_last_error.restype = ctypes.c_char_p
    L.sf_last_error.argtypes = []
    for f in (L.sf_fwd_workspace_bytes, L.sf_bwd_workspace_bytes):
        f.restype = sz
        f.argtypes = [sp, tp]
    L.sf_segment_fwd.restype = ctypes.c_int
    L.sf_segment_fwd.argtypes = [sp] + [vp] * 8 + [sz, tp, vp]
    L.sf_segment_fwd_noalloc.restype = ctypes.c_int
    L.sf_segment_fwd_noalloc.argtypes = [sp] + [vp] * 7 + [tp, vp]
    L.sf_segment_bwd.restype = ctypes.c_int
    L.sf_segment_bwd.argtypes = [sp] + [vp] * 13 + [sz, tp, vp]
    L.sf_chain_workspace_bytes.restype = sz
    L.sf_chain_workspace_bytes.argtypes = [sp, i32, i64p, tp]
    L.sf_chain_fwd.restype = ctypes.c_int
    L.sf_chain_ckpt_bytes.restype = sz
    L.sf_chain_ckpt_bytes.argtypes = [sp, i32, i64p, tp]
    # (..., o, S_bnd, ckpt, ckpt_bytes, ws, ws_bytes, tuning, main, aux)
    L.sf_chain_fwd.argtypes = [sp, i32, i64p] + [vp] * 7 + [sz, vp, sz, tp, vp, vp]
    L.sf_chain_bwd.restype = ctypes.c_int
    # (..., g, S_bnd, ckpt, ckpt_bytes, dO, dS_final, dq, dk, dv, dg, dS_init, ws, ws_bytes, ...)
    L.sf_chain_bwd.argtypes = [sp, i32, i64p] + [vp] * 6 + [sz] + [vp] * 8 + [sz, tp, vp, vp]
    cp = ctypes.POINTER(SfConvShape)
    L.sf_conv_bwd_workspace_bytes.restype = sz
    L.sf_conv_bwd_workspace_bytes.argtypes = [cp]
    L.sf_conv_fwd.restype = ctypes.c_int
    L.sf_conv_fwd.argtypes = [cp] + [vp] * 5 + [tp, vp]
    L.sf_conv_bwd.restype = ctypes.c_int
    L.sf_conv_bwd.argtypes = [cp] + [vp] * 9 + [sz, tp, vp]
    L.sf_gdn_fwd_workspace_bytes.restype = sz
    L.sf_gdn_fwd_workspace_bytes.argtypes = [sp, tp]
    L.sf_gdn_fwd.restype = ctypes.c_int
    L.sf_gdn_fwd.argtypes = [sp] + [vp] * 10 + [sz, tp, vp]
    L.sf_gdn_bwd_workspace_bytes.restype = sz
    L.sf_gdn_bwd_workspace_bytes.argtypes = [sp, tp]
    L.sf_gdn_bwd.restype = ctypes.c_int
    L.sf_gdn_bwd.argtypes = [sp] + [vp] * 15 + [sz, tp, vp]
    L.sf_gdn_chain_workspace_bytes.restype = sz
    L.sf_gdn_chain_workspace_bytes.argtypes = [sp, i32, i64p, tp]
    L.sf_gdn_chain_fwd.restype = ctypes.c_int
    L.sf_gdn_chain_ckpt_bytes.restype = sz
    L.sf_gdn_chain_ckpt_bytes.argtypes = [sp, i32, i64p, tp]
    # (..., beta, o, S_bnd, ckpt, ckpt_bytes, v_new, ws, ws_bytes, tuning, main, aux)
    L.sf_gdn_chain_fwd.argtypes = [sp, i32, i64p] + [vp] * 8 + [sz] + [vp] * 2 + [sz, tp, vp, vp]
    L.sf_gdn_chain_bwd.restype = ctypes.c_int
    # (..., beta, S_bnd, ckpt, ckpt_bytes, dO, dS_final, dq, dk, dv, dg, dbeta, dS_init, ws, ws_bytes, ...)
    L.sf_gdn_chain_bwd.argtypes = [sp, i32, i64p] + [vp] * 7 + [sz] + [vp] * 9 + [sz, tp, vp, vp]
    L.sf_partition_hybrid.restype = ctypes.c_int
    L.sf_partition_hybrid.argtypes = [i64, i32, ctypes.c_double, ctypes.c_double, ctypes.c_double, i32, i64p]
    _lib = L
    return L


def check(fn, status):
    if status != SF_OK:
        raise StateflowError(fn, status, lib().sf_last_error().decode())
