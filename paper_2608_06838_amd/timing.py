"""Per-kernel timing for measurement: a caller-owned sf_timing record.

The library keeps no timing state of its own.  A KernelTimer owns HIP events
(created through the HIP runtime that torch already loaded) and the record
that points at them; passing it as `timing=` to a call makes every launch of
the selected kernel kinds take one event pair as the begin and end timestamps
of its own dispatch.  read() synchronises the used events, returns the summed
milliseconds and launch count per kernel kind, and frees the pairs for reuse.
"""
import ctypes

from . import _lib

_hip = None


def _hip_rt():
    global _hip
    if _hip is None:
        import torch  # noqa: F401  (loads the HIP runtime)
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        _hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        _hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        _hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        for f in (_hip.hipEventCreate, _hip.hipEventDestroy, _hip.hipEventSynchronize, _hip.hipEventElapsedTime):
            f.restype = ctypes.c_int
    return _hip


def _ok(rc, what):
    if rc != 0:
        raise RuntimeError(f"{what} failed with HIP error {rc}")


class KernelTimer:
    """Event pairs for up to `capacity` timed launches of the kernel kinds in
    `kernels` (names of paper_2608_06838_amd.KERNELS)."""

    def __init__(self, kernels=(), capacity=2048):
        hip = _hip_rt()
        self.capacity = int(capacity)
        self._start = (ctypes.c_void_p * self.capacity)()
        self._stop = (ctypes.c_void_p * self.capacity)()
        self._kind = (ctypes.c_int32 * self.capacity)()
        for arr in (self._start, self._stop):
            for i in range(self.capacity):
                ev = ctypes.c_void_p()
                _ok(hip.hipEventCreate(ctypes.byref(ev)), "hipEventCreate")
                arr[i] = ev.value
        self.rec = _lib.SfTiming()
        self.rec.capacity = self.capacity
        self.rec.start = ctypes.cast(self._start, ctypes.POINTER(ctypes.c_void_p))
        self.rec.stop = ctypes.cast(self._stop, ctypes.POINTER(ctypes.c_void_p))
        self.rec.kind = ctypes.cast(self._kind, ctypes.POINTER(ctypes.c_int32))
        self.select(kernels)

    def select(self, kernels):
        """Time the launches of these kernel kinds from now on (names)."""
        mask = 0
        for k in kernels:
            mask |= 1 << _lib.KERNELS[k]
        self.rec.mask = mask

    def read(self):
        """{kernel name: (total ms, launches)} of the pairs used since the last
        read (waits for those launches to finish), then frees the pairs."""
        hip = _hip_rt()
        names = {v: k for k, v in _lib.KERNELS.items()}
        out = {}
        for i in range(self.rec.count):
            _ok(hip.hipEventSynchronize(self._stop[i]), "hipEventSynchronize")
            ms = ctypes.c_float()
            _ok(hip.hipEventElapsedTime(ctypes.byref(ms), self._start[i], self._stop[i]), "hipEventElapsedTime")
            name = names[self._kind[i]]
            t, n = out.get(name, (0.0, 0))
            out[name] = (t + ms.value, n + 1)
        if self.rec.dropped:
            raise RuntimeError(f"{self.rec.dropped} timed launches found no free event pair "
                               f"(capacity {self.capacity})")
        self.rec.count = 0
        return out

    def close(self):
        hip = _hip_rt()
        for arr in (self._start, self._stop):
            for i in range(self.capacity):
                if arr[i]:
                    hip.hipEventDestroy(arr[i])
                    arr[i] = None
