"""Per-shape settings chosen by profiling (paper Sec. 3.2 "Optimal Chunk
Search" and the per-shape parameter choice of Sec. 3.4), passed to the library
as sf_tuning by the chain calls when the caller leaves ts / overlap unset.

The library itself keeps no tuning state; this table is data written from the
tuner's measurements (bench.py --tune-ts), one row per shape:
  key   (B, H, D, io, gate, segment lengths)
  value dict(ts=superchunk stride or 0 for the library's automatic choice,
             overlap=whether the state scans run on the aux stream)
Shapes without a row get ts = 0 and the paper's overlapped schedule.
"""

DEFAULT = dict(ts=0, overlap=True)

_SEG_256K = (65536, 40960, 32768, 28672, 26624, 24576, 22528, 20480)

# Filled from the measured study tables (tuner section).
TABLE = {}


def key(B, H, D, io, gate, seg_lens):
    return (int(B), int(H), int(D), str(io), str(gate), tuple(int(x) for x in seg_lens))


def lookup(B, H, D, io, gate, seg_lens):
    """The profiled setting for this shape, else DEFAULT (a copy)."""
    return dict(TABLE.get(key(B, H, D, io, gate, seg_lens), DEFAULT))


def choice(workload_name):
    """The setting for one of the named synthetic workloads."""
    from .synth import workload
    w = workload(workload_name)
    return lookup(w["B"], w["H"], w["D"], w["io"], w["gate"], w["seg_lens"])
