"""Per-shape settings chosen by profiling (paper Sec. 3.2 "Optimal Chunk
Search" and the per-shape parameter choice of Sec. 3.4), passed to the library
as sf_tuning by the chain calls when the caller leaves ts / overlap unset.

The library itself keeps no tuning state; this table is data written from the
tuner's measurements (bench.py --tune-ts), one row per shape:
  key   (B, H, D, io, gate, segment lengths)
  value dict(ts=superchunk stride or 0 for the library's automatic choice,
             overlap=0: serial on the main stream, 1: the state scans on the
             aux stream, 2: each segment's preparation kernel and its scan
             on the aux stream)
Shapes without a row get ts = 0 (the library's cost model, fitted to these
same measurements) and the scans serialised on the main stream: on every
measured shape the serial schedule was as fast as the scans-only overlap or
faster (the dense kernels keep every CU busy, so an overlapped scan only
slows the kernel it shares a CU with).  With the preparation kernels on the
aux stream too (overlap=2), Pre and ST of one segment fill the tails of the
neighbouring segment's dense kernels: that pays on the mid layer (its
launches are a fraction of a round of workgroups) and loses on the 256K layer
and the vector gate.  overlap=1 is the paper's split-and-overlap schedule.
"""

DEFAULT = dict(ts=0, overlap=False)

_SEG_256K = (65536, 40960, 32768, 28672, 26624, 24576, 22528, 20480)

# Profiled on MI355X (bench.py --tune-ts, fwd+bwd chain steps, best of the
# ts x overlap-mode grid).  ts = 0 where the library's per-segment choice beat
# every fixed stride.
TABLE = {
    (1, 2, 64, "f32", "scalar", (1024,)): dict(ts=0, overlap=False),
    (1, 16, 128, "bf16", "scalar", (4096,) * 8): dict(ts=256, overlap=2),
    (1, 40, 128, "bf16", "scalar", _SEG_256K): dict(ts=0, overlap=False),
    (2, 16, 128, "bf16", "vector", (4096,) * 16): dict(ts=512, overlap=False),
    (4, 32, 128, "bf16", "scalar", (512,) * 32): dict(ts=512, overlap=False),
}


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
