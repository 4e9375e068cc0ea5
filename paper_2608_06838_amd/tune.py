"""Profile-guided selection of the chain's tuning knobs (paper Sec. 3.2,
"Optimal Chunk Search", and the per-shape kernel parameter choice of Sec. 3.4).

The paper picks, per shape, the fastest of a small grid of candidates by timing
them; FLOP models alone miss kernel efficiency and memory behaviour.  Here the
knobs are those of this implementation:

  * ts, the state-materialisation stride (superchunk length) of the scans,
    and whether the scans overlap the dense kernels on the aux stream;
  * the segment lengths of a sequence: N segments whose boundaries
    interpolate by alpha between equal lengths and the FLOP-balanced hybrid
    partition (sf_partition_hybrid).

Everything here is selection logic around a caller-supplied timer; the timed
work is the library's own chain (see bench.py --tune-ts and
--partition-study).  Candidates that fail (for instance a partition whose
rounding leaves a segment empty, or one over a memory limit) are reported and
skipped.
"""
import math

from . import partition_hybrid

# the paper's grids for the partition search
PARTITION_NS = (2, 4, 6, 8, 16, 32)
PARTITION_ALPHAS = (0.0, 0.1, 0.2, 0.3, 0.4, 0.5, 0.6, 0.7, 0.8, 0.9, 1.0, 1.25)


def ts_candidates(seg_lens, extra=(128, 256, 512, 1024, 2048, 4096, 8192)):
    """0 (the library's automatic choice) and fixed strides that fit the
    longest segment, each a multiple of 64."""
    longest = max(seg_lens)
    return [0] + [t for t in extra if t % 64 == 0 and t <= longest]


def partition_candidates(T, w_tok, w_soft, Ns=PARTITION_NS, alphas=PARTITION_ALPHAS, round_to=128):
    """[(N, alpha, seg_lens)] for every grid point whose rounded partition is
    valid; points that give the same lengths are kept once (the first)."""
    seen, out = set(), []
    for N in Ns:
        for a in alphas:
            try:
                lens = tuple(partition_hybrid(T, N, a, w_tok, w_soft, round_to))
            except Exception:
                continue
            if lens in seen:
                continue
            seen.add(lens)
            out.append((N, a, list(lens)))
    return out


def search(candidates, time_fn, feasible_fn=None, repeats=1):
    """Time every candidate with time_fn(candidate) -> milliseconds (the best
    of `repeats` calls) and return (best, table).  feasible_fn(candidate) ->
    bool filters candidates before timing (the paper's memory constraint).
    table rows: dict(candidate=..., ms=... or None, status="ok"|"infeasible"|
    "error: ...").  Ties keep the earlier candidate."""
    table, best = [], None
    for c in candidates:
        if feasible_fn is not None and not feasible_fn(c):
            table.append(dict(candidate=c, ms=None, status="infeasible"))
            continue
        try:
            ms = min(float(time_fn(c)) for _ in range(max(1, repeats)))
        except Exception as e:  # a failing candidate is reported, not fatal
            table.append(dict(candidate=c, ms=None, status=f"error: {e}"))
            continue
        if not math.isfinite(ms):
            table.append(dict(candidate=c, ms=None, status="error: non-finite time"))
            continue
        table.append(dict(candidate=c, ms=ms, status="ok"))
        if best is None or ms < best[1]:
            best = (c, ms)
    return (best[0] if best else None), table


def speedups(table, reference):
    """Each timed row's speedup over the row whose candidate == reference."""
    ref = next((r["ms"] for r in table if r["candidate"] == reference and r["ms"] is not None), None)
    return [None if (ref is None or r["ms"] is None) else ref / r["ms"] for r in table]
