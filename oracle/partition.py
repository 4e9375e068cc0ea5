"""fp64 oracle of the hybrid-aware segment lengths.

TEST INFRASTRUCTURE ONLY (tests/ may use it; the product path never does).

Sec. 3.2 (Hybrid-Aware Sequence Chunking) prices segment i of a T-token
sequence cut at 0 = c_0 < ... < c_N = T as
    Cost_i = w_tok * s_i + w_soft * (c_i * s_i + s_i^2 / 2),   s_i = c_{i+1} - c_i,
asks for the boundaries that make every Cost_i equal, interpolates them with
the equal-length boundaries i T / N by alpha, and rounds each boundary to the
closest multiple of round_to (half-way cases up, this package's reading).

The balanced boundaries are found here one at a time by bisection: c_i is the
point where the summed cost of the segments before it reaches i / N of the
total.  Pinned by tests/test_partition.py (equal per-segment costs at
alpha = 1, the equal-length cases, a closed form for w_tok = 0).
"""
import math


def prefix_cost(c, w_tok, w_soft):
    """Summed cost of the segments covering tokens [0, c): sum_i Cost_i for a
    cut at c, which telescopes to w_tok c + w_soft c^2 / 2 whatever the cuts
    inside [0, c) are."""
    return w_tok * c + 0.5 * w_soft * c * c


def balanced_boundaries(T, N, w_tok, w_soft, iters=200):
    """c_0..c_N (floats) with equal per-segment cost, by bisection."""
    total = prefix_cost(T, w_tok, w_soft)
    out = [0.0]
    for i in range(1, N):
        target = total * i / N
        lo, hi = 0.0, float(T)
        for _ in range(iters):
            mid = 0.5 * (lo + hi)
            if prefix_cost(mid, w_tok, w_soft) < target:
                lo = mid
            else:
                hi = mid
        out.append(0.5 * (lo + hi))
    out.append(float(T))
    return out


def candidate_boundaries(T, N, alpha, w_tok, w_soft):
    """Unrounded c_i(alpha) = (1 - alpha) i T / N + alpha c_i^hybrid."""
    hyb = balanced_boundaries(T, N, w_tok, w_soft)
    return [(1.0 - alpha) * (T * i / N) + alpha * hyb[i] for i in range(N + 1)]


def partition_hybrid(T, N, alpha, w_tok, w_soft, round_to=128):
    """Segment lengths, or None when rounding leaves a segment empty."""
    c = candidate_boundaries(T, N, alpha, w_tok, w_soft)
    r = [0] + [int(math.floor(x / round_to + 0.5)) * round_to for x in c[1:-1]] + [T]
    lens = [r[i + 1] - r[i] for i in range(N)]
    return lens if all(x > 0 for x in lens) else None


def segment_costs(bounds, w_tok, w_soft):
    """Cost_i of each segment from the per-segment formula."""
    return [w_tok * (b - a) + w_soft * (a * (b - a) + 0.5 * (b - a) ** 2) for a, b in zip(bounds[:-1], bounds[1:])]
