"""Oracle of the hybrid-aware segment lengths, in exact rational arithmetic
where it decides an integer.

TEST INFRASTRUCTURE ONLY (tests/ may use it; the product path never does).

Sec. 3.2 (Hybrid-Aware Sequence Chunking) prices segment i of a T-token
sequence cut at 0 = c_0 < ... < c_N = T as
    Cost_i = w_tok * s_i + w_soft * (c_i * s_i + s_i^2 / 2),   s_i = c_{i+1} - c_i,
asks for the boundaries that make every Cost_i equal, interpolates them with
the equal-length boundaries i T / N by alpha, and rounds each boundary to the
closest multiple of round_to (half-way cases up, this package's reading).

The summed cost of the segments before a cut at c telescopes to
A(c) = w_tok c + w_soft c^2 / 2, so the balanced boundary c_i^hyb is where A
reaches i / N of A(T).  Bisection gives c_i^hyb in floating point (used for
the cost pins); the rounded boundary is decided exactly: with every input
taken at its exact value (fractions.Fraction),
c_i(alpha) >= y holds iff
    alpha = 0:  i T / N >= y
    alpha > 0:  x <= 0 or A(x) <= (i / N) A(T),  x = (y - (1 - alpha) i T / N) / alpha
(A increases on x >= 0 and c_i^hyb >= 0), and the rounded boundary is the
multiple m * round_to with (m - 1/2) round_to <= c_i(alpha) < (m + 1/2) round_to,
m at most T / round_to (a boundary past T leaves a segment empty).
Pinned by tests/test_partition.py (equal per-segment costs at alpha = 1, the
equal-length cases, the closed form for w_tok = 0, exact ties).
"""
from fractions import Fraction


def prefix_cost(c, w_tok, w_soft):
    """Summed cost of the segments covering tokens [0, c): sum_i Cost_i for a
    cut at c, which telescopes to w_tok c + w_soft c^2 / 2 whatever the cuts
    inside [0, c) are."""
    return w_tok * c + w_soft * c * c / 2


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
    """Unrounded c_i(alpha) = (1 - alpha) i T / N + alpha c_i^hybrid (floats)."""
    hyb = balanced_boundaries(T, N, w_tok, w_soft)
    return [(1.0 - alpha) * (T * i / N) + alpha * hyb[i] for i in range(N + 1)]


def boundary_at_least(T, N, i, alpha, w_tok, w_soft, y):
    """Exactly: is c_i(alpha) >= y?  (inputs at their exact values)"""
    a, p, s, y = Fraction(alpha), Fraction(w_tok), Fraction(w_soft), Fraction(y)
    equal = Fraction(i * T, N)
    if a == 0:
        return equal >= y
    x = (y - (1 - a) * equal) / a
    if x <= 0:
        return True
    return prefix_cost(x, p, s) <= Fraction(i, N) * prefix_cost(Fraction(T), p, s)


def rounded_boundary(T, N, i, alpha, w_tok, w_soft, round_to):
    """The multiple of round_to closest to c_i(alpha), half-way cases up: the
    largest m in [0, T / round_to] with c_i(alpha) >= (m - 1/2) round_to, by
    bisection over m on the exact comparison (m = 0 always qualifies)."""
    half = Fraction(round_to, 2)
    lo, hi = 0, T // round_to
    while lo < hi:
        mid = (lo + hi + 1) // 2
        if boundary_at_least(T, N, i, alpha, w_tok, w_soft, mid * round_to - half):
            lo = mid
        else:
            hi = mid - 1
    return lo * round_to


def partition_hybrid(T, N, alpha, w_tok, w_soft, round_to=128):
    """Segment lengths, or None when rounding leaves a segment empty."""
    r = [0] + [rounded_boundary(T, N, i, alpha, w_tok, w_soft, round_to) for i in range(1, N)] + [T]
    lens = [r[i + 1] - r[i] for i in range(N)]
    return lens if all(x > 0 for x in lens) else None


def segment_costs(bounds, w_tok, w_soft):
    """Cost_i of each segment from the per-segment formula."""
    return [w_tok * (b - a) + w_soft * (a * (b - a) + 0.5 * (b - a) ** 2) for a, b in zip(bounds[:-1], bounds[1:])]
