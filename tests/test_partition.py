"""Hybrid-aware segment lengths (Sec. 3.2): the fp64 oracle against closed
forms, and the library's sf_partition_hybrid (host-only, runs without a GPU)
against the oracle, integer for integer."""
import math
import random

import pytest

from oracle import partition as op
from paper_2608_06838_amd import _lib
import paper_2608_06838_amd as sf


@pytest.mark.parametrize("N", [2, 3, 8, 32])
@pytest.mark.parametrize("ratio", [0.5, 4.0, 50.0])
def test_balanced_costs_are_equal(N, ratio):
    """At alpha = 1, before rounding, every segment's cost (the paper's
    per-segment formula) equals total / N."""
    T, w_tok = 262144, 1.0
    w_soft = ratio / T
    b = op.balanced_boundaries(T, N, w_tok, w_soft)
    costs = op.segment_costs(b, w_tok, w_soft)
    total = op.prefix_cost(T, w_tok, w_soft)
    for c in costs:
        assert abs(c - total / N) <= 1e-9 * total
    assert all(x < y for x, y in zip(b, b[1:]))
    lens = [y - x for x, y in zip(b, b[1:])]
    assert all(x > y for x, y in zip(lens, lens[1:]))  # later segments see longer prefixes


def test_equal_length_cases():
    T, N = 262144, 8
    assert op.partition_hybrid(T, N, 0.0, 1.0, 5.0 / T) == [T // N] * N     # alpha = 0
    assert op.partition_hybrid(T, N, 1.0, 1.0, 0.0) == [T // N] * N         # no softmax layers
    b = op.balanced_boundaries(T, N, 3.0, 0.0)
    assert all(abs(x - T * i / N) <= 1e-6 for i, x in enumerate(b))


def test_softmax_only_closed_form():
    """w_tok = 0: the prefix cost is w_soft c^2 / 2, so c_i = T sqrt(i / N)."""
    T, N = 1 << 20, 4
    b = op.balanced_boundaries(T, N, 0.0, 1e-3)
    for i in range(N + 1):
        assert abs(b[i] - T * math.sqrt(i / N)) <= 1e-6 * T


def test_rounding():
    T, N = 262144, 8
    lens = op.partition_hybrid(T, N, 1.0, 1.0, 4.0 / T, round_to=128)
    assert sum(lens) == T and all(x % 128 == 0 for x in lens)
    assert op.partition_hybrid(1024, 16, 1.0, 1.0, 1.0, round_to=128) is None  # segments collapse


def test_library_matches_oracle():
    """sf_partition_hybrid (closed-form root, exact rounding decision) against
    the oracle (bisection, exact rational rounding decision), integer for
    integer on every draw: equal-length splits whose boundaries fall exactly
    half-way between multiples of round_to included."""
    rng = random.Random(42)
    ties = 0
    for _ in range(400):
        round_to = rng.choice([64, 128, 256, 2048])
        T = round_to * rng.randint(16, 4096)
        N = rng.choice([1, 2, 4, 6, 8, 16, 32])
        alpha = rng.choice([0.0, 0.1, 0.3, 0.5, 0.7, 1.0, 1.25])
        w_tok = rng.choice([0.0, 1.0, 7.5])
        w_soft = rng.choice([0.0, 1.0 / T, 30.0 / T, 1e-3]) if w_tok > 0 else rng.choice([1.0 / T, 1e-3])
        c = op.candidate_boundaries(T, N, alpha, w_tok, w_soft)
        ties += any(abs((x / round_to) % 1.0 - 0.5) < 1e-6 / round_to for x in c[1:-1])
        ref = op.partition_hybrid(T, N, alpha, w_tok, w_soft, round_to)
        if ref is None:
            with pytest.raises(sf.StateflowError):
                sf.partition_hybrid(T, N, alpha, w_tok, w_soft, round_to)
        else:
            assert sf.partition_hybrid(T, N, alpha, w_tok, w_soft, round_to) == ref, (T, N, alpha, w_tok, w_soft)
    assert ties > 50  # the half-way cases are well represented


@pytest.mark.parametrize("T,N,alpha,w_tok,w_soft,want", [
    # alpha = 0: boundary i T / N = 192 = 1.5 * 128, half-way: rounds up
    (384, 2, 0.0, 1.0, 1.0, [256, 128]),
    # no softmax layers: every alpha gives i T / N; 0.25 * 1.5 ... = 192 again
    (384, 2, 0.5, 1.0, 0.0, [256, 128]),
    (384, 2, 1.25, 1.0, 0.0, [256, 128]),
    # softmax only, alpha = 1: c_1 = T sqrt(1/4) = 320 = 2.5 * 128 exactly; c_2 = T sqrt(1/2),
    # c_3 = T sqrt(3/4) are irrational (453.5..., 554.2...)
    (640, 4, 1.0, 0.0, 1e-3, [384, 128, 128, 0]),
    (1280, 4, 1.0, 0.0, 1.0, [640, 256, 256, 128]),
])
def test_half_way_rounds_up(T, N, alpha, w_tok, w_soft, want):
    """Exact ties, decided by the oracle's rational arithmetic: the half-up
    reading of "the closest multiple of 128"."""
    ref = op.partition_hybrid(T, N, alpha, w_tok, w_soft, 128)
    if 0 in want:
        assert ref is None
        with pytest.raises(sf.StateflowError):
            sf.partition_hybrid(T, N, alpha, w_tok, w_soft, 128)
        return
    assert ref == want
    assert sf.partition_hybrid(T, N, alpha, w_tok, w_soft, 128) == want


def test_exact_decision_pins():
    """The oracle's exact comparison against hand-computed boundaries."""
    # equal lengths: c_1 = 1 * 1000 / 3 = 333.33...
    assert op.boundary_at_least(1000, 3, 1, 0.0, 1.0, 0.0, 333)
    assert not op.boundary_at_least(1000, 3, 1, 0.0, 1.0, 0.0, 334)
    # softmax only, alpha = 1: c_1 = 400 sqrt(1/4) = 200 exactly
    assert op.boundary_at_least(400, 4, 1, 1.0, 0.0, 2.0, 200)
    assert not op.boundary_at_least(400, 4, 1, 1.0, 0.0, 2.0, 200 + 1e-9)
    # alpha = 1/2 between 100 (equal) and 200 (balanced): 150
    assert op.boundary_at_least(400, 4, 1, 0.5, 0.0, 2.0, 150)
    assert not op.boundary_at_least(400, 4, 1, 0.5, 0.0, 2.0, 150.000001)


def test_library_validation():
    import ctypes
    L = _lib.lib()
    out = (ctypes.c_int64 * 8)()
    assert L.sf_partition_hybrid(262144, 8, 1.0, 1.0, 1e-5, 128, None) == _lib.SF_E_NULL
    for args in ((0, 8, 1.0, 1.0, 0.0, 128), (1000, 8, 1.0, 1.0, 0.0, 128), (262144, 0, 1.0, 1.0, 0.0, 128),
                 (262144, 8, -0.5, 1.0, 0.0, 128), (262144, 8, 1.0, 0.0, 0.0, 128),
                 (262144, 8, 1.0, -1.0, 0.0, 128), (262144, 8, float("nan"), 1.0, 0.0, 128)):
        assert L.sf_partition_hybrid(*args, out) == _lib.SF_E_SHAPE, args
