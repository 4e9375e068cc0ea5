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
    """sf_partition_hybrid (closed-form root) against the oracle (bisection).
    A boundary within 1e-6 tokens of a rounding midpoint can round either way
    in fp64 (the two sides reach it by different arithmetic); such draws are
    skipped: about a quarter of these seeds, mostly equal-length splits whose
    boundaries fall exactly half-way between multiples of round_to."""
    rng = random.Random(42)
    checked = 0
    for _ in range(400):
        round_to = rng.choice([64, 128, 256, 2048])
        T = round_to * rng.randint(16, 4096)
        N = rng.choice([1, 2, 4, 6, 8, 16, 32])
        alpha = rng.choice([0.0, 0.1, 0.3, 0.5, 0.7, 1.0, 1.25])
        w_tok = rng.choice([0.0, 1.0, 7.5])
        w_soft = rng.choice([0.0, 1.0 / T, 30.0 / T, 1e-3]) if w_tok > 0 else rng.choice([1.0 / T, 1e-3])
        c = op.candidate_boundaries(T, N, alpha, w_tok, w_soft)
        if any(abs((x / round_to) % 1.0 - 0.5) < 1e-6 / round_to for x in c[1:-1]):
            continue
        ref = op.partition_hybrid(T, N, alpha, w_tok, w_soft, round_to)
        if ref is None:
            with pytest.raises(sf.StateflowError):
                sf.partition_hybrid(T, N, alpha, w_tok, w_soft, round_to)
        else:
            assert sf.partition_hybrid(T, N, alpha, w_tok, w_soft, round_to) == ref, (T, N, alpha, w_tok, w_soft)
        checked += 1
    assert checked > 250


def test_library_validation():
    import ctypes
    L = _lib.lib()
    out = (ctypes.c_int64 * 8)()
    assert L.sf_partition_hybrid(262144, 8, 1.0, 1.0, 1e-5, 128, None) == _lib.SF_E_NULL
    for args in ((0, 8, 1.0, 1.0, 0.0, 128), (1000, 8, 1.0, 1.0, 0.0, 128), (262144, 0, 1.0, 1.0, 0.0, 128),
                 (262144, 8, -0.5, 1.0, 0.0, 128), (262144, 8, 1.0, 0.0, 0.0, 128),
                 (262144, 8, 1.0, -1.0, 0.0, 128), (262144, 8, float("nan"), 1.0, 0.0, 128)):
        assert L.sf_partition_hybrid(*args, out) == _lib.SF_E_SHAPE, args
