"""Selection logic of the profile-guided tuner (CPU only: the timer is a
stand-in; the GPU studies live in bench.py --tune-ts / --partition-study)."""
import math

from paper_2608_06838_amd import tune


def test_ts_candidates():
    c = tune.ts_candidates([65536, 20480])
    assert c[0] == 0 and all(t % 64 == 0 and 0 < t <= 65536 for t in c[1:])
    assert tune.ts_candidates([640]) == [0, 128, 256, 512]


def test_partition_candidates():
    T, w_tok, w_soft = 262144, 1.0, 2.0 / 262144
    cands = tune.partition_candidates(T, w_tok, w_soft)
    assert cands, "no candidates"
    seen = set()
    for N, a, lens in cands:
        assert len(lens) == N and sum(lens) == T and all(x > 0 and x % 128 == 0 for x in lens)
        assert tuple(lens) not in seen
        seen.add(tuple(lens))
        if a > 0:  # later segments see longer prefixes: non-increasing lengths, up to the
            # one rounding step by which two independently rounded boundaries can differ
            assert all(x >= y - 128 for x, y in zip(lens, lens[1:]))
            assert lens[0] > lens[-1]
    # without softmax layers every alpha gives equal lengths: one candidate per N
    flat = tune.partition_candidates(T, 1.0, 0.0)
    assert sorted(N for N, _, _ in flat) == sorted(tune.PARTITION_NS)
    assert all(max(lens) - min(lens) <= 128 for _, _, lens in flat)  # 262144 / 6 is not a multiple of 128


def test_search_picks_fastest_and_reports_failures():
    cands = [(2, 0.0), (8, 0.5), (8, 1.0), (16, 0.0), (32, 1.25)]

    def fake_ms(c):
        if c == (16, 0.0):
            raise RuntimeError("does not fit")
        return abs(c[0] - 8) + c[1]

    best, table = tune.search(cands, fake_ms, feasible_fn=lambda c: c[0] != 32)
    assert best == (8, 0.5)
    status = {r["candidate"]: r["status"] for r in table}
    assert status[(32, 1.25)] == "infeasible"
    assert status[(16, 0.0)].startswith("error")
    assert [r["ms"] for r in table if r["status"] == "ok"] == [6.0, 0.5, 1.0]
    sp = tune.speedups(table, (2, 0.0))
    assert sp[0] == 1.0 and math.isclose(sp[1], 12.0) and sp[3] is None


def test_search_ties_keep_first():
    best, _ = tune.search(["a", "b"], lambda c: 1.0)
    assert best == "a"
    best, table = tune.search(["x"], lambda c: float("nan"))
    assert best is None and table[0]["status"].startswith("error")
