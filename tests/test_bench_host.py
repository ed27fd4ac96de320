"""Host-side helpers of bench.py that decide the timed workload: the knee of
a timing-table row, fitting the deployed slot counts into the GPU, and
packing them into disjoint partitions (no GPU needed)."""
import random

import bench
from oracle import sched


def test_knee_at_matches_oracle_knee():
    """bench's knee (argmax of b / (L^2 s), ties to fewer slots, Sec. 4.1's
    efficacy) equals the oracle scheduler's on random rows and on ties."""
    rng = random.Random(5)
    slots = [3, 6, 10, 13, 16, 19, 22, 26, 29, 32]
    for _ in range(500):
        b = rng.randint(1, 32)
        row = {s: rng.randint(50, 5000) for s in slots}
        assert bench.knee_at(row, b) == sched.knee(row, b)
    # a tie in eta keeps the smaller slot count: L^2 s equal for s = 4 and 9
    assert bench.knee_at({4: 300, 9: 200}, 8) == 4
    # latency flat beyond the knee: the smallest share wins
    assert bench.knee_at({8: 100, 16: 100, 32: 100}, 4) == 8


def test_fit_slots():
    assert bench.fit_slots([10, 12], 32) == [10, 12]  # fits: unchanged
    assert bench.fit_slots([18, 18], 32) == [16, 16]  # knee + 2 each, shrunk evenly
    out = bench.fit_slots([30, 9, 5], 32)
    assert sum(out) <= 32 and all(o >= 1 for o in out)
    assert out[0] >= out[1] >= out[2]  # proportional order kept
    for dep in ([32, 32], [1, 40], [7, 7, 7, 7, 7]):
        out = bench.fit_slots(dep, 32)
        assert sum(out) <= 32 and all(o >= 1 for o in out)


def test_pack_lanes_disjoint_and_bounded():
    lanes = bench.pack_lanes([16, 16], 32, 4)
    assert lanes == [(0, 0, 16), (1, 16, 16)]
    lanes = bench.pack_lanes([8, 5], 32, 4)
    assert len(lanes) == 4  # at most 4 partitions
    used = set()
    for mi, off, n in lanes:
        span = set(range(off, off + n))
        assert not (span & used) and off + n <= 32
        used |= span
    assert {mi for mi, _, _ in lanes} == {0, 1}  # round-robin over the models
