"""Host-side helpers of bench.py that decide the timed workload: the knee of
a timing-table row, fitting the deployed slot counts into the GPU, packing
them into disjoint partitions, and the capacity search with its confirming
timed run (on a stand-in for the live mix; no GPU needed)."""
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


class FakeMix:
    """Stands in for the live four-model mix: a run at rate scale k violates
    when k exceeds a threshold (the probes) or a lower one for the longer
    timed runs (saturation grows with the trace length)."""

    def __init__(self, probe_limit, timed_limit):
        self.probe_limit, self.timed_limit, self.calls = probe_limit, timed_limit, []

    def run(self, k, dur_us, policy, param=0):
        self.calls.append(("run", k))
        bad = k > (self.timed_limit if dur_us > 1600000 else self.probe_limit)
        return dict(k=k, offered_req_s=k * 1650, on_time_per_s=k * 1650 * (0.5 if bad else 1.0),
                    violation_frac=0.5 if bad else 0.0, utilisation_ppm=0)

    def timed(self, k, policy, param, steps, warmup):
        self.calls.append(("timed", k))
        return self.run(k, steps * bench.PERIOD_US, policy, param)


def test_capacity_search_doubles_then_bisects():
    m = FakeMix(probe_limit=19.0, timed_limit=19.0)
    k, probes = bench.Mix4.capacity(m, "dstack", (0, 0), 1.5)
    ks = [p["k"] for p in probes]
    assert ks[:6] == [1.0, 2.0, 4.0, 8.0, 16.0, 32.0]  # doubling until a probe fails
    assert len(ks) == 6 + bench.CAPACITY_BISECTIONS  # then bisections on the geometric mean
    assert 16.0 <= k <= 19.0 and all(p["violation_frac"] == 0.0 for p in probes if p["k"] <= k)
    assert k == max(p["k"] for p in probes if p["violation_frac"] <= bench.VIOLATION_BAR)
    # below 1: halving
    k2, probes2 = bench.Mix4.capacity(FakeMix(0.3, 0.3), "temporal", 15000, 1.5)
    assert [p["k"] for p in probes2][:3] == [1.0, 0.5, 0.25] and 0.25 <= k2 <= 0.3


def test_timed_run_falls_back_to_the_next_passing_probe():
    m = FakeMix(probe_limit=19.0, timed_limit=17.0)
    k, probes = bench.Mix4.capacity(m, "dstack", (0, 0), 1.5)
    entry = dict(k=k, probes=probes)
    k_run, run = bench.confirm_capacity(m, "dstack", (0, 0), entry, 20, 3)
    assert run["violation_frac"] <= bench.VIOLATION_BAR and k_run <= 17.0
    tried = entry["timed_k"]
    assert tried[0] == k
    lower = max(p["k"] for p in probes if p["k"] <= 17.0)
    # the passing probes below k in descending order until one holds, then
    # timed bisection steps between the last k that held and the last that failed
    i = tried.index(lower)
    passing = sorted((p["k"] for p in probes if p["violation_frac"] <= bench.VIOLATION_BAR and lower <= p["k"] < k),
                     reverse=True)
    assert tried[1:i + 1] == passing and len(tried) == i + 1 + bench.CONFIRM_BISECTIONS
    lo, hi = lower, tried[i - 1]
    for mid in tried[i + 1:]:
        assert abs(mid - (lo * hi) ** 0.5) < 1e-9
        lo, hi = (mid, hi) if mid <= 17.0 else (lo, mid)
    assert k_run == lo and lo <= 17.0
    # a capacity that holds over the timed run is kept as it is
    m2 = FakeMix(probe_limit=19.0, timed_limit=19.0)
    k2, probes2 = bench.Mix4.capacity(m2, "dstack", (0, 0), 1.5)
    e2 = dict(k=k2, probes=probes2)
    assert bench.confirm_capacity(m2, "dstack", (0, 0), e2, 20, 3)[0] == k2 and e2["timed_k"] == [k2]


def test_work_rate_weights_on_time_requests_by_flops():
    """The FLOP-weighted guard: each model's on-time requests per second
    (served less late ones; unserved ones were never served) x its FLOP per
    inference, for both policies, and their ratio."""
    class Info:
        def __init__(self, f):
            self.flops_per_item = f

    class M:
        def __init__(self, f):
            self.info = Info(f)

    class Mix:
        models = [M(8e9), M(6e8)]
    run_d = dict(run_us=2_000_000, per_model=[dict(served=1000, violations=10, unserved=4),
                                              dict(served=2000, violations=0, unserved=0)])
    run_t = dict(run_us=2_000_000, per_model=[dict(served=500, violations=0, unserved=0),
                                              dict(served=1000, violations=0, unserved=0)])
    w = bench.work_rate(Mix(), run_d, run_t)
    # D-STACK: (1000 - 6) x 8e9 / 2 s + 2000 x 6e8 / 2 s = 4.576 TFLOP/s; temporal 2.3
    assert abs(w["dstack_tflops"] - 4.576) < 1e-9 and abs(w["timesliced_tflops"] - 2.3) < 1e-9
    assert abs(w["ratio"] - 4.576 / 2.3) < 1e-12
    assert abs(w["dstack_frac_of_chip_peak"] - 4.576 / bench.PEAK_BF16_TFLOPS) < 1e-12
