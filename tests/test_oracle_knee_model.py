"""Pins for the analytical-model oracle (CPU only).

Pinned against: hand-evaluated sequences of Eq. layer_num_ops, closed forms
(one kernel is Amdahl's law, L = a + c/S, whose 1/(L^2 S) peaks at S = c/a;
all kernels at S = 1 and at S >= max N_i), the memory-only model (Amdahl
again through Eq. memory_latency), monotonicity in S, and the one printed
maximum of the paper's simulation that the literal reading reproduces
(N1 = 20 -> 9 SMs).  The other printed maxima (24 and 31 SMs, and 34 for
the batching variant) are not reproduced by any reading tried; they stay
parity unpinned.
"""
import json
import os
import random

from oracle import knee_model as km

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_sequence_by_hand():
    assert km.sequence(20, 1, 50) == [float(v) for v in list(range(20, 0, -1)) + [0] * 30]
    assert km.sequence(60, 1, 50) == [float(max(0, 62 - 2 * i)) for i in range(1, 51)]
    assert km.sequence(40, 2, 50) == [float(max(0, 82 - 2 * i)) for i in range(1, 51)]
    assert km.sequence(10, 1, 4) == [10.0, 7.0, 4.0, 1.0]
    assert km.sequence(5, 3, 1) == [15.0]


def test_single_kernel_is_amdahl():
    # E(S) = t_np + c*t_p/min(S, c): 1/(E^2 S) peaks at S = c*t_p/t_np
    for c, tp, tnp, expect in [(100, 10, 40, 25), (64, 5, 20, 16), (90, 4, 12, 30)]:
        s_values = list(range(1, c + 1))
        et, k = km.knee([float(c)], [float(tp)], s_values, float(tnp))
        assert s_values[k] == expect
        assert et[expect - 1] == tnp + c * tp / expect


def test_limits_in_s():
    rnd = random.Random(5)
    for _ in range(50):
        k = rnd.randint(1, 40)
        n = [float(rnd.randint(0, 90)) for _ in range(k)]
        tp = [float(rnd.randint(1, 50)) for _ in range(k)]
        tnp = float(rnd.randint(0, 20))
        # S = 1: every kernel runs its whole work serially
        assert km.total_time(n, tp, 1, tnp) == sum([tnp] * k) + sum(a * b for a, b in zip(n, tp))
        # S >= max N: a kernel with work takes one t_p, an empty one nothing
        big = int(max(n)) + 1
        expect = sum([tnp] * k) + sum(t for a, t in zip(n, tp) if a >= 1)
        assert abs(km.total_time(n, tp, big, tnp) - expect) < 1e-9 * max(1.0, expect)
        # more SMs never make it slower
        prev = None
        for s in range(1, big + 2):
            e = km.total_time(n, tp, s, tnp)
            assert prev is None or e <= prev + 1e-9 * prev
            prev = e


def test_memory_only_model_is_amdahl():
    # t_p = 0: E_t = b * sum R (t_np + d/(M S)) = a + C/S, knee at C/a
    reps = [1.0, 2.0, 1.0]
    data = [3000.0, 1500.0, 6000.0]
    m = 10.0
    tnp = 5.0
    b = 2.0
    a = b * sum(r * tnp for r in reps)          # 40
    c = b * sum(r * d / m for r, d in zip(reps, data))  # 2400
    s_values = list(range(1, 200))
    _, k = km.knee([1.0, 1.0, 1.0], [0.0, 0.0, 0.0], s_values, tnp, b, reps, data, m)
    assert s_values[k] == c / a == 60


def test_paper_simulation_n1_20():
    g = json.load(open(os.path.join(GOLDEN, "knee_model_simulation.json")))
    n = km.sequence(20, 1, g["kmax"])
    s_values = list(range(1, 81))
    _, k = km.knee(n, [float(g["t_p"])] * len(n), s_values, float(g["t_np"]))
    assert s_values[k] == g["printed_maxima_sms"]["N1=20"]
