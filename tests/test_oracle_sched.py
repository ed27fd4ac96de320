"""Pins for the scheduler oracle (CPU only).

Pinned against: closed forms (Amdahl tables, where argmax_s 1/(L(s)^2 s) for
L = a + c/s sits at s = c/a), the utilisation figures the paper prints for
its own model table, planted optima, brute force on small grids, and the
invariants of a valid schedule.
"""
import itertools
import json
import os
import random

import pytest

from oracle import sched

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def amdahl_row(a, c, slots):
    return {s: a + c // s for s in slots}


def test_knee_amdahl_closed_form():
    # L(s) = a + c/s; eta ~ 1/(L^2 s) peaks at s = c/a.  Grids where c/s is exact.
    for a, c, expect in [(1000, 16000, 16), (500, 2000, 4), (250, 2500, 10), (2000, 64000, 32)]:
        slots = [s for s in range(1, 33) if c % s == 0]
        assert sched.knee(amdahl_row(a, c, slots), b=8) == expect


def test_knee_ties_prefer_fewer_slots_and_flat_latency():
    row = {4: 100, 8: 100, 16: 100}          # flat curve: fewest slots is best
    assert sched.knee(row, 1) == 4
    row = {1: 400, 4: 200}                   # eta equal: 1/(160000*1) vs 1/(40000*4)
    assert sched.knee(row, 1) == 1


def test_knee_brute_force_random():
    rnd = random.Random(3)
    for _ in range(300):
        slots = sorted(rnd.sample(range(1, 33), rnd.randint(1, 10)))
        row = {s: rnd.randint(50, 5000) for s in slots}
        b = rnd.choice(sched.BATCH_GRID)
        best = max(slots, key=lambda s: (b / (row[s] ** 2 * s), -s))
        assert sched.knee(row, b) == best


def test_assembly_time():
    # one 224x224x3 fp32 image over 10 Gb/s: 224*224*3*4*8 bits / 1e10 b/s = 481.7 us
    assert abs(224 * 224 * 3 * 4 * 8 / 10e9 * 1e6 - 481.7) < 0.05
    assert sched.assembly_us(16, 0) == 16 * 482
    assert sched.assembly_us(10, 400) == 25000
    assert sched.assembly_us(3, 800) == 3750
    assert sched.assembly_us(1, 300) == 3334  # ceil(1e6/300)


def test_optimize_planted_optimum_and_constraints():
    # latency grows with batch, shrinks with slots; one point is planted far better
    table = {b: {s: 1000 * b + 40000 // s for s in (4, 8, 16, 32)} for b in (1, 2, 4, 8, 16)}
    table[8][8] = 3000
    ch = sched.optimize(table, slo=50000, bmax=16)
    assert (ch.batch, ch.slots, ch.latency, ch.feasible) == (8, 8, 3000, True)
    # the SLO/2 constraint (Eq. meet_half_slo) excludes a point that meets Eq. meet_slo
    t2 = {1: {8: 6000}, 2: {8: 7000}}
    ch = sched.optimize(t2, slo=13000, bmax=2)
    assert ch.feasible and ch.batch == 1  # 7000 > 13000//2 although 7000 + 964 <= 13000
    # Bmax (Eq. max_batch_size) excludes larger batches
    ch = sched.optimize(table, slo=50000, bmax=4)
    assert ch.batch <= 4


def test_optimize_brute_force_random():
    rnd = random.Random(5)
    for _ in range(300):
        table = {}
        for b in sched.BATCH_GRID:
            if rnd.random() < 0.8:
                table[b] = {s: rnd.randint(200, 20000) for s in sorted(rnd.sample(range(1, 33), 4))}
        if not table:
            continue
        slo, bmax, rate = rnd.randint(2000, 40000), rnd.choice([4, 8, 16, 32]), rnd.choice([0, 150, 400, 800])
        pts = [(b, s, L) for b, row in table.items() if b <= bmax for s, L in row.items()
               if L + sched.assembly_us(b, rate) <= slo and L <= slo // 2]
        ch = sched.optimize(table, slo, bmax, rate)
        if pts:
            from fractions import Fraction
            best = max(pts, key=lambda p: (Fraction(p[0], p[2] * p[2] * p[1]), -p[1], p[0]))
            assert (ch.batch, ch.slots, ch.latency, ch.feasible) == (best[0], best[1], best[2], True)
        else:
            assert not ch.feasible


def _paper_models():
    # Table model_characteristics: Alexnet 30%/25 ms/8 ms, ResNet-50 40%/50 ms/28 ms,
    # VGG-19 50%/100 ms/55 ms.  Shares in units of 10% (10 slots = the GPU).
    return [sched.PlanModel(slo=25000, knee=3, slots=3, row={3: 8000}),
            sched.PlanModel(slo=50000, knee=4, slots=4, row={4: 28000}),
            sched.PlanModel(slo=100000, knee=5, slots=5, row={5: 55000})]


def test_paper_st_only_utilisation():
    """Sec. 6.1.1 prints 60% for the ST-only schedule of these three models in a
    100 ms session; the exact knee%-time sum is 59.5%."""
    jobs = sched.plan(_paper_models(), period=100000, total=10)
    assert [sum(1 for j in jobs if j.model == i) for i in range(3)] == [4, 2, 1]
    assert not any(j.missed for j in jobs)
    u = sched.utilisation_ppm(jobs, 100000, total=10)
    assert u == 595000 and round(u / 1e4) == 60
    with open(os.path.join(GOLDEN, "paper_st_schedule.json")) as f:
        golden = json.load(f)
    assert golden["utilisation_percent_printed"] == 60


def test_paper_temporal_utilisation():
    """Sec. 6.1 prints 44% mean utilisation for SLO-proportional time slices."""
    u = sched.temporal_utilisation([(25, 30), (50, 40), (100, 50)])
    assert abs(u - 44.2857) < 1e-3 and round(u) == 44


def _check_valid(models, jobs, period, total):
    placed = [j for j in jobs if not j.missed]
    points = sorted({j.start for j in placed})
    for t in points:
        act = [j for j in placed if j.start <= t < j.end]
        assert sum(j.slots for j in act) <= total
        masks = [j.slot_mask for j in act]
        for a, b in itertools.combinations(masks, 2):
            assert a & b == 0
    for j in placed:
        assert j.release <= j.start and j.end <= j.deadline <= period
        assert bin(j.slot_mask).count("1") == j.slots
        assert j.duration == sched.latency_at(models[j.model].row, j.slots)
    for i, m in enumerate(models):
        assert sum(1 for j in jobs if j.model == i) == sched.ceil_div(period, m.slo)


def test_plan_invariants_random():
    rnd = random.Random(11)
    for _ in range(200):
        models = []
        for _ in range(rnd.randint(1, 5)):
            grid = sorted(rnd.sample(range(1, 33), rnd.randint(2, 8)))
            row, L = {}, rnd.randint(20000, 60000)
            for s in grid:
                L = max(500, int(L * rnd.uniform(0.5, 1.0)))
                row[s] = L
            kn = sched.knee(row, 8)
            models.append(sched.PlanModel(slo=rnd.choice([15000, 25000, 30000, 50000, 100000]), knee=kn,
                                          slots=sched.deployed_slots(kn), row=row))
        period = 100000
        jobs = sched.plan(models, period)
        _check_valid(models, jobs, period, sched.TOTAL_SLOTS)


def test_plan_even_early_odd_late():
    m = [sched.PlanModel(slo=25000, knee=4, slots=4, row={4: 5000})]
    jobs = sched.plan(m, 100000)
    assert [(j.k, j.start) for j in jobs] == [(0, 0), (1, 45000), (2, 50000), (3, 95000)]


def test_plan_below_knee_fallback_and_miss():
    # model 0 (shorter SLO, so placed first by EDF) fills 28 slots for the whole
    # period; model 1 cannot get its 8 and runs on 4, below its knee
    m = [sched.PlanModel(slo=25000, knee=28, slots=28, row={28: 25000}),
         sched.PlanModel(slo=50000, knee=8, slots=8, row={2: 40000, 4: 30000, 8: 10000})]
    jobs = sched.plan(m, 100000)
    j1 = [j for j in jobs if j.model == 1]
    assert all(not j.missed and j.slots == 4 and j.duration == 30000 for j in j1)
    # with 31 slots taken and latencies longer than the window, model 1 is missed
    m[0] = sched.PlanModel(slo=25000, knee=31, slots=31, row={31: 25000})
    m[1] = sched.PlanModel(slo=50000, knee=8, slots=8, row={2: 60000, 4: 55000, 8: 10000})
    jobs = sched.plan(m, 100000)
    assert all(j.missed for j in jobs if j.model == 1)


def test_plan_brute_force_small():
    """On tiny grids (1 ms steps, <= 3 models) every job the plan places is at a
    start that brute force also finds feasible, and when brute force finds
    all jobs of a model-set placeable with slack the plan misses none."""
    rnd = random.Random(17)
    for _ in range(60):
        models = []
        for _ in range(rnd.randint(1, 3)):
            s = rnd.randint(1, 3)
            models.append(sched.PlanModel(slo=rnd.choice([5000, 10000]), knee=s, slots=s,
                                          row={s: 1000 * rnd.randint(1, 3)}))
        jobs = sched.plan(models, 10000, total=4)
        _check_valid(models, jobs, 10000, 4)
        if sum(m.slots * m.row[m.slots] * sched.ceil_div(10000, m.slo) for m in models) <= 4 * 10000 // 4:
            # load at most a quarter of capacity and each job fits its window alone
            assert not any(j.missed for j in jobs)


# ---- home placement (one fixed slot range per model) ----

def test_home_offsets_hand_cases():
    # disjoint when they fit: largest first at 0, then the first zero-overlap offsets
    assert sched.home_offsets([6, 10, 8], 32) == [18, 0, 10]
    # 20 + 20 > 32: the second range goes where it overlaps the first least (offset 12, 8 slots)
    assert sched.home_offsets([20, 20], 32) == [0, 12]
    # equal sizes keep index order; a full-width range overlaps everything equally -> offset 0
    assert sched.home_offsets([32, 4], 32) == [0, 0]
    assert sched.home_offsets([5, 5, 5], 10) == [0, 5, 0]
    assert sched.range_mask(3, 4) == 0b1111000


def test_home_plan_disjoint_homes_closed_form():
    """With disjoint homes nothing conflicts, so every job starts at its window
    edge: even k at the window start, odd k at the window end minus L."""
    models = [sched.PlanModel(slo=25000, knee=8, slots=10, row={10: 4000, 8: 5000}),
              sched.PlanModel(slo=15000, knee=6, slots=8, row={8: 3000}),
              sched.PlanModel(slo=50000, knee=10, slots=12, row={12: 20000})]
    homes = sched.home_offsets([m.slots for m in models], 32)
    assert homes == [12, 22, 0]
    jobs = sched.plan(models, 100000, 32, homes)
    for j in jobs:
        m = models[j.model]
        L = m.row[m.slots]
        assert not j.missed and j.slots == m.slots and j.duration == L
        assert j.slot_mask == sched.range_mask(homes[j.model], m.slots)
        assert j.start == (j.release if j.k % 2 == 0 else j.deadline - L)


def test_home_plan_overlapping_homes_serialise():
    """Two models whose homes overlap never run at the same time; jobs keep
    their windows, and the plan matches a hand-worked case."""
    models = [sched.PlanModel(slo=50000, knee=18, slots=20, row={20: 30000}),
              sched.PlanModel(slo=50000, knee=18, slots=20, row={20: 15000})]
    homes = sched.home_offsets([20, 20], 32)
    jobs = sched.plan(models, 100000, 32, homes)
    # EDF order: (deadline 50000: m0 k0, m1 k0), (100000: m0 k1, m1 k1).
    # m0 k0 at 0; m1 k0 earliest start clear of [0, 30000) is 30000; m0 k1
    # (odd: latest) at 100000 - 30000; m1 k1 (odd: latest) cannot overlap
    # [70000, 100000), so it ends there: 70000 - 15000.
    got = [(j.model, j.k, j.start, j.missed) for j in jobs]
    assert got == [(0, 0, 0, False), (1, 0, 30000, False), (0, 1, 70000, False), (1, 1, 55000, False)]


def test_home_plan_invariants_random():
    rnd = random.Random(17)
    for _ in range(200):
        models = []
        for _ in range(rnd.randint(1, 5)):
            grid = sorted(rnd.sample(range(1, 33), rnd.randint(2, 8)))
            row, L = {}, rnd.randint(5000, 40000)
            for s in grid:
                L = max(500, int(L * rnd.uniform(0.5, 1.0)))
                row[s] = L
            kn = sched.knee(row, 8)
            models.append(sched.PlanModel(slo=rnd.choice([15000, 25000, 30000, 50000, 100000]), knee=kn,
                                          slots=sched.deployed_slots(kn), row=row))
        homes = sched.home_offsets([m.slots for m in models], 32)
        jobs = sched.plan(models, 100000, 32, homes)
        _check_valid(models, jobs, 100000, sched.TOTAL_SLOTS)
        for j in jobs:
            if not j.missed:
                assert j.slots == models[j.model].slots
                assert j.slot_mask == sched.range_mask(homes[j.model], j.slots)


# ---- knee search without a profile (binary search from 30%) ----

GRID = [3, 6, 10, 13, 16, 19, 22, 26, 29, 32]  # the sweep's 10%..100% slot counts


def _eta_argmax(table, b):
    """Brute force: argmax of b / (L^2 s), ties to fewer slots."""
    best = None
    for s in sorted(table):
        if best is None or sched.eta_gt(b, table[s], s, b, table[best], best):
            best = s
    return best


def test_knee_search_unimodal_equals_brute_force():
    """Where the efficacy over the candidates rises then falls, the search
    ends on the same slot count as scanning them all, with few probes."""
    rnd = random.Random(5)
    checked = 0
    for trial in range(600):
        cand = GRID if trial % 2 else list(range(1, 33))
        a, c, d = rnd.uniform(100, 3000), rnd.uniform(500, 60000), rnd.uniform(0, 30)
        table = {s: max(1, int(a + c / s + d * s)) for s in cand}  # Amdahl plus a per-slot cost
        b = rnd.choice([1, 2, 4, 8, 16, 32])
        etas = [b / (table[s] ** 2 * s) for s in cand]
        peak = max(range(len(cand)), key=lambda i: etas[i])
        if any(etas[i] >= etas[i + 1] for i in range(peak)) or any(etas[i] <= etas[i + 1] for i in range(peak, len(cand) - 1)):
            continue  # not strictly unimodal after integer rounding
        k, probes = sched.knee_search(lambda s: table[s], b, cand, 10)
        assert k == _eta_argmax(table, b)
        assert len(probes) <= (10 if cand is GRID else 14)  # the confirmation walk adds at most 4
        assert len({s for s, _ in probes}) == len(probes)
        checked += 1
    assert checked >= 200


def test_knee_search_hand_cases():
    # efficacy strictly falling: the knee is the smallest candidate; first probes at 10 and 13
    k, probes = sched.knee_search(lambda s: 1000, 4, GRID, 10)
    assert k == 3 and [s for s, _ in probes][:2] == [10, 13]
    # latency exactly c / s: eta = b s / c^2 rises with s -> the whole GPU
    k, _ = sched.knee_search(lambda s: 64000 // s, 8, GRID, 10)
    assert k == 32
    # a single candidate needs no probe
    assert sched.knee_search(lambda s: 5, 1, [7], 10) == (7, [])
    # Amdahl a + c/s on every slot count: eta = b s / (a s + c)^2 peaks at s = c / a (here 8)
    amd = {s: 1000 + 8000 // s for s in range(1, 33)}
    k, probes = sched.knee_search(lambda s: amd[s], 16, range(1, 33), 10)
    assert k == _eta_argmax(amd, 16) == 8
    assert [s for s, _ in probes][:2] == [10, 11]
    # a start below every candidate begins at the first
    k, probes = sched.knee_search(lambda s: 1000, 1, GRID, 1)
    assert probes[0][0] == 3 and k == 3


def test_knee_search_stepped_curve_is_confirmed():
    """Latency falling in steps (whole rounds of workgroups): eta(13) <
    eta(10) sends the bisection down to 10, a local maximum; the confirmation
    walk sees eta(16) above it and ends on the grid's argmax."""
    table = dict(zip(GRID, [2405, 1717, 1120, 1014, 755, 758, 704, 726, 585, 583]))
    b = 16
    assert sched.eta_gt(b, table[10], 10, b, table[13], 13)   # the dip that misleads the bisection
    k, probes = sched.knee_search(lambda s: table[s], b, GRID, 10)
    assert k == _eta_argmax(table, b) == 16
    assert [s for s, _ in probes][:2] == [10, 13]
    # without the dip the walk adds nothing beyond the neighbours
    flat = {s: 100000 // s + 200 for s in GRID}
    assert sched.knee_search(lambda s: flat[s], 4, GRID, 10)[0] == _eta_argmax(flat, 4)


def test_ideal_single_model_closed_form():
    # kernels (32 slots, 30 us), (16 slots, 10 us) in 10 us slots: 4 slots per
    # forward, 3 x 32 + 16 = 112 of 128 share-slots used
    m = dict(slots=[32, 16], dur=[30, 10], batch=8, slo_us=10**9)
    r = sched.simulate_ideal([m], 1000, 10)
    assert r["forwards"] == [25] and r["items"] == [200] and r["late"] == [0]
    assert r["utilisation_ppm"] == 875000
    assert r["busy_slot_us"] == [25 * (3 * 32 + 16) * 10]


def test_ideal_models_that_fit_together_run_as_alone():
    a = dict(slots=[16, 16], dur=[20, 40], batch=1, slo_us=10**9)
    r = sched.simulate_ideal([a, dict(a)], 1200, 10)
    assert r["forwards"] == [20, 20] and r["utilisation_ppm"] == 1000000


def test_ideal_largest_fitting_sum():
    # shares 10, 12, 22 of 32: {10, 22} fills the GPU, 12 waits
    ms = [dict(slots=[s], dur=[1000], batch=1, slo_us=10**9) for s in (10, 12, 22)]
    r = sched.simulate_ideal(ms, 10, 10)
    assert r["busy_slot_us"] == [100, 0, 220] and r["utilisation_ppm"] == 1000000


def test_ideal_ties_go_to_the_earliest_deadline():
    # two 20-slot models (never together), one 20 us kernel each, 10 us slots,
    # SLOs 100 and 50 us: by hand, model 1 runs [0, 60) (deadlines 50, 70, 90
    # against 100), model 0 [60, 80), model 1 again from 80 (deadline 110 < 180)
    ms = [dict(slots=[20], dur=[20], batch=1, slo_us=100), dict(slots=[20], dur=[20], batch=1, slo_us=50)]
    r = sched.simulate_ideal(ms, 80, 10)
    assert r["forwards"] == [1, 3] and r["late"] == [0, 0]
    r = sched.simulate_ideal(ms, 100, 10)
    assert r["forwards"] == [1, 4]


# ---- temporal sharing (Sec. 6.1's time slices proportional to the SLOs) ----

def _dense(duration, every=10):
    """A request every `every` us: the queue is never empty."""
    return list(range(0, duration, every))


def test_temporal_one_model_closed_form():
    """One model owns the whole cycle (C = its SLO = 10 ms).  From the second
    cycle on, batch 4 (3 ms) runs at 0, 3 and 6 ms into the cycle, then only
    batch 1 (0.9 ms) fits the 1 ms left, then nothing; the first cycle starts
    with one request queued (batch 1 at 0, then batch 4 at 0.9, 3.9 and 6.9
    ms, and the 0.1 ms left fits nothing).  Either way 4 jobs, 13 items and
    9.9 ms busy per cycle: 99% of the time on all slots."""
    m = [dict(slo_us=10000, max_batch=4, rate_per_s=0, table={1: {32: 900}, 4: {32: 3000}})]
    r = sched.simulate(m, 100000, 100000, [_dense(100000)], policy="temporal")
    starts = [(j[0], j[5]) for j in r["log"]]
    assert starts[:8] == [(0, 1), (900, 4), (3900, 4), (6900, 4), (10000, 4), (13000, 4), (16000, 4), (19000, 1)]
    assert r["models"][0]["served"] == 130 and r["models"][0]["planned_runs"] == 40
    assert r["utilisation_ppm"] == 990000


def test_temporal_two_models_hand_worked():
    """SLOs 10 and 30 ms: cycle 10 ms, slices 2.5 and 7.5 ms.  Model 0 fits
    batch 2 (1.8 ms) then nothing in its 0.7 ms left (batch 1 takes 1 ms);
    model 1 fits batch 8 (7 ms).  In the first cycle model 0 starts with one
    request queued (batch 1 at 0) and then has 1.5 ms left (batch 1 again).
    Per cycle 2 + 8 items."""
    m = [dict(slo_us=10000, max_batch=32, rate_per_s=0, table={1: {32: 1000}, 2: {32: 1800}}),
         dict(slo_us=30000, max_batch=8, rate_per_s=0, table={4: {32: 4000}, 8: {32: 7000}})]
    r = sched.simulate(m, 100000, 50000, [_dense(50000), _dense(50000)], policy="temporal")
    assert [(j[0], j[2], j[5]) for j in r["log"][:5]] == [(0, 0, 1), (1000, 0, 1), (2500, 1, 8), (10000, 0, 2),
                                                          (12500, 1, 8)]
    assert r["models"][0]["served"] == 10 and r["models"][1]["served"] == 40


def test_temporal_slices_are_strict():
    """A model with nothing queued leaves its slice idle: the other model
    never runs outside its own slice, even with requests waiting."""
    m = [dict(slo_us=20000, max_batch=8, rate_per_s=0, table={8: {32: 500}}),
         dict(slo_us=20000, max_batch=8, rate_per_s=0, table={8: {32: 500}})]
    r = sched.simulate(m, 100000, 100000, [[], _dense(100000)], policy="temporal")
    assert all(10000 <= j[0] % 20000 and j[1] % 20000 <= 20000 and j[2] == 1 for j in r["log"])
    assert r["models"][1]["served"] == 5 * 20 * 8


def test_temporal_invariants_random():
    """One job at a time, on every slot, inside its model's slice."""
    rng = random.Random(17)
    for _ in range(40):
        n = rng.randint(1, 4)
        models = [dict(slo_us=rng.choice([5000, 10000, 25000, 50000]), max_batch=rng.choice([8, 32]), rate_per_s=0,
                       table={b: {32: rng.randint(100, 4000) * b // 4 + 50} for b in (1, 4, 8, 32)})
                  for _ in range(n)]
        cyc = rng.choice([0, 3000, 20000])
        C = cyc or min(m["slo_us"] for m in models)
        tot = sum(m["slo_us"] for m in models)
        lens = [C * m["slo_us"] // tot for m in models]
        offs = [sum(lens[:i]) for i in range(n)]
        arr = [sorted(rng.randrange(200000) for _ in range(rng.randint(0, 300))) for _ in range(n)]
        r = sched.simulate(models, 100000, 200000, arr, policy="temporal", slice_cycle=cyc)
        log = sorted(r["log"])
        for (s0, e0, i, mask, kind, b), nxt in zip(log, log[1:] + [None]):
            assert mask == (1 << 32) - 1 and kind == 0
            assert nxt is None or nxt[0] >= e0
            k = s0 // C
            assert k * C + offs[i] <= s0 and e0 <= k * C + offs[i] + lens[i]


# ---- GPU% change on SLO violations (Sec. 3.5's dynamic reconfiguration) ----

def test_resize_on_violations_hand_worked():
    """One model at batch 1 whose optimum share (2 slots, 2 ms a request) is
    slower than its arrivals (one every 1.5 ms): requests turn late, and every
    3 late requests (late completions, or starts more than half the SLO after
    arrival) it moves up its table's columns, 2 -> 4 -> 8 slots,
    where 1 ms a request keeps up.  Before the first change every job runs on
    slots 0-1, between the changes on 0-3, after them on 0-7."""
    table = {1: {2: 2000, 4: 1800, 8: 1000}}
    m = [dict(slo_us=5000, max_batch=1, rate_per_s=0, table=table)]
    _, plan = sched.schedule(m, 100000, overprov=0, placement="home")[:2]
    assert sched.schedule(m, 100000, overprov=0, placement="home")[0][0].slots == 2
    arr = list(range(0, 300000, 1500))
    r = sched.simulate(m, 100000, 300000, [arr], overprov=0, placement="home", resize_violations=3)
    st = r["models"][0]
    assert st["resizes"] == 2 and st["final_slots"] == 8
    sizes = [bin(j[3]).count("1") for j in r["log"]]
    assert sizes == sorted(sizes) and sizes[0] == 2 and sizes[-1] == 8 and 4 in sizes
    assert all(j[3] == (1 << bin(j[3]).count("1")) - 1 for j in r["log"])  # home offset 0 kept
    # without the trigger it stays on 2 slots and falls behind
    r0 = sched.simulate(m, 100000, 300000, [arr], overprov=0, placement="home")
    assert r0["models"][0]["resizes"] == 0 and r0["models"][0]["violations"] > st["violations"]


def test_resize_counts_half_slo_waits_at_job_start():
    """A request counts towards the next GPU% change when its job starts
    more than half its SLO after its arrival (the share Eq. meet_half_slo
    leaves to waiting is used up), else when it completes late; never twice.
    One model at batch 1: 1000 us a job on its 2-slot knee (800 us on 4),
    SLO 3000 us, requests at 0, 1, 2, 3 us.  The planned start at 0 finds the
    queue empty and still bounds a fill at 0, so the jobs start at 1, 1001,
    2001 and 3001 us: the third request has waited 1999 us > 1500 at its
    start (and ends 2999 us after arriving: on time), the fourth 2998 us (it
    ends 3998 us after arriving: late, counted once).  Threshold 2: the count
    reaches 2 at the fourth start and the change to 4 slots comes at its end;
    threshold 1: at the end of the third job, so the fourth runs on 4 slots
    (800 us).  Counting late completions alone would give 1 request, so no
    change at threshold 2.  The library's simulation takes the same jobs."""
    table = {1: {2: 1000, 4: 800}}
    m = [dict(slo_us=3000, max_batch=1, rate_per_s=0, table=table)]
    arr = [[0, 1, 2, 3]]
    two = sched.simulate(m, 100000, 20000, arr, overprov=0, placement="home", resize_violations=2)
    assert [(j[0], j[1], bin(j[3]).count("1")) for j in two["log"]] == \
        [(1, 1001, 2), (1001, 2001, 2), (2001, 3001, 2), (3001, 4001, 2)]
    assert two["models"][0]["resizes"] == 1 and two["models"][0]["final_slots"] == 4
    assert two["models"][0]["violations"] == 1
    one = sched.simulate(m, 100000, 20000, arr, overprov=0, placement="home", resize_violations=1)
    assert [(j[0], j[1], bin(j[3]).count("1")) for j in one["log"]] == \
        [(1, 1001, 2), (1001, 2001, 2), (2001, 3001, 2), (3001, 3801, 4)]
    import paper_2304_13541_amd as ds
    for rv, ref in ((2, two), (1, one)):
        lib = ds.simulate(m, 100000, 20000, arr, overprov_slots=0, placement="home", resize_violations=rv)
        assert lib["job_hash"] == ref["job_hash"]
        assert [(s["resizes"], s["final_slots"], s["violations"]) for s in lib["models"]] == \
            [(s["resizes"], s["final_slots"], s["violations"]) for s in ref["models"]]


def test_resize_never_adds_contention():
    """A GPU% change is not made when the larger range would meet the range
    of a model that the current one does not meet.  Model 0 falls behind on
    its 16-slot knee at [0, 16) (1000 us a request, one every 700 us); its
    next columns, 24 and 32 slots, would reach model 1's [16, 32): with model
    1 there it keeps its range, alone it grows to 24 and then 32.  The
    library's simulation takes the same jobs."""
    import paper_2304_13541_amd as ds
    t0 = {1: {16: 1000, 24: 950, 32: 900}}
    t1 = {1: {16: 300, 24: 290, 32: 280}}
    m = [dict(slo_us=5000, max_batch=1, rate_per_s=0, table=t0), dict(slo_us=20000, max_batch=1, rate_per_s=0, table=t1)]
    st, plan = ds.schedule(m, 100000, overprov_slots=0, placement="home")
    assert plan["deployed_slots"] == [16, 16] and plan["home_offset"] == [0, 16]
    arr = [list(range(0, 300000, 700)), list(range(0, 300000, 10000))]
    both = sched.simulate(m, 100000, 300000, arr, overprov=0, placement="home", resize_violations=3)
    assert [s["resizes"] for s in both["models"]] == [0, 0] and both["models"][0]["violations"] > 0
    lib = ds.simulate(m, 100000, 300000, arr, overprov_slots=0, placement="home", resize_violations=3)
    assert lib["job_hash"] == both["job_hash"]
    alone = sched.simulate(m[:1], 100000, 300000, arr[:1], overprov=0, placement="home", resize_violations=3)
    assert alone["models"][0]["resizes"] == 2 and alone["models"][0]["final_slots"] == 32


def test_resize_keeps_ranges_inside_the_gpu_and_disjoint():
    """Random four-model tables under load: a model's size only grows, along
    its table's columns; its range stays inside the slots (a range that
    would pass the last slot ends there); running jobs never share a slot."""
    rng = random.Random(23)
    for trial in range(20):
        n = 4
        models = []
        for _ in range(n):
            cols = sorted(rng.sample(GRID, 6))
            models.append(dict(slo_us=rng.choice([10000, 20000, 40000]), max_batch=8, rate_per_s=0,
                               table={b: {s: int((300 + 2000 * rng.random()) * b ** 0.6 * (32 / s) ** 0.6)
                                          for s in cols} for b in (1, 2, 4, 8)}))
        arr = [sorted(rng.randrange(400000) for _ in range(rng.randint(100, 900))) for _ in range(n)]
        r = sched.simulate(models, 100000, 400000, arr, overprov=0, placement="home", resize_violations=2)
        log = sorted(r["log"])
        for i in range(n):
            sizes = [bin(j[3]).count("1") for j in log if j[2] == i]
            assert sizes == sorted(sizes)
            cols = set().union(*[set(row) for row in models[i]["table"].values()])
            assert all(s in cols for s in set(sizes[1:]) - {sizes[0]})
            # a change at the model's last completion leaves it larger than any job it ran
            fin = r["models"][i]["final_slots"]
            assert not sizes or fin == sizes[-1] or (fin > sizes[-1] and fin in cols)
        for a in range(len(log)):
            for b in range(a + 1, len(log)):
                if log[b][0] >= log[a][1]:
                    break
                assert log[a][3] & log[b][3] == 0
        assert all(m < (1 << 32) for *_, m, _, _ in [(j[0], j[1], j[2], j[3], j[4], j[5]) for j in log])
