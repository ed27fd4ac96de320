"""Host-side checks of the HIP library (no GPU needed): it loads, exports every
entry point its header declares, generates weights bit-identical to the
oracle's independent generator, and makes scheduling decisions identical to
the scheduler oracle's."""
import math
import os
import random
import re

import numpy as np
import pytest

import paper_2304_13541_amd as ds
from oracle import sched

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "dstack.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dstack_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = ds.lib()
    names = declared_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(ds._SIGS)


def test_fraction_to_slots():
    table = {0.1: 3, 0.2: 6, 0.25: 8, 0.3: 10, 0.4: 13, 0.5: 16, 0.6: 19, 0.7: 22, 0.8: 26, 0.9: 29, 1.0: 32,
             0.001: 1}
    for f, s in table.items():
        assert ds.fraction_to_slots(f) == s == min(32, max(1, math.floor(32 * f + 0.5)))
    for bad in (0.0, -0.1, 1.0001, float("nan"), float("inf")):
        with pytest.raises(ds.DStackError) as e:
            ds.fraction_to_slots(bad)
        assert e.value.status == ds.E_INVALID


@pytest.mark.parametrize("arch", ["tinycnn", "resnet50", "mobilenetv2", "lstm2", "vgg19", "bert"])
def test_weights_bit_identical_to_oracle(oracle_mod, arch):
    m = oracle_mod.Model(arch, 1234)
    n = m.num_tensors()
    idxs = {"vgg19": [0, 1, 2, 5, 17, 30, 33, 35, 37],
            "bert": [0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 50, 99, 100, 101, 102]}.get(arch, range(n))
    if arch == "bert":
        assert n == 3 + 12 * 8 + 4
    for i in idxs:
        lib_bits = ds.generate_params(arch, 1234, i)
        assert np.array_equal(lib_bits, m.tensor_bf16(i)), (arch, i)


def test_generate_params_errors():
    with pytest.raises(ds.DStackError) as e:
        ds.generate_params("alexnet", 1, 0)
    assert e.value.status == ds.E_UNSUPPORTED
    with pytest.raises(ds.DStackError) as e:
        ds.generate_params("tinycnn", 1, 99)
    assert e.value.status == ds.E_INVALID


def _lib_vs_oracle(models, period, total=32, overprov=2, placement="lowest"):
    st, got = ds.schedule(models, period, total, overprov, placement)
    choices, jobs, util, ok = sched.schedule(models, period, total, overprov, placement)
    assert (st == ds.OK) == ok
    assert got["batch"] == [c.batch for c in choices]
    assert got["knee_slots"] == [c.slots for c in choices]
    assert got["latency_us"] == [c.latency for c in choices]
    assert got["feasible"] == [int(c.feasible) for c in choices]
    assert got["deployed_slots"] == [min(total, c.slots + overprov) for c in choices]
    assert got["utilisation_ppm"] == util
    assert len(got["jobs"]) == len(jobs)
    for a, b in zip(got["jobs"], jobs):
        assert (a["model"], a["k"], a["release"], a["deadline"], a["start"], a["duration"], a["slots"], a["missed"],
                a["slot_mask"]) == (b.model, b.k, b.release, b.deadline, b.start, b.duration, b.slots,
                                    int(b.missed), b.slot_mask)
    return got


def _amdahl_table(a_us, c_us, batches, slots):
    return {b: {s: int(a_us * (1 + 0.1 * b) + c_us * b / s) for s in slots} for b in batches}


SWEEP_SLOTS = [3, 6, 10, 13, 16, 19, 22, 26, 29, 32]


def test_schedule_parity_config_shaped_tables():
    # two-model mix (ResNet-50-like SLO 25 ms, MobileNetV2-like 15 ms) and the four-model mix
    r50 = dict(slo_us=25000, max_batch=16, rate_per_s=0, table=_amdahl_table(400, 9000, [1, 2, 4, 8, 16], SWEEP_SLOTS))
    mb = dict(slo_us=15000, max_batch=32, rate_per_s=0, table=_amdahl_table(300, 2500, [1, 2, 4, 8, 16, 32], SWEEP_SLOTS))
    _lib_vs_oracle([r50, mb], 100000)
    vgg = dict(slo_us=50000, max_batch=32, rate_per_s=150, table=_amdahl_table(800, 30000, [1, 2, 4, 8], SWEEP_SLOTS))
    lstm = dict(slo_us=30000, max_batch=32, rate_per_s=300, table=_amdahl_table(3000, 2000, [1, 2, 4, 8], SWEEP_SLOTS))
    r50r = dict(r50, rate_per_s=400)
    mbr = dict(mb, rate_per_s=800)
    _lib_vs_oracle([r50r, mbr, vgg, lstm], 100000)
    for ms in ([r50, mb], [r50r, mbr, vgg, lstm]):
        got = _lib_vs_oracle(ms, 100000, placement="home")
        assert got["home_offset"] == sched.home_offsets(got["deployed_slots"], 32)


def test_schedule_parity_paper_table():
    models = [dict(slo_us=25000, max_batch=16, table={16: {3: 8000}}),
              dict(slo_us=50000, max_batch=16, table={16: {4: 28000}}),
              dict(slo_us=100000, max_batch=16, table={16: {5: 55000}})]
    got = _lib_vs_oracle(models, 100000, total=10, overprov=0)
    assert got["utilisation_ppm"] == 595000


def test_schedule_parity_random():
    rnd = random.Random(2026)
    for trial in range(300):
        models = []
        total = rnd.choice([8, 16, 32])
        for _ in range(rnd.randint(1, 6)):
            batches = sorted(rnd.sample([1, 2, 4, 8, 16, 32], rnd.randint(1, 6)))
            slots = sorted(rnd.sample(range(1, total + 1), rnd.randint(1, min(10, total))))
            table = {}
            for b in batches:
                row = {}
                for s in slots:
                    if rnd.random() < 0.9:
                        row[s] = rnd.randint(100, 60000)
                if row:
                    table[b] = row
            if not table:
                continue
            models.append(dict(slo_us=rnd.choice([10000, 15000, 25000, 30000, 50000, 100000]),
                               max_batch=rnd.choice([1, 4, 8, 16, 32]), rate_per_s=rnd.choice([0, 0, 150, 400, 800]),
                               table=table))
        if not models:
            continue
        _lib_vs_oracle(models, rnd.choice([50000, 100000]), total=total, overprov=rnd.choice([0, 2]),
                       placement=rnd.choice(["lowest", "home"]))


def test_schedule_rejects_bad_arguments():
    with pytest.raises(ds.DStackError):
        ds.schedule([dict(slo_us=0, max_batch=1, table={1: {4: 10}})], 100000)
    with pytest.raises(ds.DStackError):
        ds.schedule([dict(slo_us=1000, max_batch=1, table={1: {40: 10}})], 100000)


def test_fc_workspace_bytes():
    """Depth-split plan of the FC kernel on 256 CUs: splits double while the
    grid (16-row tiles x splits) has fewer than 256 blocks and each split
    keeps 96 or more 32-deep steps; the workspace holds splits x B x O fp32
    sums."""
    import paper_2304_13541_amd as ds
    assert ds.fc_workspace_bytes(8, 25088, 40) == 8 * 8 * 40 * 4         # 3 tiles, 784 steps -> 8 splits (98 each)
    assert ds.fc_workspace_bytes(8, 25088, 1000) == 8 * 8 * 1000 * 4     # 63 tiles, 784 steps -> 8 splits (98 each)
    assert ds.fc_workspace_bytes(17, 9216, 33) == 2 * 17 * 33 * 4        # 288 steps -> 2 splits (144; 72 is too few)
    assert ds.fc_workspace_bytes(8, 25088, 4096) == 0                    # 256 tiles: a block per CU already
    assert ds.fc_workspace_bytes(8, 4096, 1000) == 0                     # 128 steps: 64 per split is too few
    assert ds.fc_workspace_bytes(16, 1280, 1000) == 0                    # 40 steps
    assert ds.fc_workspace_bytes(1, 64, 10) == 0                         # 2 steps
    assert ds.fc_workspace_bytes(0, 64, 10) == 0


def test_knee_search_table_parity():
    """dstack_knee_search_table takes the oracle's probes in the oracle's
    order and ends on its knee, on random (not necessarily unimodal) tables
    over random ascending candidate sets."""
    import paper_2304_13541_amd as ds
    rnd = random.Random(31)
    for trial in range(300):
        total = rnd.choice([1, 2, 5, 16, 32])
        cand = sorted(rnd.sample(range(1, total + 1), rnd.randint(1, min(total, 12))))
        table = {s: rnd.randint(50, 40000) for s in cand}
        b, start = rnd.choice([1, 4, 16, 32]), rnd.randint(0, total)
        got = ds.knee_search_table(b, table, total, start, overprov_slots=2)
        k, probes = sched.knee_search(lambda s: table[s], b, cand, start)
        assert got["knee_slots"] == k
        assert got["probes"] == probes and got["n_probes"] == len(probes)
        assert got["deployed_slots"] == min(total, k + 2)
    with pytest.raises(ds.DStackError):  # a latency of 0
        ds.knee_search_table(1, {3: 0, 6: 10})
    with pytest.raises(ds.DStackError):  # a slot count above the total
        ds.knee_search_table(1, {3: 5, 40: 10})


def test_knee_model_parity_random():
    """dstack_knee_model_eval reproduces the analytical-model oracle bit for
    bit (E_t on every candidate, the knee index) on random kernel sequences,
    with and without repetitions and the memory term."""
    from oracle import knee_model as km
    rnd = random.Random(77)
    for trial in range(400):
        k = rnd.randint(1, 60)
        n = [rnd.choice([0.0, float(rnd.randint(1, 300)), rnd.uniform(0.0, 2.0), rnd.uniform(1.0, 900.0)])
             for _ in range(k)]
        tp = [rnd.uniform(0.0, 80.0) for _ in range(k)]
        reps = None if rnd.random() < 0.5 else [float(rnd.randint(0, 4)) for _ in range(k)]
        data = None if rnd.random() < 0.5 else [rnd.uniform(0.0, 1e7) for _ in range(k)]
        m = rnd.choice([0.0, -1.0, rnd.uniform(1.0, 5e4)])
        tnp = rnd.uniform(0.0, 30.0)
        b = float(rnd.randint(0, 32))
        s_values = sorted(rnd.sample(range(1, 300), rnd.randint(1, 20)))
        et, ki = ds.knee_model_eval(n, tp, s_values, tnp, b, reps, data, m)
        et_o, ki_o = km.knee(n, tp, s_values, tnp, b, reps, data, m)
        assert et == et_o and ki == ki_o, trial


def test_knee_model_sequence_parity():
    from oracle import knee_model as km
    for p, b, kmax in [(20, 1, 50), (40, 1, 50), (60, 1, 50), (20, 2, 50), (7, 3, 11), (0, 1, 5), (1000, 32, 53)]:
        assert ds.knee_model_sequence(p, b, kmax) == km.sequence(p, b, kmax)


def test_knee_model_rejects_bad_arguments():
    with pytest.raises(ds.DStackError):
        ds.knee_model_eval([1.0, -2.0], [1.0, 1.0], [1, 2], 0.0)   # negative N_i
    with pytest.raises(ds.DStackError):
        ds.knee_model_eval([1.0], [float("nan")], [1], 0.0)        # non-finite t_p
    with pytest.raises(ds.DStackError):
        ds.knee_model_eval([1.0], [1.0], [0, 2], 0.0)               # S < 1
    with pytest.raises(ds.DStackError):
        ds.knee_model_eval([], [], [1], 0.0)                        # no kernels
    with pytest.raises(ds.DStackError):
        ds.knee_model_sequence(5, 0, 10)                            # b < 1


def test_ideal_schedule_parity_random():
    """dstack_simulate_ideal reproduces the oracle's slotted, preemptive
    kernel-level schedule (every slot's chosen subset through the hash)."""
    rnd = random.Random(91)
    for trial in range(120):
        n = rnd.randint(1, 6)
        total = rnd.choice([8, 16, 32])
        ms = []
        for _ in range(n):
            k = rnd.randint(1, 12)
            ms.append(dict(slots=[rnd.randint(1, total) for _ in range(k)],
                           dur=[rnd.randint(1, 400) for _ in range(k)],
                           batch=rnd.choice([1, 8, 32]), slo_us=rnd.randint(50, 5000)))
        horizon, slot = rnd.randint(1, 20000), rnd.choice([1, 7, 10, 100])
        assert ds.simulate_ideal(ms, horizon, slot, total) == sched.simulate_ideal(ms, horizon, slot, total), trial
    with pytest.raises(ds.DStackError):
        ds.simulate_ideal([dict(slots=[40], dur=[5], batch=1, slo_us=10)], 100, 10)   # share above the total
    with pytest.raises(ds.DStackError):
        ds.simulate_ideal([dict(slots=[4], dur=[0], batch=1, slo_us=10)], 100, 10)    # zero duration
