"""Live launcher (dstack_serve) on the GPU: the session plan plus the FOD fill
of Sec. 6.1.2 driving real batches on each model's home CU range.

Timing tables come from the knee sweep of the models themselves; requests are
Poisson traces.  Checked: every request is served or counted unserved; each
job runs on its model's home range with a batch from the grid; one model
never has two jobs at once and jobs whose ranges meet never overlap in time;
nothing starts after the trace; the served outputs equal an eager inference
of the same input rows.  Decision parity: the launcher's own trigger log
(each completion seen, planned or slice start due and arrival admitted,
with the clock value its decision used) replayed through the scheduler
oracle starts exactly the same jobs (time, model, batch, slots, kind), for
the D-STACK policy and for temporal sharing on the whole GPU."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2304_13541_amd as ds
    from oracle import sched
    from tests.inputs import poisson_arrivals
    return ds, sched, poisson_arrivals, torch


FRACTIONS = [0.25, 0.5, 0.75, 1.0]


def measured_table(ds, m, batches):
    table = {}
    for b in batches:
        r = m.knee_sweep(b, FRACTIONS, warmup=3, reps=10)
        table[b] = {s: max(1, int(L)) for s, L in zip(r["slots"], r["latency_us"])}
    return table


def test_serve_two_models(env):
    ds, sched, poisson_arrivals, torch = env
    models = [ds.Model("tinycnn", 7), ds.Model("tinycnn", 8)]
    batches = [1, 2, 4]
    tables = []
    for m in models:
        tab = measured_table(ds, m, batches)
        tables.append(dict(slo_us=4000, max_batch=4, rate_per_s=0, table=tab))
    duration = 300_000
    arrivals = [poisson_arrivals(11, 3000, duration), poisson_arrivals(12, 1500, duration)]
    g = torch.Generator(device="cuda").manual_seed(3)
    xs = [torch.randn(m.input_shape(4), device="cuda", generator=g).to(torch.bfloat16) for m in models]
    ys = [torch.zeros(m.output_shape(4), device="cuda", dtype=torch.float32) for m in models]
    r = ds.serve(models, tables, xs, ys, period_us=10_000, duration_us=duration, arrivals=arrivals)
    torch.cuda.synchronize()

    st, plan = ds.schedule(tables, 10_000, placement="home")
    homes = [sched.range_mask(o, d) for o, d in zip(plan["home_offset"], plan["deployed_slots"])]
    assert len(r["log"]) == r["n_jobs"] > 0
    for i, s in enumerate(r["models"]):
        assert s["served"] + s["unserved"] == len(arrivals[i])
        assert s["violations"] >= s["unserved"]
        assert s["planned_runs"] + s["fod_runs"] == sum(1 for j in r["log"] if j["model"] == i)
    for j in r["log"]:
        assert j["slot_mask"] == homes[j["model"]]
        assert j["batch"] in batches and j["start_us"] < duration
        assert j["end_us"] >= j["start_us"] and j["gpu_us"] > 0
    for a in r["log"]:
        for b in r["log"]:
            if a is b:
                continue
            overlap = a["start_us"] < b["end_us"] and b["start_us"] < a["end_us"]
            if overlap:
                assert a["model"] != b["model"]
                assert a["slot_mask"] & b["slot_mask"] == 0
    assert sum(s["served"] for s in r["models"]) > 0.9 * sum(len(a) for a in arrivals)

    # the last job of each model wrote its first b output rows from the first b input rows
    for i, m in enumerate(models):
        b = [j for j in r["log"] if j["model"] == i][-1]["batch"]
        ref = torch.zeros_like(ys[i])
        p = ds.Partition(1.0)
        m.infer(b, xs[i], ref, p)
        p.synchronize()
        got, want = ys[i][:b].float().cpu().numpy(), ref[:b].float().cpu().numpy()
        assert np.max(np.abs(got - want)) <= 1e-2 * max(1e-6, np.max(np.abs(want)))
        p.destroy()
    for m in models:
        m.destroy()


@pytest.mark.parametrize("policy", ["dstack", "temporal"])
def test_serve_decisions_replay_through_the_oracle(env, policy):
    ds, sched, poisson_arrivals, torch = env
    models = [ds.Model("tinycnn", 17), ds.Model("mobilenetv2", 18)]
    tables = [dict(slo_us=4000, max_batch=4, rate_per_s=0, table=measured_table(ds, models[0], [1, 2, 4])),
              dict(slo_us=6000, max_batch=8, rate_per_s=0, table=measured_table(ds, models[1], [1, 2, 4, 8]))]
    duration = 300_000
    arrivals = [poisson_arrivals(21, 2500, duration), poisson_arrivals(22, 2000, duration)]
    g = torch.Generator(device="cuda").manual_seed(4)
    xs = [torch.randn(m.input_shape(t["max_batch"]), device="cuda", generator=g).to(torch.bfloat16)
          for m, t in zip(models, tables)]
    ys = [torch.zeros(m.output_shape(t["max_batch"]), device="cuda", dtype=torch.float32)
          for m, t in zip(models, tables)]
    r = ds.serve(models, tables, xs, ys, period_us=10_000, duration_us=duration, arrivals=arrivals, policy=policy,
                 event_capacity=1 << 16)
    torch.cuda.synchronize()
    assert r["n_events"] == len(r["events"]) and r["n_jobs"] == len(r["log"]) > 20
    rep = sched.simulate(tables, 10_000, duration, arrivals, placement="home" if policy == "dstack" else "lowest",
                         policy=policy, replay_events=r["events"])
    live = sorted((j["start_us"], j["model"], j["batch"], j["slot_mask"], j["kind"]) for j in r["log"])
    replayed = sorted((j[0], j[2], j[5], j[3], j[4]) for j in rep["log"])
    print(policy, "jobs", len(live), "events", len(r["events"]), flush=True)
    assert live == replayed
    assert [s["plan_skips"] for s in r["models"]] == rep["plan_skips"]
    if policy == "temporal":
        assert all(j["slot_mask"] == (1 << 32) - 1 for j in r["log"])
        starts = sorted((j["start_us"], j["end_us"]) for j in r["log"])
        assert all(b[0] >= a[1] for a, b in zip(starts, starts[1:]))  # one job at a time
    for m in models:
        m.destroy()


def test_serve_rejects_bad_arguments(env):
    ds, sched, poisson_arrivals, torch = env
    m = ds.Model("tinycnn", 7)
    tab = dict(slo_us=4000, max_batch=4, table={1: {8: 100, 32: 80}, 4: {8: 200, 32: 120}})
    x = torch.zeros(m.input_shape(4), device="cuda", dtype=torch.bfloat16)
    y = torch.zeros(m.output_shape(4), device="cuda", dtype=torch.float32)
    with pytest.raises(ds.DStackError) as e:  # five models: more than four masked streams
        ds.serve([m] * 5, [tab] * 5, [x] * 5, [y] * 5, 10_000, 50_000, [[]] * 5)
    assert e.value.status == ds.E_UNSUPPORTED
    with pytest.raises(ds.DStackError) as e:  # unsorted trace
        ds.serve([m], [tab], [x], [y], 10_000, 50_000, [[30, 10]])
    assert e.value.status == ds.E_INVALID
    with pytest.raises(ds.DStackError) as e:  # table batch above the model's maximum
        ds.serve([m], [dict(tab, max_batch=10_000)], [x], [y], 10_000, 50_000, [[]])
    assert e.value.status == ds.E_INVALID
    m.destroy()


def test_serve_resizes_on_violations_and_replays(env):
    """GPU% change on SLO violations in the live launcher: a tight SLO for
    MobileNetV2 under load makes its requests late; every 3 late ones it
    moves to a larger home range on a new CU-masked stream.  The trigger log
    replayed through the oracle (which applies the same rule to the logged
    completion times) starts exactly the same jobs, and the model's job
    ranges only grow."""
    ds, sched, poisson_arrivals, torch = env
    models = [ds.Model("tinycnn", 27), ds.Model("mobilenetv2", 28)]
    tables = [dict(slo_us=4000, max_batch=4, rate_per_s=0, table=measured_table(ds, models[0], [1, 2, 4])),
              dict(slo_us=1500, max_batch=8, rate_per_s=0, table=measured_table(ds, models[1], [1, 2, 4, 8]))]
    duration = 300_000
    arrivals = [poisson_arrivals(31, 1500, duration), poisson_arrivals(32, 30000, duration)]
    xs = [torch.zeros(m.input_shape(t["max_batch"]), device="cuda", dtype=torch.bfloat16) for m, t in zip(models, tables)]
    ys = [torch.zeros(m.output_shape(t["max_batch"]), device="cuda", dtype=torch.float32) for m, t in zip(models, tables)]
    r = ds.serve(models, tables, xs, ys, period_us=10_000, duration_us=duration, arrivals=arrivals, overprov_slots=0,
                 event_capacity=1 << 16, resize_violations=3)
    torch.cuda.synchronize()
    rep = sched.simulate(tables, 10_000, duration, arrivals, overprov=0, placement="home",
                         replay_events=r["events"], resize_violations=3)
    live = sorted((j["start_us"], j["model"], j["batch"], j["slot_mask"], j["kind"]) for j in r["log"])
    replayed = sorted((j[0], j[2], j[5], j[3], j[4]) for j in rep["log"])
    print("resizes", [s["resizes"] for s in r["models"]], "final slots", [s["final_slots"] for s in r["models"]],
          "jobs", len(live), flush=True)
    assert live == replayed
    assert [s["resizes"] for s in r["models"]] == rep["resizes"]
    assert [s["final_slots"] for s in r["models"]] == rep["final_slots"]
    assert r["models"][1]["resizes"] > 0
    sizes = [bin(j[3]).count("1") for j in live if j[1] == 1]
    assert sizes == sorted(sizes) and sizes[-1] > sizes[0]
    for m in models:
        m.destroy()


def test_serve_shares_ranges_and_changes_without_waiting(env):
    """Models whose home ranges are identical share one CU-masked stream, so
    a four-model run fits beside a partition the caller holds (three
    streams for four models); a GPU% change into a range another model
    already runs on takes effect as soon as it is decided, and so does one
    whose standby stream was made ahead when the limit leaves room; the
    trigger log replays through the oracle to the same jobs, and no
    partition outlives the call.  Synthetic tables put three models on
    16-slot ranges [0, 16), [16, 32), [0, 16) and MobileNetV2 on 8 slots at
    16; its changes go to [16, 28) (a new stream) and [16, 32) (model 1's),
    and stop there: [8, 32) would meet the ranges of models 0 and 2."""
    ds, sched, poisson_arrivals, torch = env
    live0, limit = ds.partition_count()
    if live0 + 4 > limit:
        pytest.skip("partitions of other tests are live")
    tiny = {b: {8: 300 + 10 * b, 16: 150 + 5 * b, 24: 140 + 5 * b, 32: 135 + 5 * b} for b in (1, 2, 4)}
    mb = {b: {8: 400 + 50 * b, 12: 380 + 45 * b, 16: 350 + 40 * b, 24: 340 + 38 * b, 32: 335 + 37 * b}
          for b in (1, 2, 4, 8)}
    models = [ds.Model("tinycnn", 41 + i) for i in range(3)] + [ds.Model("mobilenetv2", 44)]
    tables = [dict(slo_us=20000, max_batch=4, rate_per_s=0, table=tiny) for _ in range(3)] + \
        [dict(slo_us=1500, max_batch=8, rate_per_s=0, table=mb)]
    st, plan = ds.schedule(tables, 10_000, overprov_slots=0, placement="home")
    assert plan["home_offset"] == [0, 16, 0, 16] and plan["deployed_slots"] == [16, 16, 16, 8]
    duration = 300_000
    arrivals = [poisson_arrivals(51 + i, 500, duration) for i in range(3)] + [poisson_arrivals(54, 30000, duration)]
    xs = [torch.zeros(m.input_shape(t["max_batch"]), device="cuda", dtype=torch.bfloat16) for m, t in zip(models, tables)]
    ys = [torch.zeros(m.output_shape(t["max_batch"]), device="cuda", dtype=torch.float32) for m, t in zip(models, tables)]

    def run(held):
        r = ds.serve(models, tables, xs, ys, period_us=10_000, duration_us=duration, arrivals=arrivals,
                     overprov_slots=0, event_capacity=1 << 16, resize_violations=3)
        torch.cuda.synchronize()
        assert ds.partition_count()[0] == live0 + held
        rep = sched.simulate(tables, 10_000, duration, arrivals, overprov=0, placement="home",
                             replay_events=r["events"], resize_violations=3)
        live = sorted((j["start_us"], j["model"], j["batch"], j["slot_mask"], j["kind"]) for j in r["log"])
        replayed = sorted((j[0], j[2], j[5], j[3], j[4]) for j in rep["log"])
        assert live == replayed
        assert [s["resizes"] for s in r["models"]] == rep["resizes"]
        # delay of each change of MobileNetV2 after the completion that decided it
        delays, last_done = [], None
        for e in r["events"]:
            if e["model"] != 3:
                continue
            if e["kind"] == 0:
                last_done = e["t_us"]
            elif e["kind"] == 3:
                delays.append((bin(e["slot_mask"]).count("1"), e["t_us"] - last_done))
        print("held %d: resizes %s, changes (slots, us after the deciding completion) %s" %
              (held, [s["resizes"] for s in r["models"]], delays), flush=True)
        assert [s["resizes"] for s in r["models"]] == [0, 0, 0, 2] and [d[0] for d in delays] == [12, 16]
        assert delays[1][1] < 2000  # into [16, 32), the range model 1 runs on
        return delays

    held = ds.Partition(slot_offset=0, n_slots=4)  # three streams for the four models fit beside it
    try:
        run(1)
    finally:
        held.destroy()
    run(0)
    for m in models:
        m.destroy()
