"""Live launcher (dstack_serve) on the GPU: the session plan plus the FOD fill
of Sec. 6.1.2 driving real batches on each model's home CU range.

Timing tables come from the knee sweep of the models themselves; requests are
Poisson traces.  Checked: every request is served or counted unserved; each
job runs on its model's home range with a batch from the grid; one model
never has two jobs at once and jobs whose ranges meet never overlap in time;
nothing starts after the trace; the served outputs equal an eager inference
of the same input rows."""
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
