"""Knee search from live latency and the cost of a GPU% change, on the GPU
(Sec. 3.5, 3.6).  The live search must take exactly the steps of the oracle's
search fed with the latencies it measured; the switch probe's times must be
consistent (creation inside the cold change, an active-standby handoff far
below a cold change)."""
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2304_13541_amd as ds
    from oracle import sched
    return ds, sched


def test_knee_search_live_follows_the_search(env):
    ds, sched = env
    m = ds.Model("mobilenetv2", 7)
    r = m.knee_search(8, start_slots=10, warmup=2, reps=5)
    grid = [3, 6, 10, 13, 16, 19, 22, 26, 29, 32]
    assert [s for s, _ in r["probes"][:2]] == [10, 13]
    assert 2 <= r["n_probes"] <= 8 and r["seconds"] > 0
    measured = dict(r["probes"])

    def latency(s):
        assert s in measured, "the oracle asked for a slot count the library did not measure"
        return measured[s]
    k, probes = sched.knee_search(latency, 8, grid, 10)
    assert k == r["knee_slots"] and probes == r["probes"]
    assert r["deployed_slots"] == min(32, k + 2)
    m.destroy()


def test_switch_probe(env):
    ds, sched = env
    m = ds.Model("resnet50", 7)
    r = m.switch_probe(8, 8, 16, reps=5)
    assert 0 < r["create_us"] < r["cold_us"]
    assert 0 <= r["standby_gap_us"] <= r["standby_gap_max_us"] < r["cold_us"]
    assert r["from_latency_us"] > 0 and r["to_latency_us"] > 0
    print("switch", r)
    m.destroy()


def test_reconfig_argument_errors(env):
    ds, sched = env
    m = ds.Model("tinycnn", 7)
    with pytest.raises(ds.DStackError):
        m.switch_probe(4, 0, 8)
    with pytest.raises(ds.DStackError):
        m.switch_probe(4, 8, 33)
    with pytest.raises(ds.DStackError):
        m.knee_search(64)  # batch above the model's maximum
    with pytest.raises(ds.DStackError):
        m.knee_search(4, fractions=[0.5, 0.3])  # not ascending
    m.destroy()
