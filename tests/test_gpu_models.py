"""Model-level parity on the GPU through the C ABI (dstack_model_load ->
dstack_infer on CU-masked partitions) against the fp64 oracle in parity mode
(bf16 storage at the same points).  Large batches are checked on sampled
items -- {0, b-1} plus seeded picks -- which is exact because batch items are
independent in every layer.

Also: device weights equal the oracle generator's bits; the CU mask of a
partition confines its kernels to 8 CUs per slot spread over all 8 XCDs;
the knee sweep returns a valid table; concurrent models on disjoint
partitions give the same outputs as sequential runs."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.fixture(scope="module")
def env(oracle_mod):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2304_13541_amd as ds
    from tests import gpu_util as gu
    from tests import inputs
    return ds, gu, inputs, oracle_mod, torch


def sample_items(b, seed):
    """{0, b-1} (the last item holds the ragged last pixel tile) plus two
    seeded picks from the items between them; every item when b <= 4."""
    if b <= 4:
        return list(range(b))
    rng = np.random.default_rng(seed)
    picks = rng.choice(np.arange(1, b - 1), size=2, replace=False)
    return sorted({0, b - 1} | {int(p) for p in picks})


def run_model(env, arch, seed, batch, part):
    ds, gu, inputs, oracle, torch = env
    m = ds.Model(arch, seed)
    if arch == "lstm2":
        xb = inputs.sequence_batch(seed + 1, batch)
    else:
        xb = inputs.image_batch(seed + 1, batch, hw=m.info.in_h)
    x = gu.dev_bf16(xb)
    y = gu.empty_f32(m.output_shape(batch))
    m.infer(batch, x, y, part)
    part.synchronize()
    return m, xb, gu.host(y)


def check_against_oracle(env, arch, seed, xb, got, items):
    ds, gu, inputs, oracle, torch = env
    om = oracle.Model(arch, seed)
    if arch == "lstm2":
        ref = om.forward(xb[:, items, :], parity=True)
        g = got[:, items, :]
    else:
        ref = om.forward(xb[items], parity=True)
        g = got[items]
    err = oracle.rel_err(g, ref)
    print("%s items %s rel_err %.3e" % (arch, items, err), flush=True)
    assert np.all(np.isfinite(g))
    assert err <= TOL
    return err


@pytest.mark.parametrize("fraction", [1.0, 0.5, 0.25])
def test_tinycnn_on_partitions(env, fraction):
    """Tiny CNN, batch 4, on 100%, 50% and 25% of the CUs."""
    ds, gu, inputs, oracle, torch = env
    part = ds.Partition(fraction)
    assert part.n_cu == {1.0: 256, 0.5: 128, 0.25: 64}[fraction]
    m, xb, got = run_model(env, "tinycnn", 1010, 4, part)
    check_against_oracle(env, "tinycnn", 1010, xb, got, [0, 1, 2, 3])


@pytest.mark.parametrize("batch,fraction", [(1, 0.4), (8, 1.0), (32, 0.5)])
def test_resnet50(env, batch, fraction):
    ds, gu, inputs, oracle, torch = env
    part = ds.Partition(fraction)
    m, xb, got = run_model(env, "resnet50", 1020, batch, part)
    check_against_oracle(env, "resnet50", 1020, xb, got, sample_items(batch, 7))


@pytest.mark.parametrize("arch,seed,batch,fraction", [
    ("resnet50", 1022, 16, 0.1), ("resnet50", 1022, 16, 0.5), ("resnet50", 1022, 16, 0.7),
    ("mobilenetv2", 1033, 32, 0.5), ("mobilenetv2", 1033, 32, 1.0), ("vgg19", 1042, 8, 0.2),
    ("vgg19", 1042, 8, 1.0), ("lstm2", 1043, 32, 1.0)])
def test_models_at_more_fractions(env, arch, seed, batch, fraction):
    """The launch plans change with the partition's CU count: the measured
    workloads' batches at further points of the sweep grid."""
    ds, gu, inputs, oracle, torch = env
    part = ds.Partition(fraction)
    m, xb, got = run_model(env, arch, seed, batch, part)
    check_against_oracle(env, arch, seed, xb, got, sample_items(batch, seed))


def test_partition_limit_refuses_fifth(env):
    """At most four live partitions (CU-masked streams): the fifth create
    call is refused with E_UNSUPPORTED before any stream exists, and the
    count is back to where it was once they are destroyed."""
    import gc
    ds, gu, inputs, oracle, torch = env
    gc.collect()
    live0, limit = ds.partition_count()
    assert limit == 4 and 0 <= live0 <= limit
    parts = [ds.Partition(slot_offset=8 * i, n_slots=8) for i in range(limit - live0)]
    assert ds.partition_count()[0] == limit
    for kw in (dict(fraction=0.5), dict(slot_offset=0, n_slots=1), dict(slot_mask=0x3)):
        with pytest.raises(ds.DStackError) as e:
            ds.Partition(**kw)
        assert e.value.status == ds.E_UNSUPPORTED
        assert ds.partition_count()[0] == limit
    parts.pop().destroy()
    p = ds.Partition(slot_offset=24, n_slots=8)
    assert ds.partition_count()[0] == limit
    p.destroy()
    for q in parts:
        q.destroy()
    assert ds.partition_count()[0] == live0


def test_partition_destroy_releases_workspaces(env):
    """A model's workspace for a partition (activations, split-K slices,
    captured graphs) is freed when the partition is destroyed."""
    ds, gu, inputs, oracle, torch = env
    m = ds.Model("resnet50", 9)
    x = gu.dev_bf16(inputs.image_batch(3, 16))
    y = gu.empty_f32((16, 1000))
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    for _ in range(3):
        p = ds.Partition(0.5)
        m.infer(16, x, y, p)
        p.synchronize()
        p.destroy()
    free1 = torch.cuda.mem_get_info()[0]
    assert free0 - free1 < 64 * 1024 * 1024, (free0, free1)


def test_mobilenetv2(env):
    ds, gu, inputs, oracle, torch = env
    part = ds.Partition(0.3)
    m, xb, got = run_model(env, "mobilenetv2", 1031, 32, part)
    check_against_oracle(env, "mobilenetv2", 1031, xb, got, sample_items(32, 8))


def test_vgg19(env):
    ds, gu, inputs, oracle, torch = env
    part = ds.Partition(0.5)
    m, xb, got = run_model(env, "vgg19", 1040, 8, part)
    check_against_oracle(env, "vgg19", 1040, xb, got, sample_items(8, 10))


def test_lstm2(env):
    ds, gu, inputs, oracle, torch = env
    part = ds.Partition(0.25)
    m, xb, got = run_model(env, "lstm2", 1041, 32, part)
    check_against_oracle(env, "lstm2", 1041, xb, got, sample_items(32, 9))


@pytest.mark.parametrize("arch", ["tinycnn", "mobilenetv2", "lstm2"])
def test_device_weights_match_oracle_generator(env, arch):
    ds, gu, inputs, oracle, torch = env
    m = ds.Model(arch, 77)
    om = oracle.Model(arch, 77)
    for i in range(m.info.num_tensors):
        assert np.array_equal(m.export_params(i), om.tensor_bf16(i)), (arch, i)


def test_model_info(env):
    ds, gu, inputs, oracle, torch = env
    m = ds.Model("resnet50", 1)
    # about 4.1 GMAC per 224x224 image for ResNet-50
    assert 8.0e9 < m.info.flops_per_item < 8.4e9
    assert m.info.num_params == 25557032 - 2 * 26560
    assert m.info.max_batch == 32


@pytest.mark.parametrize("via_graph", [False, True])
def test_partition_cu_mask_confines_kernels(env, via_graph):
    ds, gu, inputs, oracle, torch = env
    for off, n in [(0, 1), (5, 3), (0, 13), (0, 32), (20, 12)]:
        p = ds.Partition(slot_offset=off, n_slots=n)
        assert p.n_cu == 8 * n
        ids = p.probe_cu_ids(4096, via_graph=via_graph)
        xcc = ids[:, 0] & 0xF
        hw = ids[:, 1]
        cus = {(int(a), int((h >> 13) & 7), int((h >> 12) & 1), int((h >> 8) & 15)) for a, h in zip(xcc, hw)}
        assert len(cus) == 8 * n, (off, n, len(cus))
        assert sorted(set(int(a) for a in xcc)) == list(range(8))
        counts = np.bincount(xcc, minlength=8)
        per_xcd = {x: len({c for c in cus if c[0] == x}) for x in range(8)}
        assert all(v == n for v in per_xcd.values()), per_xcd
        assert counts.min() > 0
        p.destroy()


def test_disjoint_partitions_concurrent_equal_sequential(env):
    ds, gu, inputs, oracle, torch = env
    pa = ds.Partition(slot_offset=0, n_slots=16)
    pb = ds.Partition(slot_offset=16, n_slots=16)
    ma = ds.Model("resnet50", 5)
    mb = ds.Model("mobilenetv2", 6)
    xa = gu.dev_bf16(inputs.image_batch(1, 8))
    xb = gu.dev_bf16(inputs.image_batch(2, 16))
    ya1, yb1 = gu.empty_f32((8, 1000)), gu.empty_f32((16, 1000))
    ma.infer(8, xa, ya1, pa)
    pa.synchronize()
    mb.infer(16, xb, yb1, pb)
    pb.synchronize()
    ya2, yb2 = gu.empty_f32((8, 1000)), gu.empty_f32((16, 1000))
    for _ in range(3):
        ma.infer(8, xa, ya2, pa)
        mb.infer(16, xb, yb2, pb)
    pa.synchronize()
    pb.synchronize()
    assert torch.equal(ya1, ya2) and torch.equal(yb1, yb2)


def test_two_model_mix_launch_configuration(env):
    """The timed two-model mix as the bench launches it: ResNet-50 batch 16
    on slots 0..15 and MobileNetV2 batch 32 on slots 16..31, both replayed
    concurrently (captured graphs, 4 and 7 batches per step); sampled items
    of the last replay of each against the oracle."""
    ds, gu, inputs, oracle, torch = env
    cfg = [("resnet50", 1030, 16, 0, 4), ("mobilenetv2", 1031, 32, 16, 7)]
    runs = []
    for arch, seed, b, off, reps in cfg:
        m = ds.Model(arch, seed)
        p = ds.Partition(slot_offset=off, n_slots=16)
        assert p.n_cu == 128
        xb = inputs.image_batch(seed + 1, b)
        runs.append((arch, seed, b, reps, m, p, xb, gu.dev_bf16(xb), gu.empty_f32((b, 1000))))
    for step in range(max(r[3] for r in runs)):
        for arch, seed, b, reps, m, p, xb, x, y in runs:
            if step < reps:
                m.infer(b, x, y, p)
    for r in runs:
        r[5].synchronize()
    for arch, seed, b, reps, m, p, xb, x, y in runs:
        items = sample_items(b, seed)
        check_against_oracle(env, arch, seed, xb, gu.host(y), items)


def test_four_model_mix_launch_configuration(env):
    """The four-model mix as the live launcher deploys it at the bench's
    plan: ResNet-50 b16 and the LSTM b32 share the stream of slots 0..15,
    VGG-19 b2 runs on slots 16..31, MobileNetV2 b4 on its 3 home slots
    16..18 and, after its GPU% changes, on VGG-19's stream.  All three
    streams replay captured graphs concurrently (the 3-slot range inside the
    16-slot one included); sampled items of each model's last output against
    the oracle."""
    import gc
    ds, gu, inputs, oracle, torch = env
    gc.collect()  # earlier tests' partitions count against the four live streams
    parts = {"a": ds.Partition(slot_offset=0, n_slots=16), "b": ds.Partition(slot_offset=16, n_slots=16),
             "c": ds.Partition(slot_offset=16, n_slots=3)}
    assert [parts[k].n_cu for k in "abc"] == [128, 128, 24]
    # (arch, seed, batch, partitions it runs on); seeds as the bench's mix
    cfg = [("resnet50", 1050, 16, "a"), ("mobilenetv2", 1051, 4, "cb"), ("vgg19", 1052, 2, "b"), ("lstm2", 1053, 32, "a")]
    runs = []
    for arch, seed, b, on in cfg:
        m = ds.Model(arch, seed)
        xb = inputs.sequence_batch(seed + 1, b) if arch == "lstm2" else inputs.image_batch(seed + 1, b, hw=m.info.in_h)
        ys = [gu.empty_f32(m.output_shape(b)) for _ in on]
        runs.append((arch, seed, b, on, m, xb, gu.dev_bf16(xb), ys))
    for _ in range(3):
        for arch, seed, b, on, m, xb, x, ys in runs:
            for k, y in zip(on, ys):
                m.infer(b, x, y, parts[k])
    for p in parts.values():
        p.synchronize()
    try:
        for arch, seed, b, on, m, xb, x, ys in runs:
            for k, y in zip(on, ys):  # each partition's plans (tiles, splits) are its own
                print("%s on partition %s" % (arch, k), flush=True)
                check_against_oracle(env, arch, seed, xb, gu.host(y), sample_items(b, seed))
    finally:
        for p in parts.values():
            p.destroy()


@pytest.mark.parametrize("arch,batch,fraction", [("mobilenetv2", 4, 0.25), ("resnet50", 2, 0.5), ("lstm2", 3, 0.3)])
def test_graph_replays_equal_eager(env, arch, batch, fraction):
    """dstack_infer replays a captured graph; dstack_profile_layers runs the
    same kernels eagerly.  Every replay, with eager work and synchronisation
    in between, must equal the eager result bit for bit."""
    ds, gu, inputs, oracle, torch = env
    m = ds.Model(arch, 21)
    p = ds.Partition(fraction)
    xb = inputs.sequence_batch(5, batch) if arch == "lstm2" else inputs.image_batch(5, batch)
    x = gu.dev_bf16(xb)
    y_eager = gu.empty_f32(m.output_shape(batch))
    m.profile_layers(batch, x, y_eager, p)
    ref = y_eager.clone()
    y = gu.empty_f32(m.output_shape(batch))
    for rep in range(4):
        y.fill_(float("nan"))
        torch.cuda.synchronize()
        m.infer(batch, x, y, p)
        p.synchronize()
        assert torch.equal(y, ref), (arch, rep)
        m.profile_layers(batch, x, y_eager, p)  # eager work between replays
        assert torch.equal(y_eager, ref)


def test_knee_sweep_tiny(env):
    ds, gu, inputs, oracle, torch = env
    m = ds.Model("tinycnn", 3)
    r = m.knee_sweep(4, [1.0, 0.5, 0.25], warmup=3, reps=21)
    assert r["slots"] == [32, 16, 8]
    assert all(L >= 1 for L in r["latency_us"])
    from oracle import sched
    row = dict(zip(r["slots"], r["latency_us"]))
    assert r["knee_slots"] == sched.knee(row, 4)
    assert r["deployed_slots"] == min(32, r["knee_slots"] + 2)


def test_infer_argument_errors(env):
    ds, gu, inputs, oracle, torch = env
    m = ds.Model("tinycnn", 3)
    p = ds.Partition(1.0)
    x = gu.dev_bf16(inputs.image_batch(1, 4, hw=32))
    y = gu.empty_f32((4, 10))
    with pytest.raises(ds.DStackError) as e:
        m.infer(33, x, y, p)
    assert e.value.status == ds.E_INVALID
    with pytest.raises(ds.DStackError) as e:
        m.infer(0, x, y, p)
    assert e.value.status == ds.E_INVALID
    with pytest.raises(ds.DStackError) as e:
        ds.Model("alexnet", 1)
    assert e.value.status == ds.E_UNSUPPORTED
    with pytest.raises(ds.DStackError) as e:
        ds.Partition(1.5)
    assert e.value.status == ds.E_INVALID
