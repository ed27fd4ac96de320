"""Benchmark: multi-DNN spatial multiplexing on one MI355X.

Headline workload (one GPU): ResNet-50 v1.5 at batch 16 (SLO 25 ms) and
MobileNetV2 1.0 at batch 32 (SLO 15 ms), synthetic N(0,1) 224x224x3 bf16
images standing in for ImageNet, random-weight bf16 models.

Setup (untimed): load both models and sweep each over batches {1,2,4,8,16[,32]}
x CU fractions 10%..100% (knee sweep: median latency of 20 timed forwards per
point).  At the workload's batch each model's knee is the efficacy optimum
b/(L^2 s) over the swept slot counts; it is deployed with 2 slots of
over-provisioning (shrunk proportionally when the models do not fit together).
The CU-masked partitions (disjoint slot ranges) are packed over the 32 slots
round-robin over the models, up to 4 partitions (more concurrently active
masked queues are avoided on this part).  The SLO-constrained (batch, slots)
choice of dstack_schedule over the whole table is reported alongside.

One step = ceil(100 ms / SLO) batches of each partition's model, back to back,
all partitions concurrently (closed loop).  Value = aggregate inferences/s
over K steps.  The time-sliced full-GPU baseline runs the same per-model batch
counts one batch at a time on an unmasked partition.  Per-kernel HIP-event
timing on each partition's stream gives the conv MFMA TFLOP/s at the knee and
the roofline fraction of the dominant kernel (the implicit-GEMM convolution);
each partition's batch time alone vs in the mix gives the interference.
Rooflines per model use P(n) = 2516.6 TFLOP/s * n/256 and BW(n) measured by a
device copy on the partition's stream ("per_model[].roofline"); "mix" holds
the same-work makespan ratio, the FLOP-weighted work rate, the CU-weighted
roofline busy fraction and the same models on unmasked concurrent streams.

Also reported (not the headline): the tiny CNN at 100/50/25% ("config1");
ResNet-50 at batch 1/8/32 over the 10 fractions ("config2"); for each
headline model the knee found by a binary search from 30% against the sweep's
knee, and the cost of a GPU% change, cold and active-standby
("reconfiguration"); the VGG-19 batch 8 + LSTM batch 32 pair in the same
closed-loop form ("config4"), and the four-model Poisson mix (ResNet-50,
MobileNetV2, VGG-19, LSTM at 400/800/150/300 req/s, SLOs 25/15/50/30 ms,
100 ms sessions) through the live launcher dstack_serve for 10 s at the
stated rates plus a capacity sweep of 2 s runs at k x the rates ("config5");
--headline-only skips these.
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "aggregate inferences/s (multi-DNN, one GPU) + conv MFMA TFLOP/s at knee CU%"
PEAK_BF16_TFLOPS = 2516.6   # dense bf16 MFMA, 256 CUs at 2.4 GHz
FRACTIONS = [0.1 * i for i in range(1, 11)]
PERIOD_US = 100000
MAX_PARTITIONS = 4
OVERPROV = 2

MODELS = [
    # arch, seed, SLO us, workload batch, batches swept
    ("resnet50", 1030, 25000, 16, [1, 2, 4, 8, 16]),
    ("mobilenetv2", 1031, 15000, 32, [1, 2, 4, 8, 16, 32]),
]

TRAFFIC_FILE = os.path.join(ROOT, "profiles", "conv_igemm_mix_traffic.md")
CONV_SRC = os.path.join(ROOT, "paper_2304_13541_amd", "csrc", "conv_igemm.hip")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--sweep-warmup", type=int, default=5)
    p.add_argument("--sweep-reps", type=int, default=20)
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the oracle CPU baseline")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--table", default=None, help="load a timing table JSON instead of sweeping")
    p.add_argument("--save-table", default=None)
    p.add_argument("--steps4", type=int, default=40, help="steps of the VGG-19 + LSTM pair")
    p.add_argument("--serve-seconds", type=float, default=10.0, help="four-model mix at the stated rates")
    p.add_argument("--capacity-seconds", type=float, default=2.0, help="each point of the capacity sweep")
    p.add_argument("--headline-only", action="store_true", help="skip the GPU%% reconfiguration probes, the VGG-19 + LSTM pair and the four-model mix")
    return p.parse_args()


def sweep_tables(models, args):
    tables = []
    for (arch, seed, slo, b_work, batches), m in zip(MODELS, models):
        tab, knees = {}, {}
        for b in batches:
            r = m.knee_sweep(b, FRACTIONS, warmup=args.sweep_warmup, reps=args.sweep_reps)
            tab[b] = dict(zip(r["slots"], r["latency_us"]))
            knees[b] = r["knee_slots"]
        tables.append(dict(arch=arch, table=tab, knee_slots_per_batch=knees))
    return tables


def measured_traffic():
    """HBM bytes per conv launch from the committed FETCH_SIZE/WRITE_SIZE
    summary, or None when the kernel source changed since it was taken."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and line.split(":")[0].strip() in ("source_sha256", "traffic_bytes_per_launch"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip().strip("`")
    sha = hashlib.sha256(open(CONV_SRC, "rb").read()).hexdigest()
    if vals.get("source_sha256") != sha or "traffic_bytes_per_launch" not in vals:
        return None
    return float(vals["traffic_bytes_per_launch"])


def cpu_baseline(budget_s, sched_in):
    """The oracle, as it stands, on the host cores: sampled items of the same
    workload (batch items are independent), parity mode; and the scheduler
    oracle's time for the same scheduling decision as the library's."""
    import oracle
    from oracle import sched as osched
    from tests import inputs
    t_s = time.perf_counter()
    osched.schedule(sched_in, PERIOD_US)
    sched_s = time.perf_counter() - t_s
    done, t0 = 0, time.perf_counter()
    models = {a: oracle.Model(a, s) for a, s, *_ in MODELS}
    i = 0
    while True:
        arch, seed = MODELS[i % 2][0], MODELS[i % 2][1]
        models[arch].forward(inputs.image_batch(seed + 1 + i, 1), parity=True)
        done += 1
        i += 1
        el = time.perf_counter() - t0
        if el >= budget_s and i % 2 == 0:
            break
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return dict(value=done / el, unit="inferences/s", cores=threads, kind="oracle",
                sample="%d single 224x224 images alternating ResNet-50 / MobileNetV2 (fp64 oracle, parity mode), "
                       "%.1f s" % (done, el), scheduler_oracle_seconds=sched_s)


def knee_at(row, b):
    """Efficacy optimum b / (L^2 s) over a {slots: L} row, ties to fewer slots."""
    best = None
    for s in sorted(row):
        L = row[s]
        if best is None or b * row[best] ** 2 * best > b * L * L * s:
            best = s
    return best


def bw_probe(torch, part, mib=512, reps=5):
    """HBM bandwidth available to a partition: a plain device copy on its
    stream (bytes read + written per second, GB/s).  BW(n) of the roofline."""
    st = part.torch_stream()
    n = mib * 1024 * 1024 // 4
    with torch.cuda.stream(st):
        a = torch.zeros(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(reps):
            b.copy_(a)
        e1.record(st)
    torch.cuda.synchronize()
    gbs = 2.0 * n * 4 * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a, b
    return gbs


def model_roofline(ds, recs, n_cu, bw_gbs, latency_us):
    """Roofline of one model's forward on a partition of n_cu CUs: MFMA peak
    P(n) = 2516.6 TFLOP/s * n/256, HBM BW(n) measured; per layer the bound is
    max(FLOP/P, bytes/BW); conv layers at or above the ridge P/BW are judged
    against MFMA, the rest and the memory-bound kernels against BW."""
    P = PEAK_BF16_TFLOPS * 1e12 * n_cu / 256
    BW = bw_gbs * 1e9
    ridge = P / BW
    t_roof = sum(max(r["flops"] / P, r["bytes"] / BW) for r in recs)
    t_kern = sum(r["ms"] for r in recs) * 1e-3
    mfma_bound = [r for r in recs if r["kind"] == 0 and r["bytes"] > 0 and r["flops"] / r["bytes"] >= ridge]
    mb_ms = sum(r["ms"] for r in mfma_bound)
    conv_mfma_frac = sum(r["flops"] for r in mfma_bound) / (mb_ms * 1e-3) / P if mb_ms > 0 else None
    hbm = {}
    for r in recs:
        if r in mfma_bound:
            continue
        name = "conv_below_ridge" if r["kind"] == 0 else ds.KIND_NAMES[r["kind"]]
        d = hbm.setdefault(name, dict(n=0, ms=0.0, bytes=0.0))
        d["n"] += 1
        d["ms"] += r["ms"]
        d["bytes"] += r["bytes"]
    for d in hbm.values():
        d["achieved_gbs"] = d["bytes"] / (d["ms"] * 1e-3) / 1e9 if d["ms"] > 0 else None
        d["hbm_frac"] = d["achieved_gbs"] / bw_gbs if d["achieved_gbs"] else None
    return dict(n_cu=n_cu, hbm_gbs_measured=bw_gbs, mfma_peak_tflops=P / 1e12, ridge_flop_per_byte=ridge,
                t_roof_us=1e6 * t_roof, kernel_sum_us=1e6 * t_kern, latency_us=latency_us,
                model_roofline_frac=1e6 * t_roof / latency_us if latency_us else None,
                kernel_roofline_frac=t_roof / t_kern if t_kern > 0 else None,
                conv_mfma_frac=conv_mfma_frac, conv_mfma_frac_target=0.6, mfma_bound_conv_layers=len(mfma_bound),
                hbm_bound=hbm)


def fit_slots(dep, total):
    """Deployed slot counts that fit together: shrink proportionally (round
    half-up), then take slots from the largest until the sum fits."""
    if sum(dep) <= total:
        return list(dep)
    tot = sum(dep)
    out = [max(1, int(math.floor(s * total / tot + 0.5))) for s in dep]
    while sum(out) > total:
        out[out.index(max(out))] -= 1
    return out


def pack_lanes(dep, total, max_parts):
    """Disjoint (model, slot offset, slots) partitions, round-robin over the
    models while they fit, at most max_parts of them."""
    lanes, off, i, misses, n = [], 0, 0, 0, len(dep)
    while misses < n and len(lanes) < max_parts:
        mi = i % n
        if off + dep[mi] <= total:
            lanes.append((mi, off, dep[mi]))
            off += dep[mi]
            misses = 0
        else:
            misses += 1
        i += 1
    return lanes


class Mix:
    """Closed-loop concurrent run of several models on disjoint CU-masked
    partitions, and the time-sliced full-GPU run of the same work."""

    def __init__(self, ds, torch, models, batch, xs, out_shapes, lanes, reps):
        from tests import gpu_util as gu
        self.ds, self.torch, self.models, self.batch, self.xs = ds, torch, models, batch, xs
        self.lanes, self.reps = lanes, reps
        self.parts = [ds.Partition(slot_offset=o, n_slots=s) for _, o, s in lanes]
        self.ys = [gu.empty_f32(out_shapes[mi]) for mi, _, _ in lanes]
        self.lane_count = [sum(1 for l in lanes if l[0] == mi) for mi in range(len(models))]
        self.items_per_step = sum(reps[mi] * batch[mi] for mi, _, _ in lanes)

    def _sync(self, parts):
        for p in parts:
            p.synchronize()
        self.torch.cuda.synchronize()

    def run(self, steps, lanes=None):
        lanes = range(len(self.lanes)) if lanes is None else lanes
        for _ in range(steps):
            for li in lanes:
                mi = self.lanes[li][0]
                for _r in range(self.reps[mi]):
                    self.models[mi].infer(self.batch[mi], self.xs[mi], self.ys[li], self.parts[li])

    def timed(self, steps, warmup, lanes=None):
        """Wall time of `steps` closed-loop steps; each lane's own span (its
        partition stream, from the host's start to its last batch) is kept in
        self.lane_s."""
        sel = list(range(len(self.lanes))) if lanes is None else list(lanes)
        self.run(warmup, lanes)
        self._sync(self.parts)
        ev = [(self.torch.cuda.Event(enable_timing=True), self.torch.cuda.Event(enable_timing=True)) for _ in sel]
        streams = [self.parts[li].torch_stream() for li in sel]
        for (e0, _), s in zip(ev, streams):
            e0.record(s)
        t0 = time.perf_counter()
        self.run(steps, lanes)
        for (_, e1), s in zip(ev, streams):
            e1.record(s)
        self._sync(self.parts)
        dt = time.perf_counter() - t0
        self.lane_s = {li: e0.elapsed_time(e1) / 1e3 for li, (e0, e1) in zip(sel, ev)}
        return dt

    def timesliced(self, steps, warmup, out_shapes):
        from tests import gpu_util as gu
        full = self.ds.Partition(1.0)
        yf = [gu.empty_f32(sh) for sh in out_shapes]

        def go(k):
            for _ in range(k):
                for mi, m in enumerate(self.models):
                    for _r in range(self.lane_count[mi] * self.reps[mi]):
                        m.infer(self.batch[mi], self.xs[mi], yf[mi], full)
        go(warmup)
        full.synchronize()
        t0 = time.perf_counter()
        go(steps)
        full.synchronize()
        dt = time.perf_counter() - t0
        full.destroy()
        return dt

    def interference(self, steps, warmup, t_mix, mix_steps):
        """Per lane: time per batch alone on its partition (steps steps) vs in
        the mix (the lane's own span in the timed mix over its batches there;
        call right after the timed mix), and the mix's wall time per batch of
        the lane (the step is set by the slowest lane)."""
        mix_lane_s = dict(self.lane_s)
        out = []
        for li, (mi, o, s) in enumerate(self.lanes):
            alone = self.timed(steps, warmup, [li]) / (steps * self.reps[mi])
            mixed = mix_lane_s[li] / (mix_steps * self.reps[mi])
            wall = t_mix / (mix_steps * self.reps[mi])
            out.append(dict(lane=li, model=mi, slot_offset=o, slots=s, alone_us=1e6 * alone, mixed_us=1e6 * mixed,
                            slowdown=mixed / alone, mix_wall_us_per_batch=1e6 * wall))
        return out

    def destroy(self):
        for p in self.parts:
            p.destroy()


def layer_stats(ds, m, batch, x, y, part):
    """Per-kind kernel totals of three profiled forwards (HIP events on the partition's stream)."""
    recs = m.profile_layers(batch, x, y, part)
    for _ in range(2):
        for r, r2 in zip(recs, m.profile_layers(batch, x, y, part)):
            r["ms"] += r2["ms"]
    for r in recs:
        r["ms"] /= 3.0
    by_kind = {}
    for r in recs:
        d = by_kind.setdefault(ds.KIND_NAMES[r["kind"]], dict(n=0, ms=0.0, flops=0.0, bytes=0.0))
        d["n"] += 1
        d["ms"] += r["ms"]
        d["flops"] += r["flops"]
        d["bytes"] += r["bytes"]
    return recs, by_kind


def config1(ds):
    """Tiny CNN batch 4 (32x32x3) at 100/50/25% of the GPU: 1000 timed forwards each."""
    m = ds.Model("tinycnn", 1010)
    fr = [1.0, 0.5, 0.25]
    r = m.knee_sweep(4, fr, warmup=50, reps=1000)
    m.destroy()
    return dict(workload="tiny CNN batch 4, 32x32x3, seed 1010", fractions=fr, n_cu=r["n_cu"],
                latency_us=r["latency_us"], p99_us=r["p99_us"], inferences_per_s=[4e6 / L for L in r["latency_us"]])


def knee_model_prediction(ds, torch, m, b, n_cu_grid, latency_us):
    """Sec. 4.3's analytical model with this library's own kernels: N_i =
    workgroups of unit i / workgroups one CU holds (dstack_kernel_shapes),
    t_p from the unit's event-timed duration on the whole GPU (the durations
    scaled so that they sum to the measured latency there), t_np = 0.  E_t is
    predicted on the sweep's CU counts and its knee compared with the
    measured one; a second prediction adds the memory term d_i / (M S) with
    the unit's algorithmic bytes and M = measured HBM bandwidth per CU."""
    from tests import gpu_util as gu
    from tests import inputs
    p = ds.Partition(1.0)
    x = gu.dev_bf16(inputs.image_batch(1021, b))
    y = gu.empty_f32(m.output_shape(b))
    for _ in range(3):
        m.infer(b, x, y, p)
    p.synchronize()
    shapes = m.kernel_shapes(b, x, y, p)
    recs = [m.profile_layers(b, x, y, p) for _ in range(3)]
    assert len(shapes) == len(recs[0]) and all(s["kind"] == r["kind"] for s, r in zip(shapes, recs[0]))
    full = p.n_cu
    t = [1000.0 * sorted(r[i]["ms"] for r in recs)[1] for i in range(len(shapes))]
    scale = latency_us[n_cu_grid.index(full)] / sum(t)
    n = [s["workgroups"] / max(1, s["blocks_per_cu"]) for s in shapes]
    tp = [scale * ti * max(1.0, min(full, ni)) / ni for ti, ni in zip(t, n)]
    et, k = ds.knee_model_eval(n, tp, n_cu_grid, 0.0)
    mb = bw_probe(torch, p) * 1e3 / full  # bytes per us per CU
    d = [s["bytes"] for s in shapes]
    tp_m = [max(0.0, scale * ti - di / (mb * full)) * max(1.0, min(full, ni)) / ni for ti, ni, di in zip(t, n, d)]
    et_m, k_m = ds.knee_model_eval(n, tp_m, n_cu_grid, 0.0, 1.0, None, d, mb)
    p.destroy()
    err = lambda e: sum(abs(a - L) / L for a, L in zip(e, latency_us)) / len(latency_us)
    return dict(units=len(shapes), n_par_max=max(n), n_par_median=sorted(n)[len(n) // 2],
                predicted_knee_slots=n_cu_grid[k] // 8, predicted_latency_us=[round(v, 1) for v in et],
                mean_abs_rel_error=err(et),
                with_memory_term=dict(predicted_knee_slots=n_cu_grid[k_m] // 8,
                                      predicted_latency_us=[round(v, 1) for v in et_m], mean_abs_rel_error=err(et_m),
                                      bw_per_cu_bytes_per_us=mb))


def config2(ds, torch, args):
    """ResNet-50 at batch 1, 8 and 32 over the 10 fractions: latency, inf/s,
    efficacy b / (L^2 * CUs) and the knee (Sec. 3.2), beside the knee the
    analytical model of Sec. 4.3 predicts from the kernels' parallelism."""
    m = ds.Model("resnet50", 1020)
    rows = []
    for b in (1, 8, 32):
        r = m.knee_sweep(b, FRACTIONS, warmup=args.sweep_warmup, reps=args.sweep_reps)
        rows.append(dict(batch=b, n_cu=r["n_cu"], latency_us=r["latency_us"], p99_us=r["p99_us"],
                         inferences_per_s=[b * 1e6 / L for L in r["latency_us"]],
                         eta=[b / (L * L * c) for L, c in zip(r["latency_us"], r["n_cu"])],
                         knee_slots=r["knee_slots"], deployed_slots=r["deployed_slots"],
                         knee_model=knee_model_prediction(ds, torch, m, b, list(r["n_cu"]),
                                                          [float(v) for v in r["latency_us"]])))
    m.destroy()
    return dict(workload="ResNet-50 v1.5, 224x224x3, seed 1020", fractions=FRACTIONS, rows=rows)


def config6(ds, args):
    """The transformer workload (Sec. 4.4): BERT-base on 10-word (20-token)
    and 20-word (40-token) sentences at batch 1 and 16 over the 10
    fractions: latency, inf/s and the knee (the paper's knees were about 30%
    and 40% of a V100 for the two lengths)."""
    rows = []
    for arch, words in (("bert", 10), ("bert_long", 20)):
        m = ds.Model(arch, 1060)
        for b in (1, 16):
            r = m.knee_sweep(b, FRACTIONS, warmup=args.sweep_warmup, reps=args.sweep_reps)
            rows.append(dict(arch=arch, words=words, tokens=m.input_shape(b)[1], batch=b, n_cu=r["n_cu"],
                             latency_us=r["latency_us"], inferences_per_s=[b * 1e6 / L for L in r["latency_us"]],
                             knee_slots=r["knee_slots"], knee_fraction=r["knee_slots"] / 32.0,
                             deployed_slots=r["deployed_slots"]))
        m.destroy()
    return dict(workload="BERT-base encoder (12 layers, 768 wide, 12 heads), 2 classes, seed 1060", rows=rows)


def config4(ds, torch, args):
    """VGG-19 batch 8 + 2-layer LSTM batch 32, closed loop on deployed-knee
    partitions (shrunk proportionally to fit), vs time-sliced full GPU."""
    from tests import inputs
    specs = [("vgg19", 1040, 8, [8]), ("lstm2", 1041, 32, [32])]
    models = [ds.Model(a, s) for a, s, _, _ in specs]
    batch = [b for _, _, b, _ in specs]
    rows = []
    for (arch, seed, b, _), m in zip(specs, models):
        r = m.knee_sweep(b, FRACTIONS, warmup=args.sweep_warmup, reps=args.sweep_reps)
        rows.append(dict(zip(r["slots"], r["latency_us"])))
    knee = [knee_at(r, b) for r, b in zip(rows, batch)]
    dep = fit_slots([min(32, k + OVERPROV) for k in knee], 32)
    lanes = [(0, 0, dep[0]), (1, dep[0], dep[1])]
    lat = [rows[i][max(s for s in rows[i] if s <= dep[i])] for i in range(2)]
    reps = [max(1, int(round(20000 / L))) for L in lat]  # each lane busy about 20 ms per step
    xs = [gu_dev(inputs.image_batch(1041, 8)), gu_dev(inputs.sequence_batch(1042, 32))]
    shapes = [m.output_shape(b) for m, b in zip(models, batch)]
    mix = Mix(ds, torch, models, batch, xs, shapes, lanes, reps)
    steps = args.steps4
    t_mix = mix.timed(steps, 2)
    t_seq = mix.timesliced(steps, 2, shapes)
    inter = mix.interference(max(2, steps // 4), 1, t_mix, steps)
    res = dict(workload="VGG-19 batch 8 + 2-layer LSTM (512->1024, T=50) batch 32, closed loop on deployed-knee "
                        "partitions; inferences = images + sequences",
               knee_slots=knee, deployed_slots=dep, reps_per_step=reps, steps=steps,
               value=mix.items_per_step * steps / t_mix, timesliced=mix.items_per_step * steps / t_seq,
               speedup_vs_timesliced=t_seq / t_mix, interference=inter,
               per_model_inf_s=[reps[i] * batch[i] * steps / t_mix for i in range(2)],
               latency_rows={specs[i][0]: rows[i] for i in range(2)})
    mix.destroy()
    for m in models:
        m.destroy()
    return res


def gu_dev(a):
    from tests import gpu_util as gu
    return gu.dev_bf16(a)


def config5(ds, torch, models4, tables4, args):
    """Four-model Poisson mix through the live launcher (plan + FOD on home
    ranges): stated rates for args.serve_seconds, then a capacity sweep."""
    from tests import inputs
    rates = [400, 800, 150, 300]
    slos = [25000, 15000, 50000, 30000]
    bmax = [16, 32, 8, 32]
    xs, ys = [], []
    for m, b in zip(models4, bmax):
        shp = m.input_shape(b)
        if len(shp) == 3:
            xs.append(gu_dev(inputs.sequence_batch(1051, shp[1], shp[0], shp[2])))
        else:
            xs.append(gu_dev(inputs.image_batch(1050, b)))
        ys.append(torch.empty(m.output_shape(b), device="cuda", dtype=torch.float32))

    def one(k, dur_us):
        tabs = [dict(slo_us=slo, max_batch=b, rate_per_s=r * k, table=t)
                for slo, b, r, t in zip(slos, bmax, rates, tables4)]
        arr = [inputs.poisson_arrivals(2026 + i, r * k, dur_us) for i, r in enumerate(rates)]
        r = ds.serve(models4, tabs, xs, ys, PERIOD_US, dur_us, arr, log_capacity=0)
        n_req = sum(len(a) for a in arr)
        viol = sum(s["violations"] for s in r["models"])
        st, plan = ds.schedule(tabs, PERIOD_US, placement="home")
        return dict(k=k, offered_req_s=n_req / (dur_us * 1e-6), served_req_s=sum(s["served"] for s in r["models"]) /
                    (dur_us * 1e-6), violations_per_s=viol / (dur_us * 1e-6), violation_frac=viol / max(1, n_req),
                    utilisation_ppm=r["utilisation_ppm"], n_jobs=r["n_jobs"],
                    plan=dict(batch=plan["batch"], deployed_slots=plan["deployed_slots"],
                              home_offset=plan["home_offset"], utilisation_ppm=plan["utilisation_ppm"],
                              status="ok" if st == ds.OK else "infeasible"),
                    per_model=[dict(arch=m.arch, **s) for m, s in zip(models4, r["models"])])
    stated = one(1, int(args.serve_seconds * 1e6))
    sweep, capacity = [], None
    for k in (2, 4, 8, 16):
        r = one(k, int(args.capacity_seconds * 1e6))
        sweep.append({kk: r[kk] for kk in ("k", "offered_req_s", "served_req_s", "violation_frac", "utilisation_ppm")})
        if r["violation_frac"] <= 0.01:
            capacity = r["offered_req_s"]
        else:
            break
    if capacity is None and stated["violation_frac"] <= 0.01:
        capacity = stated["offered_req_s"]
    return dict(workload="four-model Poisson mix (ResNet-50, MobileNetV2, VGG-19, LSTM at 400/800/150/300 req/s, "
                         "SLOs 25/15/50/30 ms, 100 ms sessions) through dstack_serve on home CU ranges",
                stated_rates=stated, capacity_sweep=sweep, capacity_req_s_at_1pct=capacity,
                capacity_seconds=args.capacity_seconds)


def comparators(ds, tables4, k=32, seconds=2.0):
    """Sec. 6.3's comparators in simulate mode on the four-model mix's measured
    timing tables at k x the stated rates (far past the 1% capacity, so that
    every policy is bound by the GPU): D-STACK
    (plan + FOD), max-throughput (least runtime first) and max-min fair
    (smallest GPU% demand first), all non-preemptive on the lowest free
    slots.  Per model: served/s and GPU busy time."""
    from tests import inputs
    rates = [400, 800, 150, 300]
    slos = [25000, 15000, 50000, 30000]
    bmax = [16, 32, 8, 32]
    names = ["resnet50", "mobilenetv2", "vgg19", "lstm2"]
    dur = int(seconds * 1e6)
    tabs = [dict(slo_us=slo, max_batch=b, rate_per_s=r * k, table=t) for slo, b, r, t in zip(slos, bmax, rates, tables4)]
    arr = [inputs.poisson_arrivals(3026 + i, r * k, dur) for i, r in enumerate(rates)]
    _, plan = ds.schedule(tabs, PERIOD_US)
    out = {}
    for pol in ("dstack", "maxthroughput", "maxmin"):
        r = ds.simulate(tabs, PERIOD_US, dur, arr, policy=pol)
        out[pol] = dict(served_per_s=[m["served"] / seconds for m in r["models"]],
                        busy_s=[m["busy_us"] * 1e-6 for m in r["models"]],
                        violation_frac=sum(m["violations"] for m in r["models"]) / max(1, sum(len(a) for a in arr)),
                        utilisation_ppm=r["utilisation_ppm"])
        out[pol]["total_per_s"] = sum(out[pol]["served_per_s"])
        b = out[pol]["busy_s"]
        out[pol]["busy_min_over_max"] = min(b) / max(b) if max(b) > 0 else None
    fast = min(range(4), key=lambda i: plan["latency_us"][i])
    d, mt = out["dstack"], out["maxthroughput"]
    return dict(models=names, rate_scale=k, seconds=seconds, lowest_runtime_model=names[fast], policies=out,
                dstack_over_maxthroughput_total=d["total_per_s"] / mt["total_per_s"],
                dstack_over_maxthroughput_lowest_runtime_model=d["served_per_s"][fast] / max(1e-9, mt["served_per_s"][fast]),
                dstack_over_maxmin_total=d["total_per_s"] / out["maxmin"]["total_per_s"])


def kernel_knee_table(ds, m, b, x, y):
    """Per kernel of one forward (the timed units of the layer profile): its
    duration on each of the sweep's shares and its own knee (argmax of
    1/(d^2 s), ties to fewer slots) -- the per-kernel GPU% the ideal
    schedule of Sec. 6.2 assumes known."""
    durs = []
    for f in FRACTIONS:
        p = ds.Partition(f)
        for _ in range(2):
            m.infer(b, x, y, p)
        p.synchronize()
        runs = [m.profile_layers(b, x, y, p) for _ in range(3)]
        durs.append((p.n_cu // 8, [sorted(r[i]["ms"] for r in runs)[1] * 1000.0 for i in range(len(runs[0]))]))
        p.destroy()
    slots, dur = [], []
    for k in range(len(durs[0][1])):
        best = min(durs, key=lambda sd: (sd[1][k] ** 2 * sd[0], sd[0]))
        slots.append(best[0])
        dur.append(max(1, int(round(best[1][k]))))
    # the model-level table from the same measurements: the sum of its kernels on each share
    table = {sl: max(1, int(round(sum(d)))) for sl, d in durs}
    return slots, dur, table


def ideal_vs_dstack(ds, models, tables, batch, xs, ys, seconds=0.2, slot_us=1):
    """The headline pair under the ideal schedule of Sec. 6.2 (slotted, kernel
    granularity, preemptive, every kernel at its own knee) and under D-STACK
    in simulate mode (plan + FOD, model granularity, non-preemptive) with the
    same batches, requests always waiting.  Both take their times from the
    same per-kernel measurements (D-STACK's latency on s slots = the sum of
    the kernels' durations on s slots), so the ratio compares the schedules
    only.  Slot 1 us: these kernels last 5-50 us, where the paper's 100 us
    slots fitted its millisecond ones."""
    ideal_models, tabs = [], []
    for (arch, seed, slo, b, _), m, x, y in zip(MODELS, models, xs, ys):
        sl, du, table = kernel_knee_table(ds, m, b, x, y)
        ideal_models.append(dict(slots=sl, dur=du, batch=b, slo_us=slo))
        tabs.append(dict(slo_us=slo, max_batch=b, table={b: table}))
    hor = int(seconds * 1e6)
    idl = ds.simulate_ideal(ideal_models, hor, slot_us)
    dense = [list(range(0, hor, 20)) for _ in MODELS]
    sim = ds.simulate(tabs, PERIOD_US, hor, dense)
    d_items = [mm["served"] for mm in sim["models"]]
    return dict(slot_us=slot_us, seconds=seconds, kernel_sum_tables=[t["table"][b] for t, b in zip(tabs, batch)],
                kernels=[len(im["dur"]) for im in ideal_models],
                kernel_knee_slots_median=[sorted(im["slots"])[len(im["slots"]) // 2] for im in ideal_models],
                forward_us_at_kernel_knees=[sum(im["dur"]) for im in ideal_models],
                ideal_items_per_s=[v / seconds for v in idl["items"]], ideal_utilisation_ppm=idl["utilisation_ppm"],
                dstack_items_per_s=[v / seconds for v in d_items], dstack_utilisation_ppm=sim["utilisation_ppm"],
                dstack_over_ideal=sum(d_items) / max(1, sum(idl["items"])))


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: one GPU only -- the D-STACK hot path shards by placing whole models on GPUs and this "
              "build measures one GPU's share; run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2304_13541_amd as ds
    from tests import gpu_util as gu
    from tests import inputs

    torch.cuda.init()
    models = [ds.Model(a, s) for a, s, *_ in MODELS]
    n_models = len(MODELS)

    # ---- setup: timing tables, knees, partitions ----
    sweep_s = None
    if args.table:
        with open(args.table) as f:
            tables = json.load(f)
        for t in tables:
            t["table"] = {int(b): {int(s): int(L) for s, L in row.items()} for b, row in t["table"].items()}
    else:
        t0 = time.perf_counter()
        tables = sweep_tables(models, args)
        sweep_s = time.perf_counter() - t0
    if args.save_table:
        with open(args.save_table, "w") as f:
            json.dump(tables, f)

    batch = [b for _, _, _, b, _ in MODELS]
    knee = [knee_at(t["table"][b], b) for t, b in zip(tables, batch)]
    dep = fit_slots([min(ds.TOTAL_SLOTS, k + OVERPROV) for k in knee], ds.TOTAL_SLOTS)
    reps = [math.ceil(PERIOD_US / slo) for _, _, slo, _, _ in MODELS]
    lanes = pack_lanes(dep, ds.TOTAL_SLOTS, MAX_PARTITIONS)

    # the SLO-constrained choice over the whole table (reported; Sec. 5.1)
    sched_in = [dict(slo_us=slo, max_batch=b, rate_per_s=0, table=t["table"])
                for (arch, seed, slo, b, _), t in zip(MODELS, tables)]
    sched_st, plan = ds.schedule(sched_in, PERIOD_US)

    xs = [gu.dev_bf16(inputs.image_batch(seed + 1, b)) for (a, seed, *_), b in zip(MODELS, batch)]
    shapes = [(b, 1000) for b in batch]
    mix = Mix(ds, torch, models, batch, xs, shapes, lanes, reps)
    t_mix = mix.timed(args.steps, args.warmup)
    value = mix.items_per_step * args.steps / t_mix
    t_seq = mix.timesliced(args.steps, args.warmup, shapes)
    seq_value = mix.items_per_step * args.steps / t_seq
    inter = mix.interference(max(5, args.steps // 4), args.warmup, t_mix, args.steps)
    # the same models concurrently on unmasked streams (each stream may use every CU): the
    # MPS-default analogue, a second, non-target baseline
    full_lanes = [(mi, 0, ds.TOTAL_SLOTS) for mi, _, _ in lanes]
    umix = Mix(ds, torch, models, batch, xs, shapes, full_lanes, reps)
    t_umix = umix.timed(args.steps, args.warmup)
    umix.destroy()
    unmasked_value = mix.items_per_step * args.steps / t_umix
    # HBM bandwidth each deployed partition (and the whole GPU) can draw: BW(n) of the rooflines
    bw_lane = [bw_probe(torch, p) for p in mix.parts]
    pfull = ds.Partition(1.0)
    bw_full = bw_probe(torch, pfull)
    pfull.destroy()

    # ---- per-kernel timing at the deployed partitions (HIP events on each partition's stream) ----
    per_model = []
    conv_fl, conv_ms, conv_n, conv_by = 0.0, 0.0, 0, 0.0
    for i, m in enumerate(models):
        li = next(k for k, l in enumerate(lanes) if l[0] == i)
        recs, by_kind = layer_stats(ds, m, batch[i], xs[i], mix.ys[li], mix.parts[li])
        mf = [r for r in recs if r["kind"] == 0]
        fl = sum(r["flops"] for r in mf)
        ms = sum(r["ms"] for r in mf)
        conv_fl += fl
        conv_ms += ms
        conv_n += len(mf)
        conv_by += sum(r["bytes"] for r in mf)
        n_cu = mix.parts[li].n_cu
        tf = fl / (ms * 1e-3) / 1e12 if ms > 0 else None
        per_model.append(dict(
            arch=MODELS[i][0], batch=batch[i], knee_slots=knee[i], slots=dep[i], n_cu=n_cu,
            partitions=mix.lane_count[i], jobs_per_step=reps[i],
            latency_us_at_knee=tables[i]["table"][batch[i]][knee[i]],
            conv_mfma_tflops=tf, conv_frac_of_partition_peak=tf / (PEAK_BF16_TFLOPS * n_cu / 256) if tf else None,
            slo_optimal=dict(batch=plan["batch"][i], knee_slots=plan["knee_slots"][i],
                             deployed_slots=plan["deployed_slots"][i], latency_us=plan["latency_us"][i],
                             feasible=plan["feasible"][i]),
            kernels=by_kind,
            inferences_per_s_in_mix=mix.lane_count[i] * reps[i] * batch[i] * args.steps / t_mix,
            roofline=model_roofline(ds, recs, n_cu, bw_lane[li],
                                    next(x["alone_us"] for x in inter if x["lane"] == li))))
    mix.destroy()
    # mix-level: same-work makespan ratio (one step's jobs run one by one on the whole GPU, from the
    # timing table, over the measured step), FLOP-weighted work rate, CU-weighted roofline busy time
    full_us = sum(mix.lane_count[i] * reps[i] * tables[i]["table"][batch[i]][ds.TOTAL_SLOTS] for i in range(n_models))
    step_us = 1e6 * t_mix / args.steps
    flops_item = [m.info.flops_per_item for m in models]
    mix_metrics = dict(
        same_work_makespan_ratio=full_us / step_us,
        flop_weighted_tflops=sum(p["inferences_per_s_in_mix"] * f for p, f in zip(per_model, flops_item)) / 1e12,
        mix_roofline_frac=sum(mix.lane_count[i] * reps[i] * per_model[i]["roofline"]["t_roof_us"] *
                              per_model[i]["n_cu"] / 256 for i in range(n_models)) / step_us,
        unmasked_concurrent_inferences_per_s=unmasked_value,
        hbm_gbs_full_gpu=bw_full)
    avg_ms = conv_ms / max(conv_n, 1)
    achieved = (conv_fl / max(conv_n, 1)) / (avg_ms * 1e-3) / 1e12
    knee_cu = sum(p["n_cu"] * p["kernels"]["mfma"]["ms"] for p in per_model) / max(
        sum(p["kernels"]["mfma"]["ms"] for p in per_model), 1e-9)

    # ---- GPU% reconfiguration (Sec. 3.5, 3.6): knee search from 30% vs the sweep, cost of a change ----
    reconf = []
    for i, m in enumerate(models if not args.headline_only else []):
        ks = m.knee_search(batch[i], FRACTIONS, 10, args.sweep_warmup, args.sweep_reps)
        sw = m.switch_probe(batch[i], 10, dep[i], reps=10)
        reconf.append(dict(arch=MODELS[i][0], batch=batch[i], search_knee_slots=ks["knee_slots"],
                           sweep_knee_slots=knee[i], search_probes=ks["probes"], search_seconds=ks["seconds"],
                           switch_from_slots=10, switch_to_slots=dep[i], **sw))

    # ---- the other workloads: VGG-19 + LSTM pair, four-model Poisson mix through the live launcher ----
    c1 = c2 = c4 = c5 = c6 = cmp = ideal = None
    if not args.headline_only:
        c1 = config1(ds)
        c2 = config2(ds, torch, args)
        c6 = config6(ds, args)
        c4 = config4(ds, torch, args)
        extra = [("vgg19", 1052, [1, 2, 4, 8]), ("lstm2", 1053, [1, 2, 4, 8, 16, 32])]
        m4 = [ds.Model(a, s) for a, s, _ in extra]
        t4 = [t["table"] for t in tables]
        for (a, s, bs), m in zip(extra, m4):
            tab = {}
            for b in bs:
                r = m.knee_sweep(b, FRACTIONS, warmup=args.sweep_warmup, reps=args.sweep_reps)
                tab[b] = dict(zip(r["slots"], r["latency_us"]))
            t4.append(tab)
        c5 = config5(ds, torch, models + m4, t4, args)
        for m in m4:
            m.destroy()
        cmp = comparators(ds, t4)
        ideal = ideal_vs_dstack(ds, models, tables, batch, xs, [gu.empty_f32(m.output_shape(b))
                                                                for m, b in zip(models, batch)])

    # calibration copy for the HBM byte counters (a plain 256 MiB device copy)
    a = torch.empty(64 * 1024 * 1024, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()

    cpu = None if args.no_cpu_baseline else cpu_baseline(args.cpu_seconds, sched_in)

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "inferences/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1000.0 * t_mix / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "two-model mix: ResNet-50 v1.5 batch 16 (SLO 25 ms) + MobileNetV2 1.0 batch 32 "
                        "(SLO 15 ms), 224x224x3, each on CU-masked partitions of its knee + 2 slots packed "
                        "over the 32 slots; one step = ceil(100 ms / SLO) batches per partition, closed loop",
            "batch": batch, "knee_slots": knee, "deployed_slots": dep,
            "partitions": [(MODELS[mi][0], o, s) for mi, o, s in lanes],
            "jobs_per_step": reps, "items_per_step": mix.items_per_step, "seeds": [s for _, s, *_ in MODELS],
            "parallelism": "spatial (CU masks), 1 GPU",
        },
        "conv_mfma_tflops_at_knee": conv_fl / (conv_ms * 1e-3) / 1e12,
        "conv_knee_cu": knee_cu,
        "timesliced_inferences_per_s": seq_value,
        "speedup_vs_timesliced": value / seq_value,
        "interference": inter,
        "mix": mix_metrics,
        "roofline": {
            "bound": "mfma", "kernel": "conv_igemm (all launches of both models at their partitions)",
            "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
            "n_cu": knee_cu, "peak_partition": PEAK_BF16_TFLOPS * knee_cu / 256,
            "frac_partition": achieved / (PEAK_BF16_TFLOPS * knee_cu / 256),
            "launches": conv_n, "avg_launch_us": 1000.0 * avg_ms, "flops_per_launch": conv_fl / max(conv_n, 1),
            "algorithmic_bytes_per_launch": conv_by / max(conv_n, 1),
            "traffic": measured_traffic(),
        },
        "cpu_baseline": cpu,
        "schedule_status": "ok" if sched_st == ds.OK else "infeasible",
        "per_model": per_model,
        "reconfiguration": reconf,
        "config1": c1,
        "config2": c2,
        "config4": c4,
        "config5": c5,
        "config6": c6,
        "comparators": cmp,
        "ideal_vs_dstack": ideal,
        "timing_tables": {t["arch"]: {str(b): row for b, row in t["table"].items()} for t in tables},
        "sweep_seconds": sweep_s,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
