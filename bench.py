"""Benchmark: multi-DNN spatial multiplexing on one MI355X.

Workload (one GPU): ResNet-50 v1.5 at batch 16 (SLO 25 ms) and MobileNetV2
1.0 at batch 32 (SLO 15 ms), synthetic N(0,1) 224x224x3 bf16 images standing
in for ImageNet, random-weight bf16 models.

Setup (untimed): load both models and sweep each over batches {1,2,4,8,16[,32]}
x CU fractions 10%..100% (knee sweep: median latency of 20 timed forwards per
point).  At the workload's batch each model's knee is the efficacy optimum
b/(L^2 s) over the swept slot counts; it is deployed with 2 slots of
over-provisioning.  The CU-masked partitions (disjoint slot ranges) are packed
over the 32 slots round-robin over the models -- instances of one model share
its weights -- up to 4 partitions (more concurrently active masked queues are
avoided on this part).  The SLO-constrained (batch, slots) choice of
dstack_schedule over the whole table is reported alongside.

One step = one 100 ms session: each partition runs r = ceil(100 ms / SLO)
batches of its model back to back, all partitions concurrently.  Value =
aggregate inferences/s over K steps.  The time-sliced full-GPU baseline runs
the same per-model batch counts one batch at a time on an unmasked
partition.  Per-kernel HIP-event timing on each partition's stream gives the
conv MFMA TFLOP/s at the knee and the roofline fraction of the dominant
kernel (the implicit-GEMM convolution).
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
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--sweep-warmup", type=int, default=5)
    p.add_argument("--sweep-reps", type=int, default=20)
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the oracle CPU baseline")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--table", default=None, help="load a timing table JSON instead of sweeping")
    p.add_argument("--save-table", default=None)
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


def cpu_baseline(budget_s):
    """The oracle, as it stands, on the host cores: sampled items of the same
    workload (batch items are independent), parity mode."""
    import oracle
    from tests import inputs
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
                       "%.1f s" % (done, el))


def knee_at(row, b):
    """Efficacy optimum b / (L^2 s) over a {slots: L} row, ties to fewer slots."""
    best = None
    for s in sorted(row):
        L = row[s]
        if best is None or b * row[best] ** 2 * best > b * L * L * s:
            best = s
    return best


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
    dep = [min(ds.TOTAL_SLOTS, k + OVERPROV) for k in knee]
    reps = [math.ceil(PERIOD_US / slo) for _, _, slo, _, _ in MODELS]
    lanes, off = [], 0  # (model, slot offset, slots)
    if sum(dep) > ds.TOTAL_SLOTS:  # shrink proportionally: one partition per model
        tot = sum(dep)
        dep = [max(1, math.floor(s * ds.TOTAL_SLOTS / tot)) for s in dep]
    i, misses = 0, 0
    while misses < n_models and len(lanes) < MAX_PARTITIONS:
        mi = i % n_models
        if off + dep[mi] <= ds.TOTAL_SLOTS:
            lanes.append((mi, off, dep[mi]))
            off += dep[mi]
            misses = 0
        else:
            misses += 1
        i += 1
    parts = [ds.Partition(slot_offset=o, n_slots=s) for _, o, s in lanes]
    lane_count = [sum(1 for l in lanes if l[0] == mi) for mi in range(n_models)]

    # the SLO-constrained choice over the whole table (reported; Sec. 5.1)
    sched_in = [dict(slo_us=slo, max_batch=b, rate_per_s=0, table=t["table"])
                for (arch, seed, slo, b, _), t in zip(MODELS, tables)]
    sched_st, plan = ds.schedule(sched_in, PERIOD_US)

    xs = [gu.dev_bf16(inputs.image_batch(seed + 1, b)) for (a, seed, *_), b in zip(MODELS, batch)]
    ys = [gu.empty_f32((batch[mi], 1000)) for mi, _, _ in lanes]

    def run_mix(k):
        for _ in range(k):
            for li, (mi, _, _) in enumerate(lanes):
                for _r in range(reps[mi]):
                    models[mi].infer(batch[mi], xs[mi], ys[li], parts[li])

    def sync_all():
        for p in parts:
            p.synchronize()
        torch.cuda.synchronize()

    run_mix(args.warmup)
    sync_all()
    t0 = time.perf_counter()
    run_mix(args.steps)
    sync_all()
    t_mix = time.perf_counter() - t0
    items_per_step = sum(reps[mi] * batch[mi] for mi, _, _ in lanes)
    value = items_per_step * args.steps / t_mix

    # ---- time-sliced baseline: same batches and per-model counts, one at a time, whole GPU ----
    full = ds.Partition(1.0)
    yf = [gu.empty_f32((b, 1000)) for b in batch]

    def run_seq(k):
        for _ in range(k):
            for mi, m in enumerate(models):
                for _r in range(lane_count[mi] * reps[mi]):
                    m.infer(batch[mi], xs[mi], yf[mi], full)
    run_seq(args.warmup)
    full.synchronize()
    t0 = time.perf_counter()
    run_seq(args.steps)
    full.synchronize()
    t_seq = time.perf_counter() - t0
    seq_value = items_per_step * args.steps / t_seq
    full.destroy()

    # ---- per-kernel timing at the deployed partitions (HIP events on each partition's stream) ----
    per_model = []
    conv_fl, conv_ms, conv_n, conv_by = 0.0, 0.0, 0, 0.0
    for i, m in enumerate(models):
        li = next(k for k, l in enumerate(lanes) if l[0] == i)
        recs = m.profile_layers(batch[i], xs[i], ys[li], parts[li])
        for _ in range(2):  # average of three profiled forwards
            for r, r2 in zip(recs, m.profile_layers(batch[i], xs[i], ys[li], parts[li])):
                r["ms"] += r2["ms"]
        for r in recs:
            r["ms"] /= 3.0
        mf = [r for r in recs if r["kind"] == 0]
        fl = sum(r["flops"] for r in mf)
        ms = sum(r["ms"] for r in mf)
        conv_fl += fl
        conv_ms += ms
        conv_n += len(mf)
        conv_by += sum(r["bytes"] for r in mf)
        by_kind = {}
        for r in recs:
            d = by_kind.setdefault(ds.KIND_NAMES[r["kind"]], dict(n=0, ms=0.0, flops=0.0, bytes=0.0))
            d["n"] += 1
            d["ms"] += r["ms"]
            d["flops"] += r["flops"]
            d["bytes"] += r["bytes"]
        n_cu = parts[li].n_cu
        tf = fl / (ms * 1e-3) / 1e12 if ms > 0 else None
        per_model.append(dict(
            arch=MODELS[i][0], batch=batch[i], knee_slots=knee[i], slots=dep[i], n_cu=n_cu,
            partitions=lane_count[i], jobs_per_step=reps[i], latency_us_at_knee=tables[i]["table"][batch[i]][knee[i]],
            conv_mfma_tflops=tf, conv_frac_of_partition_peak=tf / (PEAK_BF16_TFLOPS * n_cu / 256) if tf else None,
            slo_optimal=dict(batch=plan["batch"][i], knee_slots=plan["knee_slots"][i],
                             deployed_slots=plan["deployed_slots"][i], latency_us=plan["latency_us"][i],
                             feasible=plan["feasible"][i]),
            kernels=by_kind))
    avg_ms = conv_ms / max(conv_n, 1)
    achieved = (conv_fl / max(conv_n, 1)) / (avg_ms * 1e-3) / 1e12
    knee_cu = sum(p["n_cu"] * p["kernels"]["mfma"]["ms"] for p in per_model) / max(
        sum(p["kernels"]["mfma"]["ms"] for p in per_model), 1e-9)

    # calibration copy for the HBM byte counters (a plain 256 MiB device copy)
    a = torch.empty(64 * 1024 * 1024, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()

    cpu = None if args.no_cpu_baseline else cpu_baseline(args.cpu_seconds)

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
                        "over the 32 slots; one step = one 100 ms session per partition",
            "batch": batch, "knee_slots": knee, "deployed_slots": dep,
            "partitions": [(MODELS[mi][0], o, s) for mi, o, s in lanes],
            "jobs_per_step": reps, "items_per_step": items_per_step, "seeds": [s for _, s, *_ in MODELS],
            "parallelism": "spatial (CU masks), 1 GPU",
        },
        "conv_mfma_tflops_at_knee": conv_fl / (conv_ms * 1e-3) / 1e12,
        "conv_knee_cu": knee_cu,
        "timesliced_inferences_per_s": seq_value,
        "speedup_vs_timesliced": value / seq_value,
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
        "timing_tables": {t["arch"]: {str(b): row for b, row in t["table"].items()} for t in tables},
        "sweep_seconds": sweep_s,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
