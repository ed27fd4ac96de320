"""Benchmark: multi-DNN spatial multiplexing on one MI355X.

Workload (one GPU): ResNet-50 (batch <= 16, SLO 25 ms) and MobileNetV2
(batch <= 32, SLO 15 ms), synthetic N(0,1) 224x224x3 bf16 images standing in
for ImageNet, random-weight bf16 models.

Setup (untimed): load both models, sweep each over batches {1,2,4,8,16[,32]}
x CU fractions 10%..100% (knee sweep: median latency per point), choose
(batch, slots) per model under its SLO and build the 100 ms session plan
(dstack_schedule).  Each model gets a CU-masked partition of its deployed
slots, disjoint from the other's.

One step = one session's job multiset: model i runs r_i = ceil(100 ms / SLO_i)
batches of its chosen size on its own partition, both partitions
concurrently.  Value = aggregate inferences/s over K steps.  The same
multiset run one batch at a time on the whole GPU is the time-sliced
baseline.  Per-kernel HIP-event timing on each partition's stream gives the
conv MFMA TFLOP/s at the knee and the roofline fraction of the dominant
kernel (the implicit-GEMM convolution).
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "aggregate inferences/s (multi-DNN, one GPU) + conv MFMA TFLOP/s at knee CU%"
PEAK_BF16_TFLOPS = 2516.6   # dense bf16 MFMA, 256 CUs at 2.4 GHz
PEAK_HBM_GBS = 8000.0
FRACTIONS = [0.1 * i for i in range(1, 11)]
PERIOD_US = 100000


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--sweep-warmup", type=int, default=3)
    p.add_argument("--sweep-reps", type=int, default=20)
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the oracle CPU baseline")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--table", default=None, help="load a timing table JSON instead of sweeping")
    p.add_argument("--save-table", default=None)
    return p.parse_args()


MODELS = [
    # arch, seed, SLO us, max batch, batches swept
    ("resnet50", 1030, 25000, 16, [1, 2, 4, 8, 16]),
    ("mobilenetv2", 1031, 15000, 32, [1, 2, 4, 8, 16, 32]),
]


def sweep_tables(ds, models, args):
    tables = []
    for (arch, seed, slo, bmax, batches), m in zip(MODELS, models):
        tab, knees = {}, {}
        for b in batches:
            r = m.knee_sweep(b, FRACTIONS, warmup=args.sweep_warmup, reps=args.sweep_reps)
            tab[b] = dict(zip(r["slots"], r["latency_us"]))
            knees[b] = r["knee_slots"]
        tables.append(dict(arch=arch, table=tab, knee_slots_per_batch=knees))
    return tables


def cpu_baseline(budget_s):
    """The oracle, as it stands, on the host cores: sampled items of the same
    workload (independent batch items), parity mode."""
    import oracle
    from tests import inputs
    done, t0 = 0, time.perf_counter()
    models = {a: oracle.Model(a, s) for a, s, *_ in MODELS}
    i = 0
    while True:
        arch, seed = MODELS[i % 2][0], MODELS[i % 2][1]
        x = inputs.image_batch(seed + 1 + i, 1)
        models[arch].forward(x, parity=True)
        done += 1
        i += 1
        el = time.perf_counter() - t0
        if el >= budget_s and i % 2 == 0:
            break
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return dict(value=done / el, unit="inferences/s", cores=threads, kind="oracle",
                sample="%d single images alternating ResNet-50 / MobileNetV2 (fp64, parity mode), %.1f s" % (done, el))


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU only (the D-STACK hot path shards by placing whole models "
              "per GPU; no multi-GPU mode is implemented) -- use --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2304_13541_amd as ds
    from tests import gpu_util as gu
    from tests import inputs

    torch.cuda.init()
    models = [ds.Model(a, s) for a, s, *_ in MODELS]

    # ---- setup: timing tables, schedule, partitions ----
    if args.table:
        with open(args.table) as f:
            tables = json.load(f)
        for t in tables:
            t["table"] = {int(b): {int(s): int(L) for s, L in row.items()} for b, row in t["table"].items()}
    else:
        t0 = time.perf_counter()
        tables = sweep_tables(ds, models, args)
        sweep_s = time.perf_counter() - t0
    if args.save_table:
        with open(args.save_table, "w") as f:
            json.dump(tables, f)
    sched_in = [dict(slo_us=slo, max_batch=bmax, rate_per_s=0, table=t["table"])
                for (arch, seed, slo, bmax, _), t in zip(MODELS, tables)]
    st, plan = ds.schedule(sched_in, PERIOD_US)
    batch = plan["batch"]
    slots = list(plan["deployed_slots"])
    if sum(slots) > ds.TOTAL_SLOTS:  # shrink proportionally, larger first, to keep the partitions disjoint
        tot = sum(slots)
        slots = [max(1, math.floor(s * ds.TOTAL_SLOTS / tot)) for s in slots]
    parts, off = [], 0
    for s in slots:
        parts.append(ds.Partition(slot_offset=off, n_slots=s))
        off += s
    reps = [sum(1 for j in plan["jobs"] if j["model"] == i) for i in range(len(MODELS))]

    xs = [gu.dev_bf16(inputs.image_batch(seed + 1, b)) for (a, seed, *_), b in zip(MODELS, batch)]
    ys = [gu.empty_f32((b, 1000)) for b in batch]

    def run_mix(k):
        for _ in range(k):
            for i, m in enumerate(models):
                for _r in range(reps[i]):
                    m.infer(batch[i], xs[i], ys[i], parts[i])

    def sync_all():
        for p in parts:
            p.synchronize()
        torch.cuda.synchronize()

    # ---- warmup + timed region ----
    run_mix(args.warmup)
    sync_all()
    t0 = time.perf_counter()
    run_mix(args.steps)
    sync_all()
    t_mix = time.perf_counter() - t0
    items_per_step = sum(r * b for r, b in zip(reps, batch))
    value = items_per_step * args.steps / t_mix

    # ---- time-sliced baseline: same multiset, one batch at a time, whole GPU ----
    full = ds.Partition(1.0)
    def run_seq(k):
        for _ in range(k):
            for i, m in enumerate(models):
                for _r in range(reps[i]):
                    m.infer(batch[i], xs[i], ys[i], full)
    run_seq(args.warmup)
    full.synchronize()
    t0 = time.perf_counter()
    run_seq(args.steps)
    full.synchronize()
    t_seq = time.perf_counter() - t0
    seq_value = items_per_step * args.steps / t_seq

    # ---- per-kernel timing at the deployed partitions (HIP events on each partition's stream) ----
    per_model = []
    conv_fl, conv_ms, conv_n, conv_by = 0.0, 0.0, 0, 0.0
    for i, m in enumerate(models):
        recs = m.profile_layers(batch[i], xs[i], ys[i], parts[i])
        for _ in range(2):  # average over three profiled forwards
            recs2 = m.profile_layers(batch[i], xs[i], ys[i], parts[i])
            for r, r2 in zip(recs, recs2):
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
            k = ds.KIND_NAMES[r["kind"]]
            d = by_kind.setdefault(k, dict(n=0, ms=0.0, flops=0.0, bytes=0.0))
            d["n"] += 1
            d["ms"] += r["ms"]
            d["flops"] += r["flops"]
            d["bytes"] += r["bytes"]
        n_cu = parts[i].n_cu
        per_model.append(dict(
            arch=MODELS[i][0], batch=batch[i], slots=slots[i], n_cu=n_cu, knee_slots=plan["knee_slots"][i],
            jobs_per_period=reps[i], planned_latency_us=plan["latency_us"][i],
            conv_mfma_tflops=fl / (ms * 1e-3) / 1e12 if ms > 0 else None,
            conv_frac_of_partition_peak=(fl / (ms * 1e-3) / 1e12) / (PEAK_BF16_TFLOPS * n_cu / 256) if ms > 0 else None,
            kernels=by_kind))
    avg_ms = conv_ms / max(conv_n, 1)
    achieved = (conv_fl / max(conv_n, 1)) / (avg_ms * 1e-3) / 1e12
    knee_cu = sum(p["n_cu"] * p["kernels"]["mfma"]["ms"] for p in per_model) / max(
        sum(p["kernels"]["mfma"]["ms"] for p in per_model), 1e-9)

    # calibration copy for HBM byte counters (a plain 256 MiB device copy)
    a = torch.empty(64 * 1024 * 1024, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args.cpu_seconds)

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
            "workload": "two-model mix on disjoint CU-masked partitions at their knees: ResNet-50 v1.5 "
                        "(224x224x3, batch <= 16, SLO 25 ms) + MobileNetV2 1.0 (224x224x3, batch <= 32, "
                        "SLO 15 ms); one step = one 100 ms session's job multiset",
            "batch": batch, "deployed_slots": slots, "n_cu": [p.n_cu for p in parts], "jobs_per_step": reps,
            "items_per_step": items_per_step, "seeds": [s for _, s, *_ in MODELS],
            "schedule_status": "ok" if st == ds.OK else "infeasible",
            "parallelism": "spatial (CU masks), 1 GPU",
        },
        "conv_mfma_tflops_at_knee": conv_fl / (conv_ms * 1e-3) / 1e12,
        "conv_knee_cu": knee_cu,
        "timesliced_inferences_per_s": seq_value,
        "speedup_vs_timesliced": value / seq_value,
        "roofline": {
            "bound": "mfma", "kernel": "conv_igemm (all launches at the deployed partitions)",
            "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
            "n_cu": knee_cu, "peak_partition": PEAK_BF16_TFLOPS * knee_cu / 256,
            "frac_partition": achieved / (PEAK_BF16_TFLOPS * knee_cu / 256),
            "launches": conv_n, "avg_launch_us": 1000.0 * avg_ms, "flops_per_launch": conv_fl / max(conv_n, 1),
            "algorithmic_bytes_per_launch": conv_by / max(conv_n, 1),
            "traffic": None,
        },
        "cpu_baseline": cpu,
        "per_model": per_model,
        "timing_tables": {t["arch"]: {str(b): row for b, row in t["table"].items()} for t in tables},
    }
    if not args.table:
        out["sweep_seconds"] = sweep_s
    print(json.dumps(out))


if __name__ == "__main__":
    main()
