"""Per-layer kernel times of one model on one CU-masked partition.

    python -m paper_2304_13541_amd.layer_profile --arch resnet50 --batch 16 --fraction 0.4 [--compare-blas]

Times every kernel of a forward with HIP events on the partition's stream
(dstack_profile_layers, mean of --reps forwards) and prints, per MFMA layer,
its GEMM shape (pixels, output channels, depth), time and TFLOP/s.  With
--compare-blas it also times torch.matmul (hipBLASLt) on bf16 matrices of the
same GEMM shape on the same masked stream, as a vendor-library reference.
Inputs are synthetic N(0,1) values.

    python -m paper_2304_13541_amd.layer_profile --sweep
    python -m paper_2304_13541_amd.layer_profile --summarize PASS_DIR [PASS_DIR ...] [--trace TRACE_DIR]
    python -m paper_2304_13541_amd.layer_profile --bench-kernels TRACE_DIR BENCH_LOG [UNPROFILED_BENCH_LOG]
    python -m paper_2304_13541_amd.layer_profile --bench-traffic FETCH_DIR WRITE_DIR BENCH_LOG

--sweep runs the measured workloads (ResNet-50 b16, MobileNetV2 b32, VGG-19
b8, the LSTM b32) on partitions of 25%, 50% and 100% of the CUs, or with
--cases ARCH:BATCH:SLOTS ... the given models on partitions of that many
slots (from slot 0), one eager
forward each (run it with DSTACK_GRAPH=0 under rocprofv3), every segment
preceded by a marker dispatch (the CU-id probe with 1000 + segment
workgroups), and ends with a 256 MiB device copy that calibrates the HBM
byte counters.  --summarize reads the rocprofv3 counter CSVs of such runs
(counters SQ_VALU_MFMA_BUSY_CYCLES, SQ_INSTS_VALU_MFMA_MOPS_BF16,
GRBM_GUI_ACTIVE, FETCH_SIZE, WRITE_SIZE in any passes), splits them at the
markers and prints per (partition, model, kernel class): dispatches, time,
MFMA rate from the MFMA op counter against the partition's peak, MFMA busy
cycles per CU-cycle, and calibrated HBM bytes and GB/s (give the same
--cases as to the sweep).  When the passes hold the SQ wave-state counters
(SQ_WAVE_CYCLES, SQ_WAIT_ANY, SQ_WAIT_INST_ANY, SQ_ACTIVE_INST_ANY / _VMEM /
_LDS / _VALU / _SCA, SQ_VALU_MFMA_BUSY_CYCLES) it also prints where the
waves' time goes: the share of wave-cycles waiting on dependencies (memory,
barriers), waiting to issue, and issuing each instruction kind.

--bench-kernels and --bench-traffic read rocprofv3 runs of bench.py (kernel
trace; FETCH_SIZE and WRITE_SIZE passes), whose roofline forwards are marked
the same way, and summarise its dominant kernel, the implicit-GEMM
convolution: mean dispatch duration against the bench's HIP-event figure,
and calibrated HBM bytes per launch (the figure bench.py reports as its
roofline traffic while the kernel source and the operating point match).
"""
import argparse
import collections
import csv
import glob
import hashlib
import json
import os

import torch

import paper_2304_13541_amd as ds

SWEEP_MODELS = [("resnet50", 16), ("mobilenetv2", 32), ("vgg19", 8), ("lstm2", 32)]
SWEEP_FRACTIONS = [0.25, 0.5, 1.0]
MARKER_BASE = 1000
END_MARKER = 999
CALIBRATION_BYTES = 256 << 20
TRACE_DIR = []


CASES = []  # (arch, batch, slots) from --cases; empty: SWEEP_MODELS x SWEEP_FRACTIONS


def sweep_segments():
    """(arch, batch, CUs) of each sweep segment, in order."""
    if CASES:
        return [(a, b, 8 * sl) for a, b, sl in CASES]
    return [(a, b, 8 * ds.fraction_to_slots(f)) for f in SWEEP_FRACTIONS for a, b in SWEEP_MODELS]


def sweep():
    seg = 0
    runs = {}
    for arch, b, _ in sweep_segments():
        if (arch, b) in runs:
            continue
        m = ds.Model(arch, 1)
        g = torch.Generator(device="cuda").manual_seed(1)
        x = torch.randn(m.input_shape(b), device="cuda", generator=g).to(torch.bfloat16)
        runs[(arch, b)] = (arch, b, m, x, torch.empty(m.output_shape(b), device="cuda", dtype=torch.float32))
    # one partition per case, or per fraction with every model on it
    groups = [(sl, [runs[(a, b)]]) for a, b, sl in CASES] if CASES else \
        [(ds.fraction_to_slots(f), [runs[(a, b)] for a, b in SWEEP_MODELS]) for f in SWEEP_FRACTIONS]
    for slots, group in groups:
        p = ds.Partition(slot_offset=0, n_slots=slots)
        for arch, b, m, x, y in group:
            for _ in range(2):
                m.infer(b, x, y, p)
            p.synchronize()
            torch.cuda.synchronize()
            p.probe_cu_ids(MARKER_BASE + seg)
            recs = m.profile_layers(b, x, y, p)
            p.probe_cu_ids(END_MARKER)
            print("segment %d: %s b%d on %d CUs, %d timed units, %.1f us" %
                  (seg, arch, b, p.n_cu, len(recs), 1000 * sum(r["ms"] for r in recs)), flush=True)
            seg += 1
        p.destroy()
    for _, _, m, _, _ in runs.values():
        m.destroy()
    a = torch.ones(CALIBRATION_BYTES // 4, dtype=torch.float32, device="cuda")
    c = torch.empty_like(a)
    torch.cuda.synchronize()
    pc = ds.Partition(1.0)
    pc.probe_cu_ids(MARKER_BASE + seg)
    c.copy_(a)
    torch.cuda.synchronize()
    pc.probe_cu_ids(END_MARKER)
    print("segment %d: calibration copy of %d bytes" % (seg, CALIBRATION_BYTES), flush=True)
    pc.destroy()


def kernel_class(name):
    for key, cls in (("probe_kernel", "marker"), ("conv_igemm_1x1s", "conv_1x1_stream"), ("conv_igemm", "conv"),
                     ("conv_rgb", "stem"), ("expand_dw", "expand_dw"), ("dwconv3x3", "dwconv3x3"),
                     ("fc_reduce", "fc"), ("fc_kernel", "fc"), ("lstm_step", "lstm_step"), ("maxpool", "pool"),
                     ("avgpool", "pool")):
        if key in name:
            return cls
    return "other"


def trace_times(trace_dir):
    """Per (segment, kernel class) summed kernel durations (us) of a
    rocprofv3 kernel-trace run of the same sweep."""
    out = {}
    for path in glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True):
        rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Dispatch_Id"]))
        seg = None
        for r in rows:
            cls = kernel_class(r["Kernel_Name"])
            grid = int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
            if cls == "marker":
                seg = grid // 64 - MARKER_BASE if grid // 64 >= MARKER_BASE else None
                continue
            if seg is not None:
                key = (seg, cls)
                out[key] = out.get(key, 0.0) + (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3
    return out


def summarize(dirs):
    """Per (segment, kernel class) sums of the counters of all passes (the
    dispatches between a segment's marker and the end marker); dispatch
    counts are those of the first pass; times those of a kernel-trace run
    when one is given with --trace, else of the first pass."""
    trace = trace_times(TRACE_DIR[0]) if TRACE_DIR else {}
    segs = collections.OrderedDict()
    for pi, d in enumerate(dirs):
        for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            disp = collections.OrderedDict()
            for r in csv.DictReader(open(path)):
                k = int(r["Dispatch_Id"])
                e = disp.setdefault(k, dict(name=r["Kernel_Name"], grid=int(r["Grid_Size"]),
                                            t=(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3, c={}))
                e["c"][r["Counter_Name"]] = e["c"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
            seg = None
            for k in sorted(disp):
                e = disp[k]
                cls = kernel_class(e["name"])
                if cls == "marker":
                    seg = e["grid"] // 64 - MARKER_BASE if e["grid"] // 64 >= MARKER_BASE else None
                    continue
                if seg is None:
                    continue
                agg = segs.setdefault(seg, collections.OrderedDict()).setdefault(cls, dict(n=0, us=0.0, c={}))
                if pi == 0:
                    agg["n"] += 1
                    agg["us"] += e["t"]
                for cn, v in e["c"].items():
                    agg["c"][cn] = agg["c"].get(cn, 0.0) + v
    last = max(segs) if segs else None
    cal = segs.get(last, {}).get("other", {}).get("c", {})
    f_fetch = CALIBRATION_BYTES / (1024.0 * cal["FETCH_SIZE"]) if cal.get("FETCH_SIZE") else None
    f_write = CALIBRATION_BYTES / (1024.0 * cal["WRITE_SIZE"]) if cal.get("WRITE_SIZE") else None
    print("calibration (256 MiB device copy): bytes moved per byte counted: FETCH_SIZE %s, WRITE_SIZE %s" %
          ("%.3f" % f_fetch if f_fetch else "-", "%.3f" % f_write if f_write else "-"))
    print("| CUs | model | kernel class | dispatches | us (%s) | MFMA TFLOP/s (op counter) | "
          % ("kernel trace" if trace else "counter run") +
          "of partition peak | MFMA busy cycles / (GUI cycles x CUs) | HBM MB read | HBM MB written | GB/s |")
    print("|---|---|---|---|---|---|---|---|---|---|---|")
    labels = sweep_segments()
    for seg, classes in segs.items():
        if seg == last:
            continue
        arch, b, n_cu = labels[seg]
        for cls, a in classes.items():
            c = a["c"]
            if (seg, cls) in trace:
                a["us"] = trace[(seg, cls)]
            mops = c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16")
            tf = mops * 512 / (a["us"] * 1e-6) / 1e12 if mops and a["us"] > 0 else None
            busy = c.get("SQ_VALU_MFMA_BUSY_CYCLES")
            gui = c.get("GRBM_GUI_ACTIVE")
            rd = c["FETCH_SIZE"] * 1024 * f_fetch / 1e6 if "FETCH_SIZE" in c and f_fetch else None
            wr = c["WRITE_SIZE"] * 1024 * f_write / 1e6 if "WRITE_SIZE" in c and f_write else None
            gbs = (rd + wr) * 1e6 / (a["us"] * 1e-6) / 1e9 if rd is not None and wr is not None and a["us"] else None
            fmt = lambda v, f: (f % v) if v is not None else "-"
            print("| %d | %s b%d | %s | %d | %.1f | %s | %s | %s | %s | %s | %s |" % (
                n_cu, arch, b, cls, a["n"], a["us"], fmt(tf, "%.1f"),
                fmt(tf / (2516.6 * n_cu / 256) if tf else None, "%.3f"),
                fmt(busy / (gui * n_cu) if busy and gui else None, "%.3f"), fmt(rd, "%.1f"), fmt(wr, "%.1f"),
                fmt(gbs, "%.0f")))
    if any("SQ_WAVE_CYCLES" in a["c"] for classes in segs.values() for a in classes.values()):
        stalls(segs, last, labels)
    if any("SQ_INSTS_LDS_LOAD_BANDWIDTH" in a["c"] for classes in segs.values() for a in classes.values()):
        lds_port(segs, last, labels)


def stalls(segs, last, labels):
    """Where the waves' time goes, per (partition, model, kernel class): the
    SQ wave-state counters as shares of SQ_WAVE_CYCLES (all count
    wave-cycles; the VALU share includes the MFMA instructions' issue), and
    the raw ratio of the MFMA busy counter to GRBM_GUI_ACTIVE x CUs."""
    print()
    print("| CUs | model | kernel class | waves | waiting on dependencies | waiting to issue | issuing: any | VMEM | "
          "LDS | VALU | scalar | MFMA busy / (GUI cycles x CUs) |")
    print("|---|---|---|---|---|---|---|---|---|---|---|---|")
    for seg, classes in segs.items():
        if seg == last:
            continue
        arch, b, n_cu = labels[seg]
        for cls, a in classes.items():
            c = a["c"]
            wc = c.get("SQ_WAVE_CYCLES")
            if not wc:
                continue
            sh = lambda k: ("%.2f" % (c[k] / wc)) if k in c else "-"
            busy, gui = c.get("SQ_VALU_MFMA_BUSY_CYCLES"), c.get("GRBM_GUI_ACTIVE")
            print("| %d | %s b%d | %s | %d | %s | %s | %s | %s | %s | %s | %s | %s |" % (
                n_cu, arch, b, cls, int(c.get("SQ_WAVES", 0)), sh("SQ_WAIT_ANY"), sh("SQ_WAIT_INST_ANY"),
                sh("SQ_ACTIVE_INST_ANY"), sh("SQ_ACTIVE_INST_VMEM"), sh("SQ_ACTIVE_INST_LDS"),
                sh("SQ_ACTIVE_INST_VALU"), sh("SQ_ACTIVE_INST_SCA"),
                "%.3f" % (busy / (gui * n_cu)) if busy and gui else "-"))


LDS_PORT_BYTES_PER_CLK = 128  # one CU's LDS bandwidth (bytes per clock)
SHADER_MHZ = 2400             # the MI355X's peak engine clock


def lds_port(segs, last, labels):
    """LDS traffic per (partition, model, kernel class), per CU and clock
    cycle of the class's kernel-trace time at the 2.4 GHz peak clock (a lower
    clock would raise every per-cycle figure): LDS reads =
    SQ_INSTS_LDS_LOAD_BANDWIDTH x 64 bytes (ds_read data); LDS fills by the
    buffer-to-LDS loads = TA_BUFFER_READ_LDS_WAVEFRONTS x 1 KB (every such
    load of this library moves 16 bytes per lane); the MFMA busy counter per
    SIMD-cycle; the LDS bytes the class moves per MFMA-busy cycle, and the
    MFMA share a 128-byte-per-clock LDS port would allow at that ratio; the
    bank-conflict and full-data-FIFO counters per CU-cycle as read."""
    print()
    print("| CUs | model | kernel class | us | LDS read B/clk/CU | LDS fill B/clk/CU | LDS total B/clk/CU | "
          "MFMA busy / SIMD-cycle | LDS B per MFMA-busy cycle | MFMA share the LDS port allows | "
          "bank conflict / CU-cycle | data FIFO full / CU-cycle |")
    print("|---|---|---|---|---|---|---|---|---|---|---|---|")
    for seg, classes in segs.items():
        if seg == last:
            continue
        arch, b, n_cu = labels[seg]
        for cls, a in classes.items():
            c = a["c"]
            if "SQ_INSTS_LDS_LOAD_BANDWIDTH" not in c or not a["us"]:
                continue
            cu_cyc = a["us"] * SHADER_MHZ * n_cu
            rd = c["SQ_INSTS_LDS_LOAD_BANDWIDTH"] * 64 / cu_cyc
            fill_w = c.get("TA_BUFFER_READ_LDS_WAVEFRONTS_sum", c.get("TA_BUFFER_READ_LDS_WAVEFRONTS"))
            tot = rd + (fill_w * 1024 / cu_cyc if fill_w is not None else 0.0)
            busy = c.get("SQ_VALU_MFMA_BUSY_CYCLES")
            share = busy / (4 * cu_cyc) if busy else None
            per_busy = tot / share if share else None
            per = lambda k: ("%.3f" % (c[k] / cu_cyc)) if k in c else "-"
            print("| %d | %s b%d | %s | %.1f | %.1f | %s | %.1f | %s | %s | %s | %s | %s |" % (
                n_cu, arch, b, cls, a["us"], rd, "%.1f" % (tot - rd) if fill_w is not None else "-", tot,
                "%.3f" % share if share is not None else "-", "%.0f" % per_busy if per_busy else "-",
                "%.2f" % min(1.0, LDS_PORT_BYTES_PER_CLK / per_busy) if per_busy else "-",
                per("SQ_LDS_BANK_CONFLICT"), per("SQ_LDS_DATA_FIFO_FULL")))


# bench.py's markers: the roofline forwards of model i follow 1000 + 100 + i,
# its calibration copy follows 1000 + 199
BENCH_MODEL_SEG, BENCH_CAL_SEG = 100, 199
BENCH_MODELS = ["resnet50", "mobilenetv2", "vgg19", "lstm2"]
CONV_SRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", "conv_igemm.hip")


def _segmented(rows, grid_of):
    """(segment or None, row) in dispatch order; a marker opens a segment,
    the end marker closes it."""
    seg = None
    for r in sorted(rows, key=lambda r: int(r["Dispatch_Id"])):
        if kernel_class(r["Kernel_Name"]) == "marker":
            g = grid_of(r) // 64
            seg = g - MARKER_BASE if g >= MARKER_BASE else None
            continue
        yield seg, r


def _bench_json(path):
    for line in open(path):
        line = line.strip()
        if line.startswith("{") and '"metric"' in line:
            return json.loads(line)
    raise SystemExit("no bench JSON line in %s" % path)


def bench_kernels(trace_dir, bench_log, ref_log=None):
    """Markdown summary of a kernel-trace run of bench.py: the implicit-GEMM
    convolution dispatches of the roofline forwards (the launches the
    bench's own figure averages) against the bench's HIP-event figure, and
    the top kernels of the whole command."""
    path = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)[0]
    grid = lambda r: int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
    per = collections.OrderedDict((i, []) for i in range(len(BENCH_MODELS)))
    for seg, r in _segmented(csv.DictReader(open(path)), grid):
        if seg is not None and BENCH_MODEL_SEG <= seg < BENCH_MODEL_SEG + len(BENCH_MODELS):
            if kernel_class(r["Kernel_Name"]) in ("conv", "conv_1x1_stream"):
                per[seg - BENCH_MODEL_SEG].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3)
    allv = [v for vs in per.values() for v in vs]
    bj = _bench_json(bench_log)
    rf = bj["roofline"]
    print("| quantity | value |")
    print("|---|---|")
    print("| operating point | k = %g, over-provision %d slots, batches %s, deployed slots %s, home offsets %s |" % (
        bj["config"]["capacity_k"], bj["config"]["overprov_slots"], bj["config"]["batch"],
        bj["config"]["deployed_slots"], bj["config"]["home_offset"]))
    for i, vs in per.items():
        if vs:
            print("| %s conv dispatches / mean us (rocprofv3) | %d / %.2f |" % (BENCH_MODELS[i], len(vs),
                                                                            sum(vs) / len(vs)))
    print("| all conv dispatches of the roofline forwards / mean us (rocprofv3) | %d / %.2f |" % (
        len(allv), sum(allv) / max(len(allv), 1)))
    print("| same launches, HIP events inside bench.py under the profiler: launches per pass / mean us | %d / %.2f |"
          % (rf["launches"], rf["avg_launch_us"]))
    if ref_log:
        r0 = _bench_json(ref_log)["roofline"]
        print("| same, unprofiled bench run: launches per pass / mean us | %d / %.2f |" % (r0["launches"],
                                                                                        r0["avg_launch_us"]))
    print("| algorithmic FLOP per launch (bench) | %.4g |" % rf["flops_per_launch"])
    print("| achieved TFLOP/s = FLOP per launch / rocprofv3 mean | %.1f |" % (
        rf["flops_per_launch"] / (sum(allv) / max(len(allv), 1) * 1e-6) / 1e12))
    stats = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)
    if stats:
        print("\nTop kernels of the whole command (rocprofv3 --stats):\n")
        print("| kernel | calls | total ms | avg us | min us | max us |")
        print("|---|---|---|---|---|---|")
        for r in list(csv.DictReader(open(stats[0])))[:12]:
            name = r["Name"] if len(r["Name"]) < 110 else r["Name"][:107] + "..."
            print("| `%s` | %s | %.2f | %.1f | %.1f | %.1f |" % (name, r["Calls"], int(r["TotalDurationNs"]) * 1e-6,
                                                              float(r["AverageNs"]) * 1e-3, int(r["MinNs"]) * 1e-3,
                                                              int(r["MaxNs"]) * 1e-3))


def bench_traffic(fetch_dir, write_dir, bench_log):
    """Markdown summary of two counter runs of bench.py (FETCH_SIZE, then
    WRITE_SIZE): calibrated HBM bytes per implicit-GEMM conv launch of the
    roofline forwards, with the conv source hash and the operating point the
    bench checks before using the figure."""
    tot, cal, n = {}, {}, {}
    for cname, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        path = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == cname]
        by = collections.OrderedDict()
        for r in rows:  # one row per dispatch and counter instance: sum them
            e = by.setdefault(int(r["Dispatch_Id"]), dict(r, v=0.0))
            e["v"] += float(r["Counter_Value"])
        tot[cname] = cal[cname] = 0.0
        n[cname] = 0
        for seg, e in _segmented(by.values(), lambda r: int(r["Grid_Size"])):
            if seg == BENCH_CAL_SEG:
                cal[cname] += e["v"]
            elif seg is not None and BENCH_MODEL_SEG <= seg < BENCH_MODEL_SEG + len(BENCH_MODELS) and \
                    kernel_class(e["Kernel_Name"]) in ("conv", "conv_1x1_stream"):
                tot[cname] += e["v"]
                n[cname] += 1
    cal_kib = CALIBRATION_BYTES / 1024.0
    f = {c: cal_kib / cal[c] if cal[c] else None for c in cal}
    bj = _bench_json(bench_log)
    rf = bj["roofline"]
    print("| quantity | FETCH | WRITE |")
    print("|---|---|---|")
    print("| conv dispatches counted | %d | %d |" % (n["FETCH_SIZE"], n["WRITE_SIZE"]))
    print("| calibration copy reading (KiB) vs %d KiB moved | %.0f | %.0f |" % (cal_kib, cal["FETCH_SIZE"],
                                                                              cal["WRITE_SIZE"]))
    print("| calibration factor | %.4f | %.4f |" % (f["FETCH_SIZE"], f["WRITE_SIZE"]))
    per = {c: tot[c] * 1024 * f[c] / max(n[c], 1) for c in tot}
    print("| bytes per conv launch (calibrated) | %.4g | %.4g |" % (per["FETCH_SIZE"], per["WRITE_SIZE"]))
    print("\nAlgorithmic bytes per launch (each input, weight, residual and output once): %.4g\n" %
          rf["algorithmic_bytes_per_launch"])
    plan = {k: bj["config"][k] for k in ("batch", "deployed_slots", "home_offset")}
    print("traffic_bytes_per_launch: %.6g" % (per["FETCH_SIZE"] + per["WRITE_SIZE"]))
    print("plan: %s" % json.dumps(plan))
    print("source_sha256: %s" % hashlib.sha256(open(CONV_SRC, "rb").read()).hexdigest())


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--arch", default="resnet50", choices=ds.ARCHS)
    ap.add_argument("--batch", type=int, default=16)
    ap.add_argument("--fraction", type=float, default=1.0)
    ap.add_argument("--reps", type=int, default=3)
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--compare-blas", action="store_true")
    ap.add_argument("--sweep", action="store_true")
    ap.add_argument("--cases", nargs="+", default=None, metavar="ARCH:BATCH:SLOTS",
                    help="with --sweep / --summarize: these models on partitions of that many slots")
    ap.add_argument("--summarize", nargs="+", default=None)
    ap.add_argument("--trace", default=None, help="with --summarize: a kernel-trace run of the same sweep")
    ap.add_argument("--bench-kernels", nargs="+", default=None, metavar=("TRACE_DIR", "BENCH_LOG"),
                    help="kernel-trace run of bench.py, its output, [an unprofiled bench output]")
    ap.add_argument("--bench-traffic", nargs=3, default=None, metavar=("FETCH_DIR", "WRITE_DIR", "BENCH_LOG"))
    a = ap.parse_args()
    if a.cases:
        for c in a.cases:
            arch, b, sl = c.split(":")
            CASES.append((arch, int(b), int(sl)))
    if a.bench_kernels:
        return bench_kernels(*a.bench_kernels)
    if a.bench_traffic:
        return bench_traffic(*a.bench_traffic)
    if a.sweep:
        return sweep()
    if a.summarize:
        if a.trace:
            TRACE_DIR.append(a.trace)
        return summarize(a.summarize)

    m = ds.Model(a.arch, a.seed)
    p = ds.Partition(a.fraction)
    g = torch.Generator(device="cuda").manual_seed(a.seed)
    x = torch.randn(m.input_shape(a.batch), device="cuda", generator=g).to(torch.bfloat16)
    y = torch.empty(m.output_shape(a.batch), device="cuda", dtype=torch.float32)
    for _ in range(3):
        m.infer(a.batch, x, y, p)
    p.synchronize()
    recs = m.profile_layers(a.batch, x, y, p)
    for _ in range(a.reps - 1):
        for r, r2 in zip(recs, m.profile_layers(a.batch, x, y, p)):
            r["ms"] += r2["ms"]
    for r in recs:
        r["ms"] /= a.reps

    blas = {}
    if a.compare_blas:
        s = torch.cuda.ExternalStream(p.stream_ptr)
        for r in recs:
            M, N, K = r["gemm"]
            if r["kind"] != 0 or (M, N, K) in blas:
                continue
            A = torch.randn(M, K, device="cuda", dtype=torch.bfloat16)
            B = torch.randn(N, K, device="cuda", dtype=torch.bfloat16)
            with torch.cuda.stream(s):
                for _ in range(3):
                    torch.matmul(A, B.t())
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(s)
                for _ in range(10):
                    torch.matmul(A, B.t())
                e1.record(s)
            torch.cuda.synchronize()
            blas[(M, N, K)] = e0.elapsed_time(e1) / 10

    tot = sum(r["ms"] for r in recs)
    print("%s batch %d on %d CUs: %d kernels, %.3f ms" % (a.arch, a.batch, p.n_cu, len(recs), tot))
    for r in recs:
        line = "  %-9s %-22s %8.1f us" % (ds.KIND_NAMES[r["kind"]], str(r["gemm"]), 1000 * r["ms"])
        if r["flops"]:
            line += " %7.1f TFLOP/s" % (r["flops"] / (r["ms"] * 1e-3) / 1e12)
        if r["bytes"]:
            line += " %7.1f GB/s" % (r["bytes"] / (r["ms"] * 1e-3) / 1e9)
        if r["gemm"] in blas:
            line += "   hipBLASLt %.1f us" % (1000 * blas[r["gemm"]])
        print(line)
    if blas:
        mine = sum(r["ms"] for r in recs if r["kind"] == 0)
        ref = sum(blas[r["gemm"]] for r in recs if r["kind"] == 0)
        print("MFMA layers: this kernel %.3f ms, hipBLASLt GEMMs of the same shapes %.3f ms" % (mine, ref))


if __name__ == "__main__":
    main()
