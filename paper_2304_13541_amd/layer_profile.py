"""Per-layer kernel times of one model on one CU-masked partition.

    python -m paper_2304_13541_amd.layer_profile --arch resnet50 --batch 16 --fraction 0.4 [--compare-blas]

Times every kernel of a forward with HIP events on the partition's stream
(dstack_profile_layers, mean of --reps forwards) and prints, per MFMA layer,
its GEMM shape (pixels, output channels, depth), time and TFLOP/s.  With
--compare-blas it also times torch.matmul (hipBLASLt) on bf16 matrices of the
same GEMM shape on the same masked stream, as a vendor-library reference.
Inputs are synthetic N(0,1) values.

    python -m paper_2304_13541_amd.layer_profile --sweep
    python -m paper_2304_13541_amd.layer_profile --summarize PASS_DIR [PASS_DIR ...]

--sweep runs the measured workloads (ResNet-50 b16, MobileNetV2 b32, VGG-19
b8, the LSTM b32) on partitions of 25%, 50% and 100% of the CUs, one eager
forward each (run it with DSTACK_GRAPH=0 under rocprofv3), every segment
preceded by a marker dispatch (the CU-id probe with 1000 + segment
workgroups), and ends with a 256 MiB device copy that calibrates the HBM
byte counters.  --summarize reads the rocprofv3 counter CSVs of such runs
(counters SQ_VALU_MFMA_BUSY_CYCLES, SQ_INSTS_VALU_MFMA_MOPS_BF16,
GRBM_GUI_ACTIVE, FETCH_SIZE, WRITE_SIZE in any passes), splits them at the
markers and prints per (partition, model, kernel class): dispatches, time,
MFMA rate from the MFMA op counter against the partition's peak, MFMA busy
cycles per CU-cycle, and calibrated HBM bytes and GB/s.
"""
import argparse
import collections
import csv
import glob
import os

import torch

import paper_2304_13541_amd as ds

SWEEP_MODELS = [("resnet50", 16), ("mobilenetv2", 32), ("vgg19", 8), ("lstm2", 32)]
SWEEP_FRACTIONS = [0.25, 0.5, 1.0]
MARKER_BASE = 1000
END_MARKER = 999
CALIBRATION_BYTES = 256 << 20
TRACE_DIR = []


def sweep():
    seg = 0
    runs = []
    for arch, b in SWEEP_MODELS:
        m = ds.Model(arch, 1)
        g = torch.Generator(device="cuda").manual_seed(1)
        x = torch.randn(m.input_shape(b), device="cuda", generator=g).to(torch.bfloat16)
        runs.append((arch, b, m, x, torch.empty(m.output_shape(b), device="cuda", dtype=torch.float32)))
    for f in SWEEP_FRACTIONS:
        p = ds.Partition(f)
        for arch, b, m, x, y in runs:
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
    for _, _, m, _, _ in runs:
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
    for seg, classes in segs.items():
        if seg == last:
            continue
        fi, mi = divmod(seg, len(SWEEP_MODELS))
        n_cu = 8 * ds.fraction_to_slots(SWEEP_FRACTIONS[fi])
        arch, b = SWEEP_MODELS[mi]
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--arch", default="resnet50", choices=ds.ARCHS)
    ap.add_argument("--batch", type=int, default=16)
    ap.add_argument("--fraction", type=float, default=1.0)
    ap.add_argument("--reps", type=int, default=3)
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--compare-blas", action="store_true")
    ap.add_argument("--sweep", action="store_true")
    ap.add_argument("--summarize", nargs="+", default=None)
    ap.add_argument("--trace", default=None, help="with --summarize: a kernel-trace run of the same sweep")
    a = ap.parse_args()
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
