"""Per-layer kernel times of one model on one CU-masked partition.

    python -m paper_2304_13541_amd.layer_profile --arch resnet50 --batch 16 --fraction 0.4 [--compare-blas]

Times every kernel of a forward with HIP events on the partition's stream
(dstack_profile_layers, mean of --reps forwards) and prints, per MFMA layer,
its GEMM shape (pixels, output channels, depth), time and TFLOP/s.  With
--compare-blas it also times torch.matmul (hipBLASLt) on bf16 matrices of the
same GEMM shape on the same masked stream, as a vendor-library reference.
Inputs are synthetic N(0,1) values.
"""
import argparse

import torch

import paper_2304_13541_amd as ds


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--arch", default="resnet50", choices=ds.ARCHS)
    ap.add_argument("--batch", type=int, default=16)
    ap.add_argument("--fraction", type=float, default=1.0)
    ap.add_argument("--reps", type=int, default=3)
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--compare-blas", action="store_true")
    a = ap.parse_args()

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
