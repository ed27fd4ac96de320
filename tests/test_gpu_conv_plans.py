"""Every launch plan the convolution takes in the measured workloads, on the
GPU against the fp64 oracle.

The tiled implicit-GEMM kernel chooses its tile, depth split (split-K) and
LDS ring depth from the layer shape and the CUs of the partition it runs on.
The plans are enumerated on the host (dstack_arch_convs, dstack_conv2d_plan)
for the configured models and batches -- ResNet-50 at 1/8/16/32, MobileNetV2
at 32, VGG-19 at 8, the LSTM's input projections at 32, the tiny CNN at 4 --
over the ten sweep fractions (24..256 CUs).  One layer per distinct plan
(the cheapest to check) runs through dstack_op_conv2d_ws on a partition of
that CU count with a split-K workspace, as inside a model; split plans also
get a residual so that the fused reduction's epilogue sees one.  The oracle
computes the sampled images {0, N-1} (batch items are independent), or 64
sampled rows plus the last for the LSTM projection.

Also: forced splits on small ragged shapes at several CU counts (both
reduction widths: one slice per round for 128x128 tiles, several for
smaller tiles), the arrival counters back at zero after every call, and an
fp32 output that never splits.

Bar: infinity-norm relative error <= 2e-2."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

TOL = 2e-2
FRACTIONS = [0.1 * i for i in range(1, 11)]
WORKLOADS = [("resnet50", 1), ("resnet50", 8), ("resnet50", 16), ("resnet50", 32), ("mobilenetv2", 32),
             ("vgg19", 8), ("lstm2", 32), ("tinycnn", 4)]


def _oracle_macs(c):
    Ho = (c["H"] + 2 * c["pad"] - c["R"]) // c["stride"] + 1
    Wo = (c["W"] + 2 * c["pad"] - c["S"]) // c["stride"] + 1
    items = 65 if c["H"] == 1 and c["W"] == 1 else min(c["N"], 2)
    return items * Ho * Wo * c["K"] * c["R"] * c["S"] * c["C"]


def plan_cases():
    """(plan key, n_cu, conv shape) for every distinct plan, the cheapest
    instance of each; [] when the library is not built."""
    try:
        import paper_2304_13541_amd as ds
        best = {}
        for arch, b in WORKLOADS:
            for c in ds.arch_convs(arch, b):
                for f in FRACTIONS:
                    n_cu = 8 * ds.fraction_to_slots(f)
                    p = ds.conv2d_plan(c["N"], c["H"], c["W"], c["C"], c["K"], c["R"], c["S"], c["stride"], c["pad"],
                                       c["act"], c["out_fp32"], n_cu)
                    key = (p["kernel"], p["mode"], p["tile_n"], p["tile_m"], p["splits"], p["stages"])
                    if key not in best or _oracle_macs(c) < _oracle_macs(best[key][1]):
                        best[key] = (n_cu, c, arch, b)
        return [(k,) + v for k, v in sorted(best.items())]
    except Exception:
        return []


CASES = plan_cases()


@pytest.fixture(scope="module")
def env(oracle_mod):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2304_13541_amd as ds
    from tests import gpu_util as gu
    from tests import inputs
    return ds, gu, inputs, oracle_mod, torch


def reference(oracle, xb, wb, scale, shift, resb, act, stride, pad):
    ref = oracle.conv2d(oracle.bf16_bits_to_f64(xb), oracle.bf16_bits_to_f64(wb), stride, pad)
    ref = ref * scale.astype(np.float64) + shift.astype(np.float64)
    if resb is not None:
        ref = ref + oracle.bf16_bits_to_f64(resb)
    if act == 1:
        ref = np.maximum(ref, 0)
    elif act == 2:
        ref = np.clip(ref, 0, 6)
    elif act == 3:
        from scipy.special import erf
        ref = 0.5 * ref * (1.0 + erf(ref / np.sqrt(2.0)))
    elif act == 4:
        ref = np.tanh(ref)
    return ref


def run_conv(env, c, n_cu, use_res, seed, stream=None, ws_bytes=None):
    """One conv through dstack_op_conv2d_ws; returns (host output, inputs, workspace tensor)."""
    ds, gu, inputs, oracle, torch = env
    N, H, W, C, K, R, S, st, pad, act = (c[k] for k in ("N", "H", "W", "C", "K", "R", "S", "stride", "pad", "act"))
    Ho, Wo = (H + 2 * pad - R) // st + 1, (W + 2 * pad - S) // st + 1
    xb = inputs.normal_bf16(seed, (N, H, W, C))
    wb = inputs.normal_bf16(seed + 1, (K, R, S, C), scale=(2.0 / (R * S * C)) ** 0.5)
    rng = np.random.default_rng(seed + 2)
    scale = rng.uniform(0.5, 1.5, K).astype(np.float32)
    shift = rng.uniform(-0.2, 0.2, K).astype(np.float32)
    resb = inputs.normal_bf16(seed + 3, (N, Ho, Wo, K)) if use_res else None
    f32 = bool(c["out_fp32"])
    y = gu.empty_f32((N, Ho, Wo, K)) if f32 else gu.empty_bf16((N, Ho, Wo, K))
    plan = ds.conv2d_plan(N, H, W, C, K, R, S, st, pad, act, f32, n_cu)
    nbytes = ws_bytes if ws_bytes is not None else max(plan["workspace_bytes"], 16384)
    ws = torch.zeros(nbytes // 4 + 64, dtype=torch.int32, device="cuda:0")
    ds.conv2d_ws(gu.dev_bf16(xb), gu.dev_bf16(wb), K, R, S, st, pad, gu.dev_f32(scale), gu.dev_f32(shift),
                 gu.dev_bf16(resb) if use_res else None, act, y, ws, out_fp32=f32, n_cu=n_cu, stream=stream)
    torch.cuda.synchronize()
    return gu.host(y), (xb, wb, scale, shift, resb), ws, plan


def check(env, c, got, data, items=None):
    ds, gu, inputs, oracle, torch = env
    xb, wb, scale, shift, resb = data
    if items is None:
        if c["H"] == 1 and c["W"] == 1:
            rng = np.random.default_rng(5)
            items = sorted(set(rng.choice(c["N"], size=min(64, c["N"]), replace=False).tolist()) | {c["N"] - 1})
        else:
            items = sorted({0, c["N"] - 1})
    ref = reference(oracle, xb[items], wb, scale, shift, None if resb is None else resb[items], c["act"], c["stride"],
                    c["pad"])
    err = oracle.rel_err(got[items], ref)
    print("  items %s rel_err %.3e" % (items if len(items) <= 4 else "%d rows" % len(items), err), flush=True)
    assert np.all(np.isfinite(got[items]))
    assert err <= TOL
    return err


@pytest.mark.parametrize("case", CASES, ids=["k%d-m%d-%dx%d-s%d-st%d" % k[0] for k in CASES])
def test_conv_plan(env, case):
    ds, gu, inputs, oracle, torch = env
    key, n_cu, c, arch, b = case
    use_res = bool(c["has_residual"]) or key[4] > 1
    print("plan %s on %d CUs: %s b%d layer %s residual=%d" % (key, n_cu, arch, b, c, use_res), flush=True)
    part = ds.Partition(slot_offset=0, n_slots=n_cu // 8)
    try:
        got, data, ws, plan = run_conv(env, c, n_cu, use_res, 100 + n_cu, stream=part.stream_ptr)
        assert (plan["kernel"], plan["mode"], plan["tile_n"], plan["tile_m"], plan["splits"], plan["stages"]) == key
        check(env, c, got, data)
        assert int(ws[:4096].abs().sum().item()) == 0, "split-K arrival counters must be back at zero"
    finally:
        part.destroy()


FORCED = [
    # N, H, W, C, K, R, stride, pad, act: deep, narrow layers with a ragged pixel count
    (2, 7, 7, 512, 256, 3, 1, 1, 1),
    (1, 7, 7, 2048, 512, 1, 1, 0, 0),
    (3, 5, 5, 256, 128, 3, 1, 1, 2),
    (1, 14, 14, 1024, 256, 1, 1, 0, 1),
    (1, 13, 13, 512, 512, 3, 2, 1, 1),
    (2, 9, 9, 256, 384, 3, 1, 1, 0),
    (8, 7, 7, 512, 256, 3, 1, 1, 1),   # 128 x 128 tiles, 4 slices at 24 CUs
    (8, 15, 15, 256, 128, 3, 1, 1, 2),  # 128 x 128 tiles, 2 slices at 24 CUs, ragged pixels
]


def test_conv2d_ws_forced_splits(env):
    """Small ragged shapes that split at the chosen CU counts, with and
    without a residual; both reduction widths (128x128 tiles read one slice
    per round, smaller tiles several) must appear."""
    ds, gu, inputs, oracle, torch = env
    seen_tiles, n = set(), 0
    for N, H, W, C, K, R, st, pad, act in FORCED:
        c = dict(N=N, H=H, W=W, C=C, K=K, R=R, S=R, stride=st, pad=pad, act=act, has_residual=0, out_fp32=0)
        for n_cu in (24, 104, 256):
            plan = ds.conv2d_plan(N, H, W, C, K, R, R, st, pad, act, False, n_cu)
            if plan["splits"] <= 1:
                continue
            for use_res in (False, True):
                print("forced split %s n_cu %d residual %d plan %s" % ((N, H, W, C, K, R, st, pad), n_cu, use_res,
                                                                      plan), flush=True)
                got, data, ws, p2 = run_conv(env, c, n_cu, use_res, 7 + n)
                assert p2["splits"] > 1
                check(env, c, got, data)
                assert int(ws[:4096].abs().sum().item()) == 0
                seen_tiles.add((plan["tile_n"], plan["tile_m"]))
                n += 1
    assert n >= 6
    assert (128, 128) in seen_tiles and any(t != (128, 128) for t in seen_tiles), seen_tiles


def test_conv2d_ws_small_workspace_and_fp32(env):
    """A workspace below the plan's need runs fewer splits (same values up to
    summation order); an fp32 output never splits; no workspace at all runs
    unsplit."""
    ds, gu, inputs, oracle, torch = env
    c = dict(N=2, H=7, W=7, C=512, K=256, R=3, S=3, stride=1, pad=1, act=1, has_residual=0, out_fp32=0)
    full = ds.conv2d_plan(2, 7, 7, 512, 256, 3, 3, 1, 1, 1, False, 256)
    assert full["splits"] > 1
    small = full["workspace_bytes"] // 2
    part = ds.conv2d_plan(2, 7, 7, 512, 256, 3, 3, 1, 1, 1, False, 256, workspace_bytes=small)
    assert part["splits"] < full["splits"]
    got, data, ws, _ = run_conv(env, c, 256, False, 31, ws_bytes=small)
    check(env, c, got, data)
    assert ds.conv2d_plan(2, 7, 7, 512, 256, 3, 3, 1, 1, 1, False, 256, workspace_bytes=0)["splits"] == 1
    c32 = dict(c, out_fp32=1)
    assert ds.conv2d_plan(2, 7, 7, 512, 256, 3, 3, 1, 1, 1, True, 256)["splits"] == 1
    got, data, ws, _ = run_conv(env, c32, 256, True, 41)
    check(env, c32, got, data)
