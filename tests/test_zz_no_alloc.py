"""The allocation-free convolution entry point (dstack_op_conv2d_noalloc)
against the workspace one (dstack_op_conv2d_ws) it is a variant of: two
calls in a row, the second on a smaller input, each on a shape whose plan
splits the depth (so the fixed scratch carries the slices and the arrival
counters), and one that does not split; the outputs must be identical (same
plan, slices summed in the same order) and within 2e-2 of the fp64 oracle.
A shape whose plan needs more scratch than the library holds is refused
before anything is launched."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

TOL = 2e-2

CALLS = [
    # N, H, W, C, K, R, stride, pad, act, residual, n_cu: the first split call, then a smaller one
    (2, 9, 9, 256, 384, 3, 1, 1, 1, True, 24),
    (2, 7, 7, 512, 256, 3, 1, 1, 2, False, 256),
    (1, 5, 5, 64, 96, 3, 1, 1, 1, False, 256),
]


@pytest.fixture(scope="module")
def env(oracle_mod):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2304_13541_amd as ds
    from tests import gpu_util as gu
    from tests import inputs
    return ds, gu, inputs, oracle_mod, torch


def test_noalloc_matches_workspace_entry_point(env):
    ds, gu, inputs, oracle, torch = env
    splits = []
    for i, (N, H, W, C, K, R, st, pad, act, use_res, n_cu) in enumerate(CALLS):
        print("noalloc call", i, (N, H, W, C, K, R, st, pad, act, use_res, n_cu), flush=True)
        Ho, Wo = (H + 2 * pad - R) // st + 1, (W + 2 * pad - R) // st + 1
        xb = inputs.normal_bf16(50 + i, (N, H, W, C))
        wb = inputs.normal_bf16(60 + i, (K, R, R, C), scale=(2.0 / (R * R * C)) ** 0.5)
        rng = np.random.default_rng(70 + i)
        scale = rng.uniform(0.5, 1.5, K).astype(np.float32)
        shift = rng.uniform(-0.2, 0.2, K).astype(np.float32)
        resb = inputs.normal_bf16(80 + i, (N, Ho, Wo, K)) if use_res else None
        args = (gu.dev_bf16(xb), gu.dev_bf16(wb), K, R, R, st, pad, gu.dev_f32(scale), gu.dev_f32(shift),
                gu.dev_bf16(resb) if use_res else None, act)
        plan = ds.conv2d_plan(N, H, W, C, K, R, R, st, pad, act, False, n_cu)
        splits.append(plan["splits"])
        assert plan["workspace_bytes"] <= ds.conv2d_noalloc_scratch_bytes()
        ws = torch.zeros(max(plan["workspace_bytes"], 16384) // 4 + 64, dtype=torch.int32, device="cuda:0")
        y_ws = gu.empty_bf16((N, Ho, Wo, K))
        y_na = gu.empty_bf16((N, Ho, Wo, K))
        y_na.fill_(float("nan"))
        ds.conv2d_ws(*args, y_ws, ws, n_cu=n_cu)
        ds.conv2d_noalloc(*args, y_na, n_cu=n_cu)
        torch.cuda.synchronize()
        a, b = gu.host(y_ws), gu.host(y_na)
        ref = oracle.conv2d(oracle.bf16_bits_to_f64(xb), oracle.bf16_bits_to_f64(wb), st, pad) * scale + shift
        if use_res:
            ref = ref + oracle.bf16_bits_to_f64(resb)
        ref = np.maximum(ref, 0) if act == 1 else np.clip(ref, 0, 6)
        err = oracle.rel_err(b, ref)
        print("  plan %s: noalloc == ws: %s, rel_err vs oracle %.3e" % (plan, np.array_equal(a, b), err), flush=True)
        assert np.all(np.isfinite(b))
        assert np.array_equal(a, b)
        assert err <= TOL
    assert splits[0] > 1 and splits[1] > 1 and splits[2] == 1


def test_noalloc_refuses_a_plan_beyond_its_scratch(env):
    ds, gu, inputs, oracle, torch = env
    N, H, C, K, n_cu = 8, 28, 2048, 2048, 128
    plan = ds.conv2d_plan(N, H, H, C, K, 3, 3, 1, 1, 1, False, n_cu)
    assert plan["workspace_bytes"] > ds.conv2d_noalloc_scratch_bytes()
    x = gu.empty_bf16((N, H, H, C))
    w = gu.empty_bf16((K, 3, 3, C))
    y = gu.empty_bf16((N, H, H, K))
    with pytest.raises(ds.DStackError) as e:
        ds.conv2d_noalloc(x, w, K, 3, 3, 1, 1, None, None, None, 1, y, n_cu=n_cu)
    assert e.value.status == ds.E_UNSUPPORTED and "scratch" in str(e.value)
