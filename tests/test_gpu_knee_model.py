"""Launch shapes of the library's own kernels (the per-kernel parallelism of
Sec. 4.3's analytical model), through the C ABI on the GPU: one entry per
timed unit of dstack_profile_layers with the same kind, FLOPs and bytes;
workgroup counts of kernels whose grid has a closed form (pools, the
depthwise kernel) equal that form; occupancy is at least one workgroup per
CU; recording launches nothing (the output buffer keeps its sentinel); and
the model's E_t over the partition's CU counts is non-increasing."""
import math

import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2304_13541_amd as ds
    from tests import gpu_util as gu
    from tests import inputs
    return ds, gu, inputs, torch


@pytest.mark.parametrize("arch,batch,frac", [("resnet50", 8, 0.5), ("mobilenetv2", 4, 0.25), ("lstm2", 2, 0.5),
                                             ("tinycnn", 4, 1.0)])
def test_shapes_align_with_profile(env, arch, batch, frac):
    ds, gu, inputs, torch = env
    print("kernel_shapes", arch, batch, frac, flush=True)
    m = ds.Model(arch, 7)
    p = ds.Partition(frac)
    if arch == "lstm2":
        x = gu.dev_bf16(inputs.sequence_batch(8, batch))
    else:
        x = gu.dev_bf16(inputs.image_batch(8, batch, hw=32 if arch == "tinycnn" else 224))
    y = gu.empty_f32(m.output_shape(batch))
    m.infer(batch, x, y, p)
    p.synchronize()
    recs = m.profile_layers(batch, x, y, p)
    shapes = m.kernel_shapes(batch, x, y, p)
    assert len(shapes) == len(recs) > 0
    for s, r in zip(shapes, recs):
        assert s["kind"] == r["kind"]
        assert s["flops"] == r["flops"] and s["bytes"] == r["bytes"]
        assert s["launches"] >= 1 and s["workgroups"] >= 1 and s["blocks_per_cu"] >= 1
    if arch == "resnet50":  # the 3x3/2 max pool: one thread per (pixel, 8 channels), 256 per workgroup
        pools = [s for s in shapes if s["kind"] == 4]
        assert pools[0]["workgroups"] == math.ceil(batch * 56 * 56 * 64 // 8 / 256)
    if arch == "mobilenetv2":  # the depthwise kernel of the first block: 4 outputs x 8 channels per thread
        dw = [s for s in shapes if s["kind"] == 1]
        assert dw[0]["workgroups"] == math.ceil(batch * 112 * (112 // 4) * (32 // 8) / 256)
    # recording launches nothing: a sentinel in the output buffer survives a shapes call on it
    y.fill_(123.0)
    torch.cuda.synchronize()
    m.kernel_shapes(batch, x, y, p)
    p.synchronize()
    assert bool((y == 123.0).all())
    # E_t of the model built from these shapes never grows with more CUs
    t = [1000.0 * r["ms"] for r in recs]
    n = [s["workgroups"] / s["blocks_per_cu"] for s in shapes]
    tp = [ti * max(1.0, min(p.n_cu, ni)) / ni for ti, ni in zip(t, n)]
    grid = [8 * s for s in range(1, 33)]
    et, k = ds.knee_model_eval(n, tp, grid, 0.0)
    assert all(a >= b for a, b in zip(et, et[1:])) and 0 <= k < len(grid)
    m.destroy()
    p.destroy()
