"""Kernel-level parity on the GPU: each HIP kernel, called through the C ABI,
against the fp64 oracle on the same seeded bf16 inputs.  Shapes span several
tiles with ragged tails in every GEMM dimension, odd spatial sizes with
stride 2, K not a multiple of the tile, and every epilogue variant
(ReLU, ReLU6, GELU, tanh, residual, fp32 output).

Bar: infinity-norm relative error <= 2e-2 (bf16 inputs, fp32 accumulation,
bf16 or fp32 output)."""
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


CONV_CASES = [
    # N, H, W, C, K, R, stride, pad, act, residual, out_fp32
    (2, 9, 7, 16, 36, 3, 1, 1, 1, False, False),
    (1, 15, 15, 24, 20, 3, 2, 1, 2, False, False),
    (3, 5, 5, 64, 132, 1, 1, 0, 0, True, False),
    (2, 23, 23, 8, 64, 7, 2, 3, 1, False, False),
    (2, 28, 28, 64, 192, 3, 1, 1, 1, True, False),
    (1, 14, 14, 256, 1028, 1, 2, 0, 0, False, True),
    (4, 7, 7, 512, 512, 3, 1, 1, 1, False, False),
    (1, 1, 1, 520, 4, 1, 1, 0, 0, False, True),
    # 1x1 stride 1 with C <= 32 and K % 16 == 0: the streaming small-depth kernel
    # (ragged pixel counts, depth tails inside a 32-deep step, 1..8 channel blocks per wave);
    # C = 40..128 take the tiled kernel with its two-tile ring (one or two depth tiles)
    (2, 9, 7, 16, 96, 1, 1, 0, 2, False, False),
    (1, 11, 11, 24, 144, 1, 1, 0, 2, False, False),
    (3, 5, 7, 32, 16, 1, 1, 0, 0, False, True),
    (2, 6, 6, 64, 256, 1, 1, 0, 1, True, False),
    (1, 3, 3, 8, 48, 1, 1, 0, 1, False, False),
    (1, 4, 5, 40, 80, 1, 1, 0, 2, True, True),
    (2, 7, 9, 128, 512, 1, 1, 0, 1, True, False),
    (1, 5, 9, 96, 48, 1, 1, 0, 0, False, False),
    (3, 4, 7, 64, 64, 1, 1, 0, 0, True, True),
    (1, 3, 11, 120, 32, 1, 1, 0, 2, False, False),
    # the transformer's epilogues: GELU (feed-forward in) and tanh (pooler, a
    # 1x1 convolution of stride T picking each sequence's first token)
    (2, 1, 20, 768, 3072, 1, 1, 0, 3, False, False),
    (3, 1, 20, 768, 768, 1, 20, 0, 4, False, False),
    (1, 1, 7, 24, 64, 1, 1, 0, 3, True, False),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv2d(env, case):
    ds, gu, inputs, oracle, torch = env
    N, H, W, C, K, R, st, pad, act, use_res, f32 = case
    print("conv2d case", case, flush=True)
    xb = inputs.normal_bf16(1, (N, H, W, C))
    wb = inputs.normal_bf16(2, (K, R, R, C), scale=(2.0 / (R * R * C)) ** 0.5)
    rng = np.random.default_rng(3)
    scale = rng.uniform(0.5, 1.5, K).astype(np.float32)
    shift = rng.uniform(-0.2, 0.2, K).astype(np.float32)
    Ho, Wo = (H + 2 * pad - R) // st + 1, (W + 2 * pad - R) // st + 1
    resb = inputs.normal_bf16(4, (N, Ho, Wo, K)) if use_res else None
    y = gu.empty_f32((N, Ho, Wo, K)) if f32 else gu.empty_bf16((N, Ho, Wo, K))
    ds.conv2d(gu.dev_bf16(xb), gu.dev_bf16(wb), K, R, R, st, pad, gu.dev_f32(scale), gu.dev_f32(shift),
              gu.dev_bf16(resb) if use_res else None, act, y, out_fp32=f32)
    torch.cuda.synchronize()
    x = oracle.bf16_bits_to_f64(xb)
    w = oracle.bf16_bits_to_f64(wb)
    ref = oracle.conv2d(x, w, st, pad) * scale.astype(np.float64) + shift.astype(np.float64)
    if use_res:
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
    err = oracle.rel_err(gu.host(y), ref)
    print("rel_err", err)
    assert err <= TOL


RGB_CASES = [
    # N, H, W, K, R, stride, pad, act
    (2, 17, 16, 32, 3, 2, 1, 2),    # MobileNetV2-like stem, ragged last tile; W % 8 == 0 (vector row copy)
    (1, 32, 32, 16, 3, 1, 1, 1),    # the tiny CNN's stem
    (3, 9, 13, 32, 3, 2, 1, 0),     # W % 8 != 0 (element row copy), odd sizes, no activation
    (1, 5, 300, 16, 3, 1, 0, 1),    # output rows wider than a 256-pixel tile, pad 0
    (2, 11, 21, 64, 3, 1, 1, 1),    # VGG-19-like stem (3 x 3, 64 channels)
    (2, 23, 24, 64, 7, 2, 3, 1),    # ResNet-50-like stem (7 x 7 / 2, 64 channels)
    (1, 224, 224, 32, 3, 2, 1, 2),  # the full 224 x 224 MobileNetV2 stem
    (1, 224, 224, 64, 7, 2, 3, 1),  # the full 224 x 224 ResNet-50 stem
]


@pytest.mark.parametrize("case", RGB_CASES)
def test_conv2d_rgb(env, case):
    """Direct 3-channel stem conv on the matrix cores (weights [K][R][R][4],
    channel 3 zero) against the oracle's conv2d on the unpadded tensors."""
    ds, gu, inputs, oracle, torch = env
    N, H, W, K, R, st, pad, act = case
    print("conv2d_rgb case", case, flush=True)
    xb = inputs.normal_bf16(11, (N, H, W, 3))
    wb = inputs.normal_bf16(12, (K, R, R, 3), scale=(2.0 / (3 * R * R)) ** 0.5)
    w4 = np.zeros((K, R, R, 4), dtype=wb.dtype)
    w4[..., :3] = wb
    rng = np.random.default_rng(13)
    scale = rng.uniform(0.5, 1.5, K).astype(np.float32)
    shift = rng.uniform(-0.2, 0.2, K).astype(np.float32)
    Ho, Wo = (H + 2 * pad - R) // st + 1, (W + 2 * pad - R) // st + 1
    y = gu.empty_bf16((N, Ho, Wo, K))
    ds.conv2d_rgb(gu.dev_bf16(xb), gu.dev_bf16(w4), K, R, st, pad, gu.dev_f32(scale), gu.dev_f32(shift), act, y)
    torch.cuda.synchronize()
    ref = oracle.conv2d(oracle.bf16_bits_to_f64(xb), oracle.bf16_bits_to_f64(wb), st, pad)
    ref = ref * scale.astype(np.float64) + shift.astype(np.float64)
    ref = np.maximum(ref, 0) if act == 1 else (np.clip(ref, 0, 6) if act == 2 else ref)
    err = oracle.rel_err(gu.host(y), ref)
    print("rel_err", err)
    assert err <= TOL


@pytest.mark.parametrize("case", [(2, 11, 9, 32, 1), (1, 12, 12, 96, 2), (3, 7, 7, 960, 1), (2, 15, 13, 144, 2),
                                  (1, 30, 29, 32, 1),
                                  (1, 30, 30, 16, 1), (2, 7, 33, 24, 1), (1, 29, 29, 40, 2), (1, 5, 61, 8, 2)])
def test_dwconv3x3(env, case):
    """8 output pixels per thread on stride-1 output rows >= 28 wide with more
    than 32 channels, else 4; ragged last segments; zero padding on all borders."""
    ds, gu, inputs, oracle, torch = env
    N, H, W, C, st = case
    xb = inputs.normal_bf16(5, (N, H, W, C))
    wb = inputs.normal_bf16(6, (C, 3, 3), scale=0.47)
    rng = np.random.default_rng(7)
    scale = rng.uniform(0.5, 1.5, C).astype(np.float32)
    shift = rng.uniform(-0.2, 0.2, C).astype(np.float32)
    Ho, Wo = (H + 2 - 3) // st + 1, (W + 2 - 3) // st + 1
    y = gu.empty_bf16((N, Ho, Wo, C))
    w_rsc = np.ascontiguousarray(wb.reshape(C, 9).T.reshape(3, 3, C))  # device layout [3][3][C]
    ds.dwconv3x3(gu.dev_bf16(xb), gu.dev_bf16(w_rsc), st, gu.dev_f32(scale), gu.dev_f32(shift), 2, y)
    torch.cuda.synchronize()
    ref = oracle.dwconv(oracle.bf16_bits_to_f64(xb), oracle.bf16_bits_to_f64(wb), st, 1)
    ref = np.clip(ref * scale + shift, 0, 6)
    assert oracle.rel_err(gu.host(y), ref) <= TOL


EXPAND_DW_CASES = [
    # N, H, W, Cin, Ce, stride, act_e, act_d
    (2, 14, 14, 64, 384, 1, 2, 2),    # MobileNetV2 stage 4 (one 14 x 14 tile per chunk)
    (1, 15, 13, 24, 144, 2, 2, 2),    # odd sizes, stride 2
    (3, 7, 7, 160, 960, 1, 2, 2),     # depth 160 = 5 MFMA steps, 20 channel chunks
    (1, 9, 31, 16, 96, 2, 1, 0),      # depth 16 < 32 (zero tail), other activations
    (2, 56, 56, 24, 144, 1, 2, 2),    # several tiles per image with halos
    (1, 28, 28, 32, 192, 2, 2, 2),
    (1, 5, 6, 8, 48, 1, 0, 1),        # one partial tile, depth 8
    (2, 10, 9, 16, 64, 1, 2, 2),      # 64-channel chunks (Ce = 64)
    (1, 17, 19, 24, 144, 1, 2, 2),    # stride 1, partial tiles at both edges, odd tile width
]


@pytest.mark.parametrize("case", EXPAND_DW_CASES)
def test_expand_dw(env, case):
    """Fused expand 1x1 + BN + act, bf16 rounding of the expanded tensor,
    depthwise 3x3 + BN + act, against the oracle's conv2d and dwconv."""
    ds, gu, inputs, oracle, torch = env
    N, H, W, Cin, Ce, st, act_e, act_d = case
    print("expand_dw case", case, flush=True)
    xb = inputs.normal_bf16(21, (N, H, W, Cin))
    web = inputs.normal_bf16(22, (Ce, Cin), scale=(2.0 / Cin) ** 0.5)
    wdb = inputs.normal_bf16(23, (Ce, 3, 3), scale=0.47)
    rng = np.random.default_rng(24)
    se, sd = rng.uniform(0.5, 1.5, Ce).astype(np.float32), rng.uniform(0.5, 1.5, Ce).astype(np.float32)
    he, hd = rng.uniform(-0.2, 0.2, Ce).astype(np.float32), rng.uniform(-0.2, 0.2, Ce).astype(np.float32)
    Ho, Wo = (H + 2 - 3) // st + 1, (W + 2 - 3) // st + 1
    y = gu.empty_bf16((N, Ho, Wo, Ce))
    wd_rsc = np.ascontiguousarray(wdb.reshape(Ce, 9).T.reshape(3, 3, Ce))
    ds.expand_dw(gu.dev_bf16(xb), gu.dev_bf16(web), Ce, gu.dev_f32(se), gu.dev_f32(he), act_e, gu.dev_bf16(wd_rsc), st,
                 gu.dev_f32(sd), gu.dev_f32(hd), act_d, y)
    torch.cuda.synchronize()

    def act(v, a):
        return np.maximum(v, 0) if a == 1 else (np.clip(v, 0, 6) if a == 2 else v)
    w1 = oracle.bf16_bits_to_f64(web).reshape(Ce, 1, 1, Cin)
    e = act(oracle.conv2d(oracle.bf16_bits_to_f64(xb), w1, 1, 0) * se.astype(np.float64) + he.astype(np.float64), act_e)
    e = oracle.bf16_round(e)  # the expanded tensor is stored as bf16 (in LDS), as between two layers
    ref = act(oracle.dwconv(e, oracle.bf16_bits_to_f64(wdb), st, 1) * sd.astype(np.float64) + hd.astype(np.float64),
              act_d)
    err = oracle.rel_err(gu.host(y), ref)
    print("rel_err", err)
    assert err <= TOL


@pytest.mark.parametrize("split", [False, True])
@pytest.mark.parametrize("case", [(1, 64, 10, 0, True), (8, 25088, 40, 1, False), (16, 2048, 1000, 0, True),
                                  (32, 1280, 37, 1, False), (5, 520, 9, 2, True), (8, 4096, 1000, 0, True),
                                  (3, 72, 50, 1, False), (17, 9216, 33, 0, True), (32, 4096, 4096, 1, False)])
def test_fc(env, case, split):
    """Depth tails (I % 32 != 0), o-tile and batch-tile tails, and with a
    workspace the depth-split path (partial sums + reduce)."""
    ds, gu, inputs, oracle, torch = env
    B, I, O, act, f32 = case
    xb = inputs.normal_bf16(8, (B, I))
    wb = inputs.normal_bf16(9, (O, I), scale=(2.0 / I) ** 0.5)
    bias = np.random.default_rng(10).uniform(-0.5, 0.5, O).astype(np.float32)
    y = gu.empty_f32((B, O)) if f32 else gu.empty_bf16((B, O))
    ws = None
    if split:
        nbytes = ds.fc_workspace_bytes(B, I, O)
        ws = gu.empty_f32((max(nbytes // 4, 1),))
    ds.fc(gu.dev_bf16(xb), gu.dev_bf16(wb), gu.dev_f32(bias), act, y, out_fp32=f32, workspace=ws)
    torch.cuda.synchronize()
    ref = oracle.fc(oracle.bf16_bits_to_f64(xb), oracle.bf16_bits_to_f64(wb), bias)
    ref = np.maximum(ref, 0) if act == 1 else (np.clip(ref, 0, 6) if act == 2 else ref)
    assert oracle.rel_err(gu.host(y), ref) <= TOL


@pytest.mark.parametrize("case", [(2, 8, 8, 16, 2, 2, 0), (1, 112, 112, 64, 3, 2, 1), (3, 7, 9, 8, 3, 2, 1),
                                  (2, 7, 7, 2048, 3, 2, 1), (1, 7, 7, 1288, 2, 2, 0)])
def test_pools(env, case):
    ds, gu, inputs, oracle, torch = env
    N, H, W, C, k, st, pad = case
    xb = inputs.normal_bf16(11, (N, H, W, C))
    Ho, Wo = (H + 2 * pad - k) // st + 1, (W + 2 * pad - k) // st + 1
    y = gu.empty_bf16((N, Ho, Wo, C))
    ds.maxpool(gu.dev_bf16(xb), k, st, pad, y)
    g = gu.empty_bf16((N, C))
    ds.avgpool(gu.dev_bf16(xb), g)
    torch.cuda.synchronize()
    x = oracle.bf16_bits_to_f64(xb)
    assert np.array_equal(gu.host(y), oracle.maxpool(x, k, st, pad))  # a max of bf16 values is exact
    assert oracle.rel_err(gu.host(g), oracle.avgpool(x)) <= TOL


@pytest.mark.parametrize("case", [(5, 3, 64, 64), (50, 32, 512, 1024), (7, 17, 40, 96)])
def test_lstm_layer(env, case):
    ds, gu, inputs, oracle, torch = env
    T, B, I, H = case
    xb = inputs.normal_bf16(12, (T, B, I))
    a = 1.0 / np.sqrt(H)
    wih = inputs.uniform_bf16(13, (4 * H, I), -a, a)
    whh = inputs.uniform_bf16(14, (4 * H, H), -a, a)
    bias = np.random.default_rng(15).uniform(-2 * a, 2 * a, 4 * H).astype(np.float32)
    hb = gu.empty_bf16((T, B, H))
    hf = gu.empty_f32((T, B, H))
    ws = torch.empty(ds.lstm_workspace_bytes(T, B, H), dtype=torch.uint8, device="cuda:0")
    ds.lstm_layer(gu.dev_bf16(xb), gu.dev_bf16(wih), gu.dev_bf16(whh), gu.dev_f32(bias), hb, hf, ws)
    torch.cuda.synchronize()
    h_ref, _ = oracle.lstm_layer(oracle.bf16_bits_to_f64(xb), oracle.bf16_bits_to_f64(wih),
                                 oracle.bf16_bits_to_f64(whh), bias.astype(np.float64), np.zeros(4 * H), round_h=True)
    assert oracle.rel_err(gu.host(hf), h_ref) <= TOL
    assert oracle.rel_err(gu.host(hb), h_ref) <= TOL


@pytest.mark.parametrize("slots,shape", [(1, (50, 32, 512, 1024)), (3, (50, 32, 512, 1024)), (16, (50, 32, 512, 1024)),
                                         (1, (7, 17, 40, 96)), (3, (5, 3, 64, 64)), (16, (6, 17, 72, 1024))])
def test_lstm_layer_on_partitions(env, slots, shape):
    """The layer on CU-masked streams of 8, 24 and 128 CUs: the step launch
    is chosen for the stream's CUs (H = 1024, B = 32: 16 hidden units per
    block on 8 and 24 CUs, 8 on 128, 4 on the whole GPU; the small shapes
    take ragged batches through the wider blocks); same bar as above."""
    ds, gu, inputs, oracle, torch = env
    T, B, I, H = shape
    print("lstm layer %s on %d slots" % (shape, slots), flush=True)
    xb = inputs.normal_bf16(22, (T, B, I))
    a = 1.0 / np.sqrt(H)
    wih = inputs.uniform_bf16(23, (4 * H, I), -a, a)
    whh = inputs.uniform_bf16(24, (4 * H, H), -a, a)
    bias = np.random.default_rng(25).uniform(-2 * a, 2 * a, 4 * H).astype(np.float32)
    hb = gu.empty_bf16((T, B, H))
    hf = gu.empty_f32((T, B, H))
    ws = torch.empty(ds.lstm_workspace_bytes(T, B, H), dtype=torch.uint8, device="cuda:0")
    part = ds.Partition(slot_offset=0, n_slots=slots)
    try:
        ds.lstm_layer(gu.dev_bf16(xb), gu.dev_bf16(wih), gu.dev_bf16(whh), gu.dev_f32(bias), hb, hf, ws,
                      stream=part.stream_ptr)
        part.synchronize()
        h_ref, _ = oracle.lstm_layer(oracle.bf16_bits_to_f64(xb), oracle.bf16_bits_to_f64(wih),
                                     oracle.bf16_bits_to_f64(whh), bias.astype(np.float64), np.zeros(4 * H),
                                     round_h=True)
        err = oracle.rel_err(gu.host(hf), h_ref)
        print("  rel_err %.3e" % err, flush=True)
        assert err <= TOL
        assert oracle.rel_err(gu.host(hb), h_ref) <= TOL
    finally:
        part.destroy()


def test_kernel_argument_errors(env):
    ds, gu, inputs, oracle, torch = env
    x = gu.empty_bf16((1, 4, 4, 12))
    w = gu.empty_bf16((8, 3, 3, 12))
    y = gu.empty_bf16((1, 4, 4, 8))
    with pytest.raises(ds.DStackError) as e:  # C % 8 != 0
        ds.conv2d(x, w, 8, 3, 3, 1, 1, None, None, None, 0, y)
    assert e.value.status == ds.E_UNSUPPORTED
    x3 = gu.empty_bf16((1, 8, 8, 3))
    sc = gu.dev_f32(np.ones(128, np.float32))
    with pytest.raises(ds.DStackError) as e:  # RGB stem with K = 128
        ds.conv2d_rgb(x3, gu.empty_bf16((128, 3, 3, 4)), 128, 3, 1, 1, sc, sc, 0, gu.empty_bf16((1, 8, 8, 128)))
    assert e.value.status == ds.E_UNSUPPORTED
    with pytest.raises(ds.DStackError) as e:  # RGB stem with a 5 x 5 filter
        ds.conv2d_rgb(x3, gu.empty_bf16((16, 5, 5, 4)), 16, 5, 1, 2, sc, sc, 0, gu.empty_bf16((1, 8, 8, 16)))
    assert e.value.status == ds.E_UNSUPPORTED
    with pytest.raises(ds.DStackError) as e:  # expanded channels a multiple of neither 48 nor 64
        ds.expand_dw(gu.empty_bf16((1, 4, 4, 16)), gu.empty_bf16((80, 16)), 80, sc, sc, 2, gu.empty_bf16((3, 3, 80)), 1,
                     sc, sc, 2, gu.empty_bf16((1, 4, 4, 80)))
    assert e.value.status == ds.E_UNSUPPORTED
    xb = gu.empty_bf16((33, 64))
    with pytest.raises(ds.DStackError) as e:  # batch > 32
        ds.fc(xb, gu.empty_bf16((10, 64)), None, 0, gu.empty_f32((33, 10)), out_fp32=True)
    assert e.value.status == ds.E_UNSUPPORTED
