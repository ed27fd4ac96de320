"""Pins for the fp64 numerics oracle (CPU only).

Each test checks the oracle against something other than itself: a library
routine (torch.nn.functional in float64, scipy.signal), a closed form, a
published constant or parameter count, or an invariant that a dropped term,
wrong sign, swapped index or transposed operand would break.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from scipy.signal import correlate2d

from tests.inputs import f32_to_bf16_bits


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))


def _torch_conv_nhwc(x, w, stride, pad, groups=1):
    y = F.conv2d(_t(x).permute(0, 3, 1, 2), _t(w).permute(0, 3, 1, 2), stride=stride, padding=pad, groups=groups)
    return y.permute(0, 2, 3, 1).numpy()


CONV_CASES = [
    # N, H, W, C, K, R, stride, pad
    (1, 5, 5, 1, 1, 3, 1, 1),
    (2, 6, 5, 3, 4, 3, 1, 1),
    (2, 7, 7, 4, 3, 3, 2, 1),
    (1, 6, 6, 2, 5, 1, 1, 0),
    (1, 9, 8, 3, 2, 7, 2, 3),
    (2, 5, 6, 4, 3, 1, 2, 0),
    (1, 4, 4, 2, 2, 3, 1, 0),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv2d_matches_torch(oracle_mod, case):
    N, H, W, C, K, R, st, pad = case
    rng = np.random.default_rng(7)
    x = rng.standard_normal((N, H, W, C))
    w = rng.standard_normal((K, R, R, C))
    y = oracle_mod.conv2d(x, w, st, pad)
    np.testing.assert_allclose(y, _torch_conv_nhwc(x, w, st, pad), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv2d_matches_scipy_correlate(oracle_mod, case):
    """Cross-correlation (no flip) per channel pair, summed, then strided."""
    N, H, W, C, K, R, st, pad = case
    rng = np.random.default_rng(11)
    x = rng.standard_normal((N, H, W, C))
    w = rng.standard_normal((K, R, R, C))
    xp = np.pad(x, ((0, 0), (pad, pad), (pad, pad), (0, 0)))
    ref = np.zeros_like(oracle_mod.conv2d(x, w, st, pad))
    for n in range(N):
        for k in range(K):
            acc = sum(correlate2d(xp[n, :, :, c], w[k, :, :, c], mode="valid") for c in range(C))
            ref[n, :, :, k] = acc[::st, ::st]
    np.testing.assert_allclose(oracle_mod.conv2d(x, w, st, pad), ref, rtol=1e-12, atol=1e-12)


def test_conv2d_identity_kernel(oracle_mod):
    rng = np.random.default_rng(1)
    x = rng.standard_normal((2, 6, 7, 5))
    w = np.zeros((5, 3, 3, 5))
    for c in range(5):
        w[c, 1, 1, c] = 1.0
    np.testing.assert_array_equal(oracle_mod.conv2d(x, w, 1, 1), x)


def test_conv2d_linearity(oracle_mod):
    rng = np.random.default_rng(2)
    x1, x2 = rng.standard_normal((2, 2, 6, 6, 3))
    w = rng.standard_normal((4, 3, 3, 3))
    a, b = 0.75, -1.5
    lhs = oracle_mod.conv2d(a * x1 + b * x2, w, 2, 1)
    rhs = a * oracle_mod.conv2d(x1, w, 2, 1) + b * oracle_mod.conv2d(x2, w, 2, 1)
    np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-12)


def test_conv2d_zero_padding_borders(oracle_mod):
    C = 3
    y = oracle_mod.conv2d(np.ones((1, 5, 6, C)), np.ones((1, 3, 3, C)), 1, 1)[0, :, :, 0]
    assert y[0, 0] == y[0, -1] == y[-1, 0] == y[-1, -1] == 4 * C
    assert np.all(y[0, 1:-1] == 6 * C) and np.all(y[1:-1, 0] == 6 * C)
    assert np.all(y[1:-1, 1:-1] == 9 * C)
    # 7x7 pad 3: the corner sees a 4x4 window, the centre of a 7x7 image the full 7x7
    y7 = oracle_mod.conv2d(np.ones((1, 7, 7, C)), np.ones((1, 7, 7, C)), 1, 3)[0, :, :, 0]
    assert y7[0, 0] == 16 * C and y7[3, 3] == 49 * C and y7[0, 3] == 28 * C


def test_conv2d_output_shape_formula(oracle_mod):
    for H, R, st, pad in [(224, 7, 2, 3), (56, 3, 2, 1), (7, 3, 1, 1), (28, 1, 2, 0), (112, 3, 2, 1)]:
        y = oracle_mod.conv2d(np.zeros((1, H, H, 1)), np.zeros((1, R, R, 1)), st, pad)
        assert y.shape[1] == math.floor((H + 2 * pad - R) / st) + 1


def test_conv1x1_is_matrix_product(oracle_mod):
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 4, 5, 6))
    w = rng.standard_normal((7, 1, 1, 6))
    ref = x.reshape(-1, 6) @ w.reshape(7, 6).T
    np.testing.assert_allclose(oracle_mod.conv2d(x, w, 1, 0).reshape(-1, 7), ref, rtol=1e-12, atol=1e-12)


def test_depthwise_is_block_diagonal_full_conv(oracle_mod):
    rng = np.random.default_rng(4)
    C = 5
    x = rng.standard_normal((2, 7, 6, C))
    wd = rng.standard_normal((C, 3, 3))
    wf = np.zeros((C, 3, 3, C))
    for c in range(C):
        wf[c, :, :, c] = wd[c]
    for st in (1, 2):
        np.testing.assert_allclose(oracle_mod.dwconv(x, wd, st, 1), oracle_mod.conv2d(x, wf, st, 1),
                                   rtol=1e-12, atol=1e-12)
        ref = _torch_conv_nhwc(x, wd[:, :, :, None], st, 1, groups=C)
        np.testing.assert_allclose(oracle_mod.dwconv(x, wd, st, 1), ref, rtol=1e-12, atol=1e-12)


def test_fc_matches_matmul(oracle_mod):
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, 9))
    w = rng.standard_normal((4, 9))
    b = rng.standard_normal(4)
    np.testing.assert_allclose(oracle_mod.fc(x, w, b), F.linear(_t(x), _t(w), _t(b)).numpy(), rtol=1e-12)


def test_pools(oracle_mod):
    ramp = np.arange(1 * 6 * 6 * 2, dtype=np.float64).reshape(1, 6, 6, 2)
    y = oracle_mod.maxpool(ramp, 2, 2, 0)
    # a ramp increasing along h, w and c peaks at the bottom-right cell of each window
    np.testing.assert_array_equal(y, ramp[:, 1::2, 1::2, :])
    rng = np.random.default_rng(6)
    x = -np.abs(rng.standard_normal((2, 7, 7, 3))) - 1.0  # all negative: padding must never win
    ref = F.max_pool2d(_t(x).permute(0, 3, 1, 2), 3, 2, 1).permute(0, 2, 3, 1).numpy()
    np.testing.assert_array_equal(oracle_mod.maxpool(x, 3, 2, 1), ref)
    assert np.all(oracle_mod.maxpool(x, 3, 2, 1) < 0)
    np.testing.assert_array_equal(oracle_mod.avgpool(np.full((2, 7, 7, 3), 2.5)), np.full((2, 3), 2.5))
    np.testing.assert_allclose(oracle_mod.avgpool(x), x.mean(axis=(1, 2)), rtol=1e-14)


def _torch_lstm(x, w_ih, w_hh, b_ih, b_hh):
    I, H = w_ih.shape[1], w_hh.shape[1]
    m = torch.nn.LSTM(I, H, num_layers=1).double()
    with torch.no_grad():
        m.weight_ih_l0.copy_(_t(w_ih))
        m.weight_hh_l0.copy_(_t(w_hh))
        m.bias_ih_l0.copy_(_t(b_ih))
        m.bias_hh_l0.copy_(_t(b_hh))
        out, (h, c) = m(_t(x))
    return out.numpy(), c[0].numpy()


def test_lstm_matches_torch(oracle_mod):
    rng = np.random.default_rng(8)
    T, B, I, H = 6, 3, 5, 4
    x = rng.standard_normal((T, B, I))
    w_ih = rng.standard_normal((4 * H, I)) * 0.5
    w_hh = rng.standard_normal((4 * H, H)) * 0.5
    b_ih, b_hh = rng.standard_normal((2, 4 * H)) * 0.3
    h, c = oracle_mod.lstm_layer(x, w_ih, w_hh, b_ih, b_hh)
    hr, cr = _torch_lstm(x, w_ih, w_hh, b_ih, b_hh)
    np.testing.assert_allclose(h, hr, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(c, cr, rtol=1e-12, atol=1e-13)


def test_lstm_zero_weights(oracle_mod):
    T, B, I, H = 5, 2, 3, 4
    x = np.random.default_rng(9).standard_normal((T, B, I))
    z = np.zeros
    h, c = oracle_mod.lstm_layer(x, z((4 * H, I)), z((4 * H, H)), z(4 * H), z(4 * H))
    assert np.all(h == 0) and np.all(c == 0)
    # zero weights, constant gate biases: c_t = i*g*(1 - f^t)/(1 - f), h_t = o*tanh(c_t)
    bi, bf, bg, bo = 0.3, -0.2, 0.7, 0.1
    b_ih = np.concatenate([np.full(H, v) for v in (bi, bf, bg, bo)])
    b_hh = np.full(4 * H, 0.05)
    h, c = oracle_mod.lstm_layer(x, z((4 * H, I)), z((4 * H, H)), b_ih, b_hh)
    sig = lambda v: 1 / (1 + math.exp(-v))
    i, f, g, o = sig(bi + 0.05), sig(bf + 0.05), math.tanh(bg + 0.05), sig(bo + 0.05)
    for t in range(T):
        ct = i * g * (1 - f ** (t + 1)) / (1 - f)
        np.testing.assert_allclose(h[t], o * math.tanh(ct), rtol=1e-13)
    np.testing.assert_allclose(c, i * g * (1 - f ** T) / (1 - f), rtol=1e-13)


def test_lstm_h_rounding_only_affects_gemm_input(oracle_mod):
    rng = np.random.default_rng(10)
    T, B, I, H = 3, 2, 4, 3
    args = (rng.standard_normal((T, B, I)), rng.standard_normal((4 * H, I)), rng.standard_normal((4 * H, H)),
            rng.standard_normal(4 * H), rng.standard_normal(4 * H))
    h0, _ = oracle_mod.lstm_layer(*args, round_h=False)
    h1, _ = oracle_mod.lstm_layer(*args, round_h=True)
    np.testing.assert_array_equal(h0[0], h1[0])  # step 1 sees h0 = 0 either way
    assert np.max(np.abs(h0 - h1)) < 2e-2


def test_bf16_round_matches_fp32_bit_rounding(oracle_mod):
    rng = np.random.default_rng(12)
    v = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    ref = oracle_mod.bf16_bits_to_f64(f32_to_bf16_bits(v))
    np.testing.assert_array_equal(oracle_mod.bf16_round(v.astype(np.float64)), ref)
    # ties go to even: 1 + 2^-8 is halfway between 1 and 1 + 2^-7
    assert oracle_mod.bf16_round(1 + 2 ** -8) == 1.0
    assert oracle_mod.bf16_round(1 + 3 * 2 ** -8) == 1 + 2 ** -6
    assert oracle_mod.bf16_round(-(1 + 2 ** -8 + 2 ** -30)) == -(1 + 2 ** -7)


def test_splitmix64_published_vector(oracle_mod):
    # first outputs of splitmix64 seeded with 1234567 (Vigna's reference implementation)
    ref = [6457827717110365317, 3203168211198807973, 9817491932198370423, 4593380528125082431,
           16408922859458223821]
    assert [int(v) for v in oracle_mod.splitmix64(1234567, 5)] == ref


# --- architecture pins: parameter totals of the reference architectures ---
# Published totals (torchvision): ResNet-50 25,557,032 and MobileNetV2 3,504,872,
# both including the BN affine pairs (2 per BN channel; 26,560 and 17,056 BN
# channels); VGG-19 143,667,240 (no BN).  nn.LSTM(512, 1024, 2): 4H(I+H)+8H per layer.
PARAMS = {
    "tinycnn": 3 * 9 * 16 + 16 * 9 * 32 + 32 * 9 * 32 + 32 * 9 * 64 + 64 * 10 + 10,
    "resnet50": 25557032 - 2 * 26560,
    "mobilenetv2": 3504872 - 2 * 17056,
    "vgg19": 143667240,
    "lstm2": 4 * 1024 * (512 + 1024) + 8 * 1024 + 4 * 1024 * 2048 + 8 * 1024,
}
NTENSORS = {"tinycnn": 6, "resnet50": 1 + 16 * 3 + 4 + 2, "mobilenetv2": 1 + 17 * 3 - 1 + 1 + 2,
            "vgg19": 38, "lstm2": 8}


@pytest.mark.parametrize("arch", list(PARAMS))
def test_architecture_parameter_counts(oracle_mod, arch):
    m = oracle_mod.Model(arch, 1)
    assert m.num_tensors() == NTENSORS[arch]
    assert sum(m.numel(i) for i in range(m.num_tensors())) == PARAMS[arch]


def test_weight_distributions(oracle_mod):
    m = oracle_mod.Model("resnet50", 1234)
    w = oracle_mod.bf16_bits_to_f64(m.tensor_bf16(0))  # stem 7x7x3 -> 64, fan_in 147
    assert abs(w.std() - math.sqrt(2 / 147)) < 0.05 * math.sqrt(2 / 147)
    assert abs(w.mean()) < 4 * math.sqrt(2 / 147) / math.sqrt(w.size)
    big = oracle_mod.bf16_bits_to_f64(m.tensor_bf16(m.num_tensors() - 2))  # fc 2048 -> 1000
    assert abs(big.std() - math.sqrt(2 / 2048)) < 0.01 * math.sqrt(2 / 2048)
    assert np.all(m.tensor_bf16(m.num_tensors() - 1) == 0)  # fc bias
    lstm = oracle_mod.Model("lstm2", 5)
    u = oracle_mod.bf16_bits_to_f64(lstm.tensor_bf16(1))
    assert u.min() >= -1 / 32 and u.max() <= 1 / 32
    assert abs(u.std() - (1 / 32) / math.sqrt(3)) < 0.01 * (1 / 32)
    # different seeds and different tensor indices give different streams
    m2 = oracle_mod.Model("resnet50", 1235)
    assert not np.array_equal(m.tensor_bf16(0), m2.tensor_bf16(0))


def test_tiny_cnn_zero_weights_give_zero_logits(oracle_mod):
    m = oracle_mod.Model("tinycnn", 3)
    for i in range(m.num_tensors()):
        m.set_tensor(i, np.zeros(m.numel(i)))
    x = f32_to_bf16_bits(np.random.default_rng(0).standard_normal((2, 32, 32, 3)).astype(np.float32))
    assert np.all(m.forward(x) == 0)


def test_tiny_cnn_identity_network_by_hand(oracle_mod):
    """Identity convs (channel c -> c), BN with unit stats, ReLU, 2x2 max pools,
    global mean and an identity FC give: logits[c] = mean over the 8x8 pooled
    grid of the 4x4-block maxima of relu(x_c) scaled by bn^4 (bn = 1/sqrt(1+1e-5))."""
    m = oracle_mod.Model("tinycnn", 3)
    ch = [3, 16, 32, 32, 64]
    for l in range(4):
        w = np.zeros((ch[l + 1], 3, 3, ch[l]))
        for c in range(ch[l]):
            w[c, 1, 1, c] = 1.0
        m.set_tensor(l, w)
    fcw = np.zeros((10, 64))
    for c in range(3):
        fcw[c, c] = 1.0
    m.set_tensor(4, fcw)
    x32 = np.random.default_rng(1).standard_normal((2, 32, 32, 3)).astype(np.float32)
    xb = f32_to_bf16_bits(x32)
    x = oracle_mod.bf16_bits_to_f64(xb)
    bn = 1 / math.sqrt(1 + 1e-5)
    blocks = np.maximum(x, 0).reshape(2, 8, 4, 8, 4, 3).max(axis=(2, 4))
    ref = np.zeros((2, 10))
    ref[:, :3] = blocks.mean(axis=(1, 2)) * bn ** 4
    np.testing.assert_allclose(m.forward(xb, parity=False), ref, rtol=1e-12, atol=1e-15)
