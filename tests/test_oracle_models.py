"""Pins of the oracle's model graphs (CPU only): each architecture is built
a second time from torch library modules in float64 -- nn.Conv2d,
nn.BatchNorm2d in eval mode (gamma 1, beta 0, mean 0, var 1, eps 1e-5),
ReLU / ReLU6, nn.MaxPool2d, adaptive average pooling, nn.Linear, nn.LSTM --
following the textbook definition of the network, loaded with the oracle
generator's bf16 weights (conv weights [K][R][S][C] permuted to torch's
[K][C][R][S], depthwise [C][3][3] to [C][1][3][3]), and run on the same
inputs as the oracle's pure-fp64 forward.  Agreement to 1e-9 (relative,
infinity norm) pins the wiring that parameter counts cannot: where strides
sit (ResNet v1.5 strides the 3x3), the stem max pool, which blocks add a
residual and where the activation falls relative to it, the MobileNetV2
projection without activation, VGG's flatten order (h, w, c) and the
second LSTM layer reading the first layer's h."""
import numpy as np
import pytest
import torch
import torch.nn as nn
import torch.nn.functional as F

import oracle
from tests import inputs

TOL = 1e-9


def weights(arch, seed):
    """The oracle model and its tensors as float64 torch tensors (bf16 values are exact in float64)."""
    m = oracle.Model(arch, seed)
    return m, [torch.from_numpy(m.tensor_bf16(i).view(np.int16)).view(torch.bfloat16).to(torch.float64)
               for i in range(m.num_tensors())]


def conv_w(v, K, R, C):
    return v.reshape(K, R, R, C).permute(0, 3, 1, 2)


class Loader:
    """Hands out the oracle's tensors in order (layer order, weight before bias)."""

    def __init__(self, ws):
        self.ws, self.i = ws, 0

    def next(self):
        v = self.ws[self.i]
        self.i += 1
        return v

    def conv(self, mod):
        K, C, R, _ = mod.weight.shape
        with torch.no_grad():
            mod.weight.copy_(conv_w(self.next(), K, R, C))

    def depthwise(self, mod):
        C = mod.weight.shape[0]
        with torch.no_grad():
            mod.weight.copy_(self.next().reshape(C, 1, 3, 3))

    def linear(self, mod):
        with torch.no_grad():
            mod.weight.copy_(self.next().reshape(mod.weight.shape))
            mod.bias.copy_(self.next())


def bn(c):
    return nn.BatchNorm2d(c, eps=1e-5)  # default init: gamma 1, beta 0, running mean 0, running var 1


def linear(i, o):
    """nn.Linear without its random initialisation (every value is loaded)."""
    return nn.utils.skip_init(nn.Linear, i, o, dtype=torch.float64)


class Bottleneck(nn.Module):
    """ResNet v1.5 bottleneck: 1x1 -> 3x3 (carries the stride) -> 1x1 x4, BN
    after each, ReLU after the first two and after the residual sum."""

    def __init__(self, cin, planes, stride, downsample, stride_on_1x1=False):
        super().__init__()
        s1, s2 = (stride, 1) if stride_on_1x1 else (1, stride)  # v1 (stride on the 1x1) is the planted slip
        self.conv1, self.bn1 = nn.Conv2d(cin, planes, 1, s1, bias=False), bn(planes)
        self.conv2, self.bn2 = nn.Conv2d(planes, planes, 3, s2, 1, bias=False), bn(planes)
        self.conv3, self.bn3 = nn.Conv2d(planes, 4 * planes, 1, bias=False), bn(4 * planes)
        self.down = nn.Sequential(nn.Conv2d(cin, 4 * planes, 1, stride, bias=False), bn(4 * planes)) \
            if downsample else None

    def forward(self, x):
        out = F.relu(self.bn1(self.conv1(x)))
        out = F.relu(self.bn2(self.conv2(out)))
        out = self.bn3(self.conv3(out))
        return F.relu(out + (x if self.down is None else self.down(x)))


def resnet50(ld, stride_on_1x1=False):
    stem = nn.Sequential(nn.Conv2d(3, 64, 7, 2, 3, bias=False), bn(64), nn.ReLU(), nn.MaxPool2d(3, 2, 1))
    ld.conv(stem[0])
    blocks, cin = [], 64
    for n, planes, stride in [(3, 64, 1), (4, 128, 2), (6, 256, 2), (3, 512, 2)]:
        for b in range(n):
            blk = Bottleneck(cin, planes, stride if b == 0 else 1, b == 0, stride_on_1x1)
            ld.conv(blk.conv1)
            ld.conv(blk.conv2)
            ld.conv(blk.conv3)
            if blk.down is not None:
                ld.conv(blk.down[0])
            blocks.append(blk)
            cin = 4 * planes
    fc = linear(2048, 1000)
    ld.linear(fc)
    return nn.Sequential(stem, *blocks, nn.AdaptiveAvgPool2d(1), nn.Flatten(), fc)


class InvertedResidual(nn.Module):
    """MobileNetV2 block: [1x1 expand + BN + ReLU6] -> depthwise 3x3 + BN +
    ReLU6 -> 1x1 projection + BN (linear); identity shortcut when the stride
    is 1 and the widths match."""

    def __init__(self, cin, cout, stride, t, ld):
        super().__init__()
        hid = cin * t
        layers = []
        if t != 1:
            e = nn.Conv2d(cin, hid, 1, bias=False)
            ld.conv(e)
            layers += [e, bn(hid), nn.ReLU6()]
        d = nn.Conv2d(hid, hid, 3, stride, 1, groups=hid, bias=False)
        ld.depthwise(d)
        p = nn.Conv2d(hid, cout, 1, bias=False)
        ld.conv(p)
        layers += [d, bn(hid), nn.ReLU6(), p, bn(cout)]
        self.body = nn.Sequential(*layers)
        self.res = stride == 1 and cin == cout

    def forward(self, x):
        return x + self.body(x) if self.res else self.body(x)


def mobilenetv2(ld):
    stem = nn.Conv2d(3, 32, 3, 2, 1, bias=False)
    ld.conv(stem)
    layers, cin = [stem, bn(32), nn.ReLU6()], 32
    for t, c, n, s in [(1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2), (6, 96, 3, 1), (6, 160, 3, 2),
                       (6, 320, 1, 1)]:
        for i in range(n):
            layers.append(InvertedResidual(cin, c, s if i == 0 else 1, t, ld))
            cin = c
    last = nn.Conv2d(320, 1280, 1, bias=False)
    ld.conv(last)
    fc = linear(1280, 1000)
    ld.linear(fc)
    return nn.Sequential(*layers, last, bn(1280), nn.ReLU6(), nn.AdaptiveAvgPool2d(1), nn.Flatten(), fc)


class FlattenHWC(nn.Module):
    """Flatten of an NCHW tensor in (h, w, c) order (the NHWC reading)."""

    def forward(self, x):
        return x.permute(0, 2, 3, 1).reshape(x.shape[0], -1)


def vgg19(ld):
    layers, cin = [], 3
    for n, c in [(2, 64), (2, 128), (4, 256), (4, 512), (4, 512)]:
        for _ in range(n):
            conv = nn.Conv2d(cin, c, 3, 1, 1)
            ld.conv(conv)
            with torch.no_grad():
                conv.bias.copy_(ld.next())
            layers += [conv, nn.ReLU()]
            cin = c
        layers.append(nn.MaxPool2d(2, 2))
    fcs = [linear(25088, 4096), linear(4096, 4096), linear(4096, 1000)]
    for f in fcs:
        ld.linear(f)
    return nn.Sequential(*layers, FlattenHWC(), fcs[0], nn.ReLU(), fcs[1], nn.ReLU(), fcs[2])


def tinycnn(ld):
    layers, cin = [], 3
    for i, c in enumerate([16, 32, 32, 64]):
        conv = nn.Conv2d(cin, c, 3, 1, 1, bias=False)
        ld.conv(conv)
        layers += [conv, bn(c), nn.ReLU()]
        if i in (1, 3):
            layers.append(nn.MaxPool2d(2, 2))
        cin = c
    fc = linear(64, 10)
    ld.linear(fc)
    return nn.Sequential(*layers, nn.AdaptiveAvgPool2d(1), nn.Flatten(), fc)


BUILDERS = {"resnet50": resnet50, "mobilenetv2": mobilenetv2, "vgg19": vgg19, "tinycnn": tinycnn}


@pytest.mark.parametrize("arch,seed,n,hw", [("resnet50", 501, 2, 224), ("mobilenetv2", 502, 2, 224),
                                            ("vgg19", 503, 2, 224), ("tinycnn", 504, 3, 32)])
def test_cnn_graph_vs_torch_modules(arch, seed, n, hw):
    om, ws = weights(arch, seed)
    ld = Loader(ws)
    net = BUILDERS[arch](ld).double().eval()
    assert ld.i == len(ws), "every oracle tensor is used exactly once"
    xb = inputs.image_batch(seed + 1, n, hw=hw)
    x = torch.tensor(oracle.bf16_bits_to_f64(xb)).permute(0, 3, 1, 2)
    with torch.no_grad():
        ref = net(x).numpy()
    got = om.forward(xb, parity=False)
    err = oracle.rel_err(got, ref)
    print(arch, "pure oracle vs torch modules: rel_err %.3e" % err)
    assert err < TOL
    # the storage points of parity mode move the logits by bf16 rounding only
    # (VGG-19's second pass is skipped: two 20-GFLOP fp64 images already take
    # most of this file's time)
    if arch != "vgg19":
        assert oracle.rel_err(om.forward(xb, parity=True), ref) < 5e-2


def test_lstm2_stack_vs_torch_lstm():
    """Two stacked layers: nn.LSTM(512, 1024, num_layers=2) with the
    oracle's W_ih, W_hh, b_ih, b_hh per layer; output = layer 2's h at every
    step."""
    om, ws = weights("lstm2", 505)
    net = nn.LSTM(512, 1024, num_layers=2).double()
    with torch.no_grad():
        for layer in range(2):
            w_ih, w_hh, b_ih, b_hh = ws[4 * layer: 4 * layer + 4]
            getattr(net, "weight_ih_l%d" % layer).copy_(w_ih.reshape(4096, -1))
            getattr(net, "weight_hh_l%d" % layer).copy_(w_hh.reshape(4096, 1024))
            getattr(net, "bias_ih_l%d" % layer).copy_(b_ih)
            getattr(net, "bias_hh_l%d" % layer).copy_(b_hh)
    xb = inputs.sequence_batch(506, 2)
    with torch.no_grad():
        ref, _ = net(torch.tensor(oracle.bf16_bits_to_f64(xb)))
    got = om.forward(xb, parity=False)
    err = oracle.rel_err(got, ref.numpy())
    print("lstm2 pure oracle vs nn.LSTM: rel_err %.3e" % err)
    assert err < TOL
    assert oracle.rel_err(om.forward(xb, parity=True), ref.numpy()) < 5e-2


def test_planted_wiring_mistakes_are_caught():
    """The comparison is sharp enough to see a wiring slip: the ResNet v1
    placement of the stride (on the first 1x1 instead of the 3x3) or a
    MobileNetV2 block without its residual changes the torch model's output
    far beyond the tolerance, while the oracle stays on the correct one."""
    om, ws = weights("mobilenetv2", 507)
    xb = inputs.image_batch(508, 1)
    x = torch.tensor(oracle.bf16_bits_to_f64(xb)).permute(0, 3, 1, 2)
    net = mobilenetv2(Loader(ws)).double().eval()
    with torch.no_grad():
        ref = net(x).numpy()
        blk = next(m for m in net.modules() if isinstance(m, InvertedResidual) and m.res)
        blk.res = False
        bad = net(x).numpy()
    assert oracle.rel_err(bad, ref) > 1e3 * TOL
    assert oracle.rel_err(om.forward(xb, parity=False), ref) < TOL
    om, ws = weights("resnet50", 509)
    with torch.no_grad():
        good = resnet50(Loader(ws)).double().eval()(x).numpy()
        v1 = resnet50(Loader(ws), stride_on_1x1=True).double().eval()(x).numpy()
    assert oracle.rel_err(v1, good) > 1e3 * TOL
    assert oracle.rel_err(om.forward(xb, parity=False), good) < TOL
