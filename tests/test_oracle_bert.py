"""Pins for the oracle's transformer pieces (CPU only): layer norm against
torch's F.layer_norm, attention against torch's scaled_dot_product_attention
and two closed forms (equal keys give the mean of the values; one dominant
key selects its value), and the whole BERT forward (pure fp64) against a
model assembled from torch library modules -- embeddings + F.layer_norm,
twelve nn.TransformerEncoderLayer (post-norm, erf GELU, eps 1e-12), tanh
pooler, linear classifier -- carrying the oracle generator's weights."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


def test_layernorm_vs_torch():
    rng = np.random.default_rng(3)
    for rows, C in [(1, 768), (7, 768), (5, 33)]:
        x = rng.normal(0, 2, (rows, C)) + rng.normal(0, 5, (rows, 1))
        g, b = rng.normal(1, 0.3, C), rng.normal(0, 0.3, C)
        ref = F.layer_norm(torch.tensor(x), (C,), torch.tensor(g), torch.tensor(b), 1e-12).numpy()
        assert np.max(np.abs(oracle.layernorm(x, g, b, 1e-12) - ref)) < 1e-12


def test_attention_vs_torch_sdpa():
    rng = np.random.default_rng(4)
    for B, T, heads, dh in [(2, 20, 12, 64), (1, 40, 12, 64), (3, 1, 2, 8), (1, 7, 3, 16)]:
        qkv = rng.normal(0, 1, (B, T, 3 * heads * dh))
        q, k, v = (torch.tensor(qkv[:, :, i * heads * dh:(i + 1) * heads * dh]).view(B, T, heads, dh).transpose(1, 2)
                   for i in range(3))
        ref = F.scaled_dot_product_attention(q, k, v).transpose(1, 2).reshape(B, T, heads * dh).numpy()
        assert np.max(np.abs(oracle.attention(qkv, heads) - ref)) < 1e-12


def test_attention_closed_forms():
    rng = np.random.default_rng(5)
    T, dh = 6, 8
    v = rng.normal(0, 1, (T, dh))
    # every key equal: uniform weights, each output is the mean of the values
    qkv = np.concatenate([rng.normal(0, 1, (T, dh)), np.tile(rng.normal(0, 1, (1, dh)), (T, 1)), v], 1)[None]
    assert np.max(np.abs(oracle.attention(qkv, 1)[0] - v.mean(0))) < 1e-12
    # one key aligned with a huge query: its value is selected
    q = np.zeros((T, dh)); q[:, 0] = 1e3
    k = np.zeros((T, dh)); k[2, 0] = 1.0
    out = oracle.attention(np.concatenate([q, k, v], 1)[None], 1)[0]
    assert np.max(np.abs(out - v[2])) < 1e-12


@pytest.mark.parametrize("arch,T", [("bert", 20), ("bert_long", 40)])
def test_bert_forward_vs_torch_modules(arch, T):
    m = oracle.Model(arch, 11)
    w = [oracle.bf16_bits_to_f64(m.tensor_bf16(i)) for i in range(m.num_tensors())]
    H, FF, L = 768, 3072, 12
    ids = np.random.default_rng(6).integers(0, 30522, (2, T)).astype(np.int32)
    t = lambda a, *shape: torch.tensor(a, dtype=torch.float64).view(*shape)
    with torch.no_grad():
        x = t(w[0], 30522, H)[torch.tensor(ids, dtype=torch.long)] + t(w[1], 512, H)[:T][None] + t(w[2], 2, H)[0]
        x = F.layer_norm(x, (H,), eps=1e-12)
        for l in range(L):
            wq, bq, wo, bo, w1, b1, w2, b2 = w[3 + 8 * l: 11 + 8 * l]
            layer = torch.nn.TransformerEncoderLayer(H, 12, FF, dropout=0.0, activation="gelu", layer_norm_eps=1e-12,
                                                     batch_first=True, norm_first=False).double().eval()
            layer.self_attn.in_proj_weight.copy_(t(wq, 3 * H, H))
            layer.self_attn.in_proj_bias.copy_(t(bq, 3 * H))
            layer.self_attn.out_proj.weight.copy_(t(wo, H, H))
            layer.self_attn.out_proj.bias.copy_(t(bo, H))
            layer.linear1.weight.copy_(t(w1, FF, H))
            layer.linear1.bias.copy_(t(b1, FF))
            layer.linear2.weight.copy_(t(w2, H, FF))
            layer.linear2.bias.copy_(t(b2, H))
            x = layer(x)
        wp, bp, wc, bc = w[3 + 8 * L:]
        pooled = torch.tanh(F.linear(x[:, 0], t(wp, H, H), t(bp, H)))
        ref = F.linear(pooled, t(wc, 2, H), t(bc, 2)).numpy()
    got = m.forward(ids, parity=False)
    assert np.max(np.abs(got - ref)) < 1e-9 * max(1.0, np.max(np.abs(ref)))
    # the encoder's final hidden states too, and layer by layer the same chain
    assert oracle.rel_err(oracle.bert_hidden(m, ids, parity=False), x.numpy()) < 1e-9
    h = oracle.bert_hidden(m, ids, parity=True, layers=0)
    for l in range(1, L + 1):
        h = oracle.bert_layer(m, l, h, parity=True)
    assert np.array_equal(h, oracle.bert_hidden(m, ids, parity=True))
    # parity mode stays within bf16 storage error of the pure result
    assert oracle.rel_err(m.forward(ids, parity=True), ref) < 5e-2
