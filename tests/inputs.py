"""Seeded synthetic inputs shared by the oracle side and the GPU side of the tests.

Holds none of the method's arithmetic: it only draws random tensors and
arrival times (numpy's PCG64 generator) and packs them as bf16 bit patterns.
Stand-ins for the paper's ImageNet images (224x224x3) and IMDB-style token
sequences: N(0, 1) values of the same shapes.
"""
import numpy as np


def f32_to_bf16_bits(x):
    """float32 -> bf16 bit patterns, round-to-nearest-even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = ((u >> 16) & 1) + 0x7FFF
    return ((u + r) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b):
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def normal_bf16(seed, shape, scale=1.0):
    """N(0, scale^2) values as bf16 bit patterns."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(scale)
    return f32_to_bf16_bits(x)


def uniform_bf16(seed, shape, lo, hi):
    rng = np.random.default_rng(seed)
    return f32_to_bf16_bits(rng.uniform(lo, hi, size=shape).astype(np.float32))


def image_batch(seed, batch, hw=224):
    """[b, hw, hw, 3] bf16 NHWC image stand-in."""
    return normal_bf16(seed, (batch, hw, hw, 3))


def sequence_batch(seed, batch, T=50, I=512):
    """[T, b, I] bf16 sequence stand-in (sequence-major)."""
    return normal_bf16(seed, (T, batch, I))


def poisson_arrivals(seed, rate_per_s, duration_us):
    """Sorted integer-us arrival times of a Poisson process on [0, duration)."""
    rng = np.random.default_rng(seed)
    out, t = [], 0.0
    while True:
        t += rng.exponential(1e6 / rate_per_s)
        if t >= duration_us:
            return out
        out.append(int(t))
