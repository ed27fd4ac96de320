"""Device-tensor helpers for the GPU tests (marshalling only)."""
import numpy as np
import torch


def dev_bf16(bits):
    """uint16 bf16 bit patterns (numpy) -> bfloat16 tensor on cuda:0."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).to("cuda:0")


def dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda:0")


def host(t):
    """Device tensor -> float64 numpy (bf16 values are exact in float64)."""
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def empty_bf16(shape):
    return torch.empty(shape, dtype=torch.bfloat16, device="cuda:0")


def empty_f32(shape):
    return torch.empty(shape, dtype=torch.float32, device="cuda:0")
