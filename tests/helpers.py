"""Small conversions shared by the tests (raw element bits <-> float64)."""
import numpy as np
import torch


def to_bits(x, dtype):
    """float array -> stored bits (float32 for fp32, uint16 for fp16/bf16), round-to-nearest."""
    t = torch.as_tensor(np.asarray(x, np.float64))
    if dtype == "fp32":
        return t.to(torch.float32).numpy()
    td = torch.bfloat16 if dtype == "bf16" else torch.float16
    return t.to(torch.float32).to(td).view(torch.int16).numpy().view(np.uint16)


def from_bits(a, dtype):
    """stored bits -> float64 array (exact)."""
    a = np.asarray(a)
    if dtype == "fp32":
        return a.astype(np.float64)
    td = torch.bfloat16 if dtype == "bf16" else torch.float16
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(td).to(torch.float64).numpy()


def rng(seed):
    return np.random.default_rng(seed)
