"""Moving bf16 bit patterns between numpy (uint16) and torch device tensors.

Pure data movement: bf16 matrices travel as their 16-bit patterns, unchanged."""
from __future__ import annotations

import numpy as np


def bits_to_device(bits: np.ndarray, device: str = "cuda"):
    """uint16 bf16 patterns -> contiguous torch.bfloat16 tensor on `device`."""
    import torch
    a = np.ascontiguousarray(bits, dtype=np.uint16)
    return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)


def device_to_bits(t) -> np.ndarray:
    """torch.bfloat16 tensor -> uint16 bf16 patterns on the host."""
    import torch
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)
