"""Device-side placement of the seeded inputs (torch is used for memory only).

The 131072-token decode caches of the decode workload (two [64, 64, cap, 128]
bf16 tensors, about 35 GB) are drawn directly on the device with a seeded
torch generator: N(0,1) float32 draws times the workload scale, rounded to
bf16.  The rows a test needs on the host are copied back from the device
before the layer runs.
"""
from __future__ import annotations

import numpy as np
import torch


def to_device(x: np.ndarray, dtype: str, device) -> torch.Tensor:
    """numpy float32 / bf16-bits (uint16) array -> device tensor."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(x)).to(device)


def fill_normal_(t: torch.Tensor, seed: int, scale: float) -> torch.Tensor:
    """Fill t (any float dtype, [B, ...]) with N(0,1)*scale, one batch row
    at a time, from a generator seeded with ``seed``."""
    g = torch.Generator(device=t.device)
    g.manual_seed(int(seed))
    for b in range(t.shape[0]):
        tmp = torch.empty(t.shape[1:], dtype=torch.float32, device=t.device)
        tmp.normal_(generator=g)
        tmp.mul_(float(scale))
        t[b].copy_(tmp)
        del tmp
    return t


def decode_caches(B: int, H: int, cap: int, d: int, dtype: str, seed: int, scale: float,
                  device) -> tuple:
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    kc = torch.empty(B, H, cap, d, dtype=tdt, device=device)
    vc = torch.empty(B, H, cap, d, dtype=tdt, device=device)
    fill_normal_(kc, seed * 16 + 4, scale)
    fill_normal_(vc, seed * 16 + 5, scale)
    return kc, vc
