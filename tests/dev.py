"""Helpers for the GPU tests: upload the seeded host tensors, download results."""
from __future__ import annotations

import numpy as np
import torch

import dar_inputs as di


def to_dev(t: "di.Tensor", device="cuda"):
    if t is None:
        return None
    if t.dtype == "bf16":
        return torch.from_numpy(t.store.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(t.store).to(device)


def to_host64(x: torch.Tensor) -> np.ndarray:
    return x.detach().float().cpu().numpy().astype(np.float64)


def bf16_bits(x: torch.Tensor) -> np.ndarray:
    assert x.dtype == torch.bfloat16
    return x.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def tol(dtype: str) -> float:
    """Max-abs tolerance on unit-scale data: 1e-4 for fp32 paths, 2e-2 for bf16
    storage with fp32 accumulation."""
    return 1e-4 if dtype == "f32" else 2e-2
