"""Helpers for the GPU parity tests: moving the generator's arrays to the
device with their exact bits, and comparing against the oracle."""
from __future__ import annotations

import sys

import numpy as np
import torch

DEV = torch.device("cuda:0")


def say(*a):
    """Flush a line naming the case before each GPU step."""
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(x: np.ndarray) -> torch.Tensor:
    """numpy -> device tensor with identical bits; uint16 arrays are bf16."""
    x = np.ascontiguousarray(x)
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(x).to(DEV)


def to_host(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def max_abs(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b))) if a.size else 0.0


def tol_for(kv_dtype: str) -> float:
    """Acceptance bound for attention outputs: 1e-5 max-abs with fp32 K/V,
    2e-3 with bf16 K/V (fp32 accumulation vs an fp64 oracle on the same
    bf16 values)."""
    return 1e-5 if kv_dtype == "f32" else 2e-3
