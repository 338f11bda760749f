"""Helpers shared by the GPU tests: host <-> device marshalling of BF16 bit
arrays and the comparison metrics.  (Not a test module.)"""
from __future__ import annotations

import numpy as np
import torch


def to_dev(bits: np.ndarray) -> torch.Tensor:
    """uint16 BF16 bit array -> bf16 tensor on cuda:0 (bit-exact)."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).to("cuda:0")


def to_host(t: torch.Tensor) -> np.ndarray:
    """bf16 / fp32 tensor -> float64 numpy array (exact)."""
    return t.detach().float().cpu().numpy().astype(np.float64)


def bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> uint16 bit array (for bitwise comparisons)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def rel_l2(a, b) -> float:
    a = np.asarray(a, dtype=np.float64).ravel()
    b = np.asarray(b, dtype=np.float64).ravel()
    den = np.linalg.norm(b)
    return float(100.0 * np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a - b))


def log(msg: str):
    print(msg, flush=True)
