"""Seeded synthetic attention inputs.

This module only draws random numbers and stores them as BF16 bit patterns.
It holds none of the attention arithmetic, so both the HIP path and the
CPU oracle may consume what it produces.

The workloads stand in for the paper's captured layer inputs (Appendix on
accuracy and cost, "Captured inputs": one causal 4096-token sequence, 16
query heads, head dimension 64, scale 1/8), which are not available.  They
reproduce the large common key component of late training: every token's key
row gets the same per-channel bias vector b (one b per batch/head).

Recipe for one (batch b, head h) of a workload with seed s:
  rng = numpy Generator(PCG64(SeedSequence([s, b, h])))
  Q0, K0, V0, U0 = four (N, d) standard normal FP64 draws, in that order
  kb = rng.normal(0, k_bias_std, d); qb = rng.normal(0, q_bias_std, d)
  Q = Q0*q_std + qb;  K = K0 + kb;  V = V0;  dO = U0*do_std
  every tensor is rounded to FP32 (round-to-nearest-even) and then to BF16
  (round-to-nearest-even).
Per-head seeding lets any subset of heads be regenerated on its own.

Grouped-query workloads (Hkv < H) draw every query head as above and give key/value
head j the K and V drawn for query head j*G (G = H / Hkv), the first head of
its group; the other heads' K, V draws are discarded.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

__all__ = [
    "Workload",
    "WORKLOADS",
    "make_inputs",
    "make_head",
    "f32_to_bf16_bits",
    "bf16_bits_to_f32",
    "seeds_for",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    N: int
    d: int
    causal: bool = True
    q_std: float = 1.0
    q_bias_std: float = 0.0
    k_bias_std: float = 0.0
    do_std: float = 1.0
    Hkv: int | None = None  # key/value heads (None: H, multi-head attention)

    @property
    def kv_heads(self) -> int:
        return self.H if self.Hkv is None else self.Hkv

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    def with_shape(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads of the hot-path contract.  Index 2 is the headline one.
WORKLOADS = {
    1: Workload("tiny", 1, 1, 128, 64, k_bias_std=8.0, do_std=1.0),
    2: Workload("h16_n4096_d64", 1, 16, 4096, 64, k_bias_std=4.0, do_std=0.01),
    3: Workload("h16_n4096_d128", 1, 16, 4096, 128, q_bias_std=2.0, k_bias_std=4.0,
                do_std=0.01),
    4: Workload("h16_n16384_d64", 1, 16, 16384, 64, k_bias_std=8.0, do_std=0.01),
    5: Workload("b8_h32_n8192_d128", 8, 32, 8192, 128, k_bias_std=4.0, do_std=0.01),
    # The paper's capture layout: 16 query heads sharing 4 key/value heads.
    6: Workload("gqa_h16kv4_n4096_d64", 1, 16, 4096, 64, k_bias_std=4.0, do_std=0.01, Hkv=4),
}


def seeds_for(index: int, count: int = 8) -> list[int]:
    """Seeds 1000*index + s, s = 0..count-1."""
    return [1000 * index + s for s in range(count)]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to BF16 (nearest, ties to even); return uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    nan = np.isnan(x)
    out = rounded.astype(np.uint16)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen BF16 bit patterns to float32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def _to_bf16(x64: np.ndarray) -> np.ndarray:
    return f32_to_bf16_bits(x64.astype(np.float32))


def make_head(w: Workload, seed: int, b: int, h: int, N: int | None = None):
    """Draw one head; returns uint16 arrays (N, d) for Q, K, V, dO."""
    N = w.N if N is None else N
    d = w.d
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, b, h])))
    q0 = rng.standard_normal((N, d))
    k0 = rng.standard_normal((N, d))
    v0 = rng.standard_normal((N, d))
    u0 = rng.standard_normal((N, d))
    kb = rng.normal(0.0, w.k_bias_std, d) if w.k_bias_std > 0 else np.zeros(d)
    qb = rng.normal(0.0, w.q_bias_std, d) if w.q_bias_std > 0 else np.zeros(d)
    q = q0 * w.q_std + qb[None, :]
    k = k0 + kb[None, :]
    u = u0 * w.do_std
    return _to_bf16(q), _to_bf16(k), _to_bf16(v0), _to_bf16(u)


def make_inputs(w: Workload, seed: int, heads=None, workers: int = 1):
    """Generate a workload as uint16 BF16 bit arrays: q, do [B, H, N, d] and
    k, v [B, Hkv, N, d].

    heads: optional list of (b, h) pairs (multi-head workloads only); if given,
    the arrays are shaped [len(heads), 1, N, d] holding only those heads (same
    values as in the full tensor).
    workers: threads drawing heads concurrently (every head has its own
    generator, so the values do not depend on it).
    """
    Hkv = w.kv_heads
    if heads is not None and Hkv != w.H:
        raise ValueError("head subsets are for multi-head workloads")
    if heads is None:
        pairs = [(b, h) for b in range(w.B) for h in range(w.H)]
        shape = (w.B, w.H, w.N, w.d)
        kv_shape = (w.B, Hkv, w.N, w.d)
    else:
        pairs = list(heads)
        shape = kv_shape = (len(pairs), 1, w.N, w.d)
    G = w.H // Hkv
    out = {n: np.empty(shape, dtype=np.uint16) for n in ("q", "do")}
    out.update({n: np.empty(kv_shape, dtype=np.uint16) for n in ("k", "v")})

    def one(idx):
        b, h = pairs[idx]
        q, k, v, u = make_head(w, seed, b, h)
        bi, hi = divmod(idx, shape[1])
        out["q"][bi, hi] = q
        out["do"][bi, hi] = u
        if heads is not None:
            out["k"][bi, hi] = k
            out["v"][bi, hi] = v
        elif hi % G == 0:
            out["k"][bi, hi // G] = k
            out["v"][bi, hi // G] = v

    if workers > 1 and len(pairs) > 1:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(one, range(len(pairs))))
    else:
        for idx in range(len(pairs)):
            one(idx)
    return out
