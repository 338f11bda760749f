"""Seeded cases of the synthetic numerical suite.

The paper scores its kernels on a suite of synthetic cases that stress the
layouts and numerical regimes an attention kernel must handle (appendix
"Synthetic Numerical Suite"): packed segments, unequal lengths, singleton and
tile-boundary rows, batch size two, non-causal attention, common key and value
shifts, constant values, sharp attention, zero and tiny upstream gradients and
long sequences, with grouped-query heads and d = 64.  The paper lists the
categories but not its cases; these are this repository's own, one or more per
category, plus d = 128 variants.

Like the rest of this package, this module only draws random numbers and
stores BF16 bit patterns: it holds none of the attention arithmetic.

A case is either dense ([B, H, N, d] tensors) or packed ([H, total, d]
tensors with sequence offsets cu, sequence s = tokens cu[s] .. cu[s+1]-1).
A packed case may give its keys their own lengths (lens_k, offsets cu_k, key
axis of total_k tokens); otherwise the keys share the query lengths.
Every query head h draws, from Generator(PCG64(SeedSequence([seed, index,
h]))), standard normal arrays Q0 (total, d), K0, V0 (total_k, d) and
U0 (total, d) in that order, then
the per-channel biases kb ~ N(0, k_shift^2), vb ~ N(0, v_shift^2) and
qb ~ N(0, q_bias^2) (zero when the spread is 0), then for constant values one
row c ~ N(0, 1):
  Q = q_std * Q0 + qb,  K = K0 + kb,  V = V0 + vb (or every row = c),
  dO = do_std * U0 (all zero when do_std == 0);
each rounded to FP32 and then to BF16, nearest even.  Key/value head j takes
K, V of query head j * G (G = Hq / Hkv).  Dense cases draw the B batches as
one packed axis of B * N tokens and reshape.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from . import f32_to_bf16_bits

__all__ = ["SuiteCase", "CASES", "make_case"]


@dataclasses.dataclass(frozen=True)
class SuiteCase:
    index: int
    name: str
    category: str
    lens: tuple            # packed: sequence lengths; dense: (N,) * B
    packed: bool = True
    causal: bool = True
    Hq: int = 4
    Hkv: int = 2
    d: int = 64
    q_std: float = 1.0
    q_bias: float = 0.0
    k_shift: float = 0.0
    v_shift: float = 0.0
    v_const: bool = False
    do_std: float = 1.0
    lens_k: tuple = ()     # packed only: key lengths when they differ from lens

    @property
    def cross(self) -> bool:
        """Keys have lengths of their own."""
        return len(self.lens_k) > 0

    @property
    def key_lens(self) -> tuple:
        return self.lens_k if self.cross else self.lens

    @property
    def total(self) -> int:
        return int(sum(self.lens))

    @property
    def total_k(self) -> int:
        return int(sum(self.key_lens))

    @property
    def cu(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.lens)]).astype(np.int32)

    @property
    def cu_k(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.key_lens)]).astype(np.int32)

    @property
    def max_seqlen(self) -> int:
        return int(max(self.lens))

    @property
    def max_seqlen_k(self) -> int:
        return int(max(self.key_lens))

    def unseen_keys(self) -> np.ndarray:
        """Boolean [total_k]: keys no query sees (those of sequences without
        queries; with causal the last query of a sequence sees all its keys)."""
        e = np.zeros(self.total_k, dtype=bool)
        for a, nq, nk in zip(self.cu_k[:-1], self.lens, self.key_lens):
            if nq == 0:
                e[a:a + nk] = True
        return e

    def empty_rows(self) -> np.ndarray:
        """Boolean [total]: queries that see no key (no keys in their
        sequence, or, with causal, the first nq - nk queries)."""
        e = np.zeros(self.total, dtype=bool)
        for a, nq, nk in zip(self.cu[:-1], self.lens, self.key_lens):
            if nk == 0:
                e[a:a + nq] = True
            elif self.causal and nq > nk:
                e[a:a + nq - nk] = True
        return e

    @property
    def scale(self) -> float:
        return 1.0 / float(np.sqrt(self.d))


def _cases():
    C = []

    def add(name, category, lens, **kw):
        C.append(SuiteCase(len(C), name, category, tuple(int(x) for x in lens), **kw))

    add("singleton", "singleton", (1,), packed=False)
    add("packed four segments", "packed", (37, 64, 100, 27))
    add("packed two full tiles", "packed", (128, 128))
    add("packed singleton and long", "packed", (1, 200, 55))
    add("packed twenty short", "packed", (5,) * 20)
    add("unequal lengths 17/300", "unequal", (17, 300))
    add("unequal lengths around a tile", "unequal", (64, 65, 63))
    add("unequal lengths around two tiles", "unequal", (127, 128, 129))
    add("unequal lengths mixed", "unequal", (250, 3, 90, 1))
    add("unequal lengths halving", "unequal", (512, 256, 128))
    add("singleton sequences", "singleton", (1, 1, 1, 1))
    add("singletons between tile edges", "tile boundary", (1, 63, 1, 64, 1, 65))
    add("whole tiles", "tile boundary", (64,) * 4)
    add("tile plus one, tile minus one", "tile boundary", (65, 127))
    add("empty sequences", "empty", (0, 40, 0, 17, 0))
    add("empty around a singleton", "empty", (0, 1, 0))
    add("batch two", "batch", (200, 200), packed=False)
    add("batch two, one tile", "batch", (64, 64), packed=False)
    add("non-causal dense", "non-causal", (150,), packed=False, causal=False)
    add("non-causal packed", "non-causal", (40, 90, 7), causal=False)
    add("non-causal one tile", "non-causal", (64,), packed=False, causal=False)
    add("non-causal ragged", "non-causal", (257,), packed=False, causal=False)
    add("key shift 8", "key shift", (256,), packed=False, k_shift=8.0)
    add("key shift 64", "key shift", (256,), packed=False, k_shift=64.0)
    add("key shift 512", "key shift", (256,), packed=False, k_shift=512.0)
    add("key shift 32 packed", "key shift", (100, 156), k_shift=32.0)
    add("key shift 64 non-causal", "key shift", (200,), packed=False, causal=False, k_shift=64.0)
    add("key shift 16 with query bias", "key shift", (300,), packed=False, k_shift=16.0, q_bias=2.0)
    add("value shift 64", "value shift", (256,), packed=False, v_shift=64.0)
    add("value shift 1024", "value shift", (256,), packed=False, v_shift=1024.0)
    add("value shift packed", "value shift", (90, 60), v_shift=256.0)
    add("constant values", "constant values", (100,), packed=False, v_const=True)
    add("constant values packed", "constant values", (30, 50), v_const=True)
    add("constant values non-causal", "constant values", (70,), packed=False, causal=False,
        v_const=True)
    add("sharp attention std 10", "sharp", (256,), packed=False, q_std=10.0)
    add("sharp attention std 30", "sharp", (256,), packed=False, q_std=30.0)
    add("sharp attention with key shift", "sharp", (256,), packed=False, q_std=10.0, k_shift=16.0)
    add("large logits std 100", "sharp", (128,), packed=False, q_std=100.0)
    add("zero upstream", "zero upstream", (200,), packed=False, do_std=0.0)
    add("zero upstream packed", "zero upstream", (50, 80), do_std=0.0)
    add("tiny upstream 1e-4", "tiny upstream", (200,), packed=False, do_std=1e-4)
    add("tiny upstream 1e-6", "tiny upstream", (200,), packed=False, do_std=1e-6)
    add("tiny upstream with key shift", "tiny upstream", (200,), packed=False, do_std=1e-5,
        k_shift=32.0)
    add("multi-head", "heads", (300,), packed=False, Hq=4, Hkv=4)
    add("one key/value head", "heads", (300,), packed=False, Hq=8, Hkv=1)
    add("capture-like 16/4 heads", "heads", (1024,), packed=False, Hq=16, Hkv=4, k_shift=4.0,
        do_std=0.01)
    add("four 4096-token sequences", "long", (4096,) * 4, Hq=4, Hkv=2, k_shift=4.0, do_std=0.01)
    add("4096 and short packed", "long", (4096, 33, 1000), Hq=4, Hkv=2, k_shift=8.0, do_std=0.01)
    add("d128 packed", "head dim 128", (100, 200), d=128)
    add("d128 unequal around tiles", "head dim 128", (63, 64, 65, 1), d=128)
    add("d128 non-causal", "head dim 128", (150,), packed=False, causal=False, d=128)
    add("d128 key shift", "head dim 128", (300,), packed=False, d=128, k_shift=64.0)
    add("d128 constant values", "head dim 128", (80,), packed=False, d=128, v_const=True)
    add("d128 sharp", "head dim 128", (256,), packed=False, d=128, q_std=20.0)
    # Queries and keys of unequal lengths in one sequence (the causal diagonal
    # aligned at the last query and key): fewer queries than keys, more
    # queries than keys (leading queries see no key), sequences without keys.
    add("fewer queries than keys", "unequal query/key", (30, 100, 64), lens_k=(100, 130, 64))
    add("fewer queries, tile-aligned offset", "unequal query/key", (64, 100),
        lens_k=(192, 228))
    add("more queries than keys", "unequal query/key", (100, 70, 130), lens_k=(40, 70, 2))
    add("sequences without keys", "unequal query/key", (20, 50, 5), lens_k=(0, 80, 0))
    add("single queries on long keys", "unequal query/key", (1, 1, 1, 1),
        lens_k=(500, 64, 1, 129))
    add("non-causal unequal query/key", "unequal query/key", (50, 200, 3), causal=False,
        lens_k=(300, 17, 64))
    add("whole query tiles without keys", "unequal query/key", (200,), lens_k=(10,))
    add("d128 unequal query/key", "unequal query/key", (100, 33), d=128, lens_k=(37, 200))
    add("d128 fewer queries, tile-aligned offset", "unequal query/key", (64, 40), d=128,
        lens_k=(128, 104))
    add("non-causal sequence without keys", "unequal query/key", (10, 20), causal=False,
        lens_k=(30, 0))
    add("sequence without queries", "unequal query/key", (0, 30, 7), lens_k=(50, 30, 70))
    return C


CASES = _cases()


def make_case(case: SuiteCase, seed: int = 7000):
    """BF16 bit arrays of one case: q, do [Hq, total, d] and k, v [Hkv,
    total_k, d] on the packed axis (dense cases: B consecutive blocks of N
    tokens)."""
    T, Tk, d, Hq, Hkv = case.total, case.total_k, case.d, case.Hq, case.Hkv
    G = Hq // Hkv
    out = {"q": np.empty((Hq, T, d), np.uint16), "do": np.empty((Hq, T, d), np.uint16),
           "k": np.empty((Hkv, Tk, d), np.uint16), "v": np.empty((Hkv, Tk, d), np.uint16)}
    for h in range(Hq):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, case.index, h])))
        q0, k0, v0, u0 = (rng.standard_normal((n, d)) for n in (T, Tk, Tk, T))
        kb = rng.normal(0.0, case.k_shift, d) if case.k_shift > 0 else np.zeros(d)
        vb = rng.normal(0.0, case.v_shift, d) if case.v_shift > 0 else np.zeros(d)
        qb = rng.normal(0.0, case.q_bias, d) if case.q_bias > 0 else np.zeros(d)
        crow = rng.standard_normal(d)
        q = case.q_std * q0 + qb[None, :]
        k = k0 + kb[None, :]
        v = np.broadcast_to(crow, (Tk, d)) if case.v_const else v0 + vb[None, :]
        u = case.do_std * u0 if case.do_std > 0 else np.zeros((T, d))
        out["q"][h] = f32_to_bf16_bits(q.astype(np.float32))
        out["do"][h] = f32_to_bf16_bits(u.astype(np.float32))
        if h % G == 0:
            out["k"][h // G] = f32_to_bf16_bits(k.astype(np.float32))
            out["v"][h // G] = f32_to_bf16_bits(np.ascontiguousarray(v).astype(np.float32))
    return out
