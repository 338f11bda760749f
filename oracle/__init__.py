"""CPU oracle for BF16 attention with the GProj correction.

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` import this package.  The product library
(``paper_2609_34272_amd``) never imports, links or runs anything in here, and
this package shares no code with it.

Contents
  exact(...)            FP64 exact attention forward + VJP (C, OpenMP; also
                        grouped-query attention when k, v have fewer heads
                        than q, key/value gradients summed over each group), the
                        accuracy target: the paper measures errors against the
                        exact VJP in FP64 on the same BF16 inputs (Section 3.2,
                        and the appendix "Reference and metric").
  jacobian_reference    independent FP64 reference with different algebra
                        (uncentered, explicit softmax Jacobian).
  algo_model            step-by-step model of the paper's BF16 forward and
                        Algorithm 1 backward with the implemented rounding
                        points, used for semantics checks (the -24 witness,
                        mode identities) and to predict error magnitudes.
  exact_varlen          exact() over packed variable-length sequences (each
                        sequence its own attention problem).
  rel_l2                the paper's metric: 100 ||G_hat - G64||_2 / ||G64||_2
                        over a full tensor (appendix "Reference and metric").
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import algo_model, jacobian_ref  # noqa: F401
from .jacobian_ref import jacobian_reference  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle_exact.so")
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    dp = ctypes.POINTER(ctypes.c_double)
    lib.oracle_attention_f64.restype = ctypes.c_int
    lib.oracle_attention_f64.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                         ctypes.c_int, ctypes.c_double,
                                         dp, dp, dp, dp, dp, dp, dp, dp, dp, ctypes.c_int]
    lib.oracle_attention_gqa_f64.restype = ctypes.c_int
    lib.oracle_attention_gqa_f64.argtypes = [ctypes.c_int64] * 5 + [ctypes.c_int, ctypes.c_double] \
        + [dp] * 9 + [ctypes.c_int]
    lib.oracle_max_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def widen_bf16(bits) -> np.ndarray:
    """BF16 bit patterns (uint16) -> float64, exactly."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def as_f64(x) -> np.ndarray:
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return widen_bf16(x)
    return np.ascontiguousarray(x, dtype=np.float64)


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def exact(q, k, v, do, causal: bool, scale: float, nthreads: int = 0):
    """Exact FP64 attention forward and VJP.

    q, k, v, do: arrays [..., N, d] (uint16 BF16 bits or floats; any leading
    dims, flattened to heads).  Returns a dict with float64 arrays O, LSE,
    dQ, dK, dV of the matching shapes (LSE without the d axis).  With 4-D
    [B, Hq, N, d] q, do and [B, Hkv, N, d] k, v (Hkv dividing Hq, fewer heads)
    it computes grouped-query attention: query head h reads key/value head
    h // (Hq // Hkv), and dK, dV are shaped like k, v.
    """
    lib = _load()
    Q, K, V, U = (as_f64(t) for t in (q, k, v, do))
    if Q.ndim == 4 and K.ndim == 4 and K.shape[1] != Q.shape[1]:
        return _exact_gqa(lib, Q, K, V, U, causal, scale, nthreads)
    shape = Q.shape
    N, d = shape[-2], shape[-1]
    BH = int(np.prod(shape[:-2])) if len(shape) > 2 else 1
    Q, K, V, U = (np.ascontiguousarray(t.reshape(BH, N, d)) for t in (Q, K, V, U))
    O = np.empty_like(Q)
    LSE = np.empty((BH, N))
    dQ = np.empty_like(Q)
    dK = np.empty_like(Q)
    dV = np.empty_like(Q)
    dp = ctypes.POINTER(ctypes.c_double)
    ptr = lambda a: a.ctypes.data_as(dp)  # noqa: E731
    rc = lib.oracle_attention_f64(BH, N, d, int(bool(causal)), float(scale),
                                  ptr(Q), ptr(K), ptr(V), ptr(U),
                                  ptr(O), ptr(LSE), ptr(dQ), ptr(dK), ptr(dV), int(nthreads))
    if rc != 0:
        raise RuntimeError(f"oracle_attention_f64 failed with code {rc}")
    return dict(O=O.reshape(shape), LSE=LSE.reshape(shape[:-1]), dQ=dQ.reshape(shape),
                dK=dK.reshape(shape), dV=dV.reshape(shape))


def _exact_gqa(lib, Q, K, V, U, causal, scale, nthreads):
    B, Hq, N, d = Q.shape
    Hkv = K.shape[1]
    if K.shape != (B, Hkv, N, d) or V.shape != K.shape or U.shape != Q.shape or Hq % Hkv:
        raise ValueError("grouped-query shapes: q, do [B, Hq, N, d]; k, v [B, Hkv, N, d]")
    Q, K, V, U = (np.ascontiguousarray(t) for t in (Q, K, V, U))
    O = np.empty_like(Q)
    LSE = np.empty((B, Hq, N))
    dQ = np.empty_like(Q)
    dK = np.empty_like(K)
    dV = np.empty_like(K)
    dp = ctypes.POINTER(ctypes.c_double)
    ptr = lambda a: a.ctypes.data_as(dp)  # noqa: E731
    rc = lib.oracle_attention_gqa_f64(B, Hq, Hkv, N, d, int(bool(causal)), float(scale),
                                      ptr(Q), ptr(K), ptr(V), ptr(U), ptr(O), ptr(LSE),
                                      ptr(dQ), ptr(dK), ptr(dV), int(nthreads))
    if rc != 0:
        raise RuntimeError(f"oracle_attention_gqa_f64 failed with code {rc}")
    return dict(O=O, LSE=LSE, dQ=dQ, dK=dK, dV=dV)


def exact_varlen(q, k, v, do, cu_seqlens, causal: bool, scale: float, nthreads: int = 0):
    """Exact FP64 attention over packed sequences.

    q, do: [Hq, total, d]; k, v: [Hkv, total, d] (Hkv dividing Hq); sequence
    s holds tokens cu_seqlens[s] .. cu_seqlens[s+1]-1.  Attention never crosses
    a sequence boundary, so each sequence is its own attention problem
    (Section 3.2 with the support L_i restricted to the query's sequence): this
    slices every sequence out and calls exact() on it.  Returns O, LSE ([Hq,
    total]), dQ, dK, dV shaped like the inputs; rows outside every sequence
    are zero.
    """
    Q, K, V, U = (as_f64(t) for t in (q, k, v, do))
    cu = [int(x) for x in np.asarray(cu_seqlens).ravel()]
    Hq, total, d = Q.shape
    Hkv = K.shape[0]
    if K.shape != (Hkv, total, d) or V.shape != K.shape or U.shape != Q.shape or Hq % Hkv:
        raise ValueError("packed shapes: q, do [Hq, total, d]; k, v [Hkv, total, d]")
    if cu[0] != 0 or cu[-1] != total or any(b < a for a, b in zip(cu, cu[1:])):
        raise ValueError("cu_seqlens must start at 0, end at total and be non-decreasing")
    out = dict(O=np.zeros_like(Q), LSE=np.zeros((Hq, total)), dQ=np.zeros_like(Q),
               dK=np.zeros_like(K), dV=np.zeros_like(K))
    for a, b in zip(cu, cu[1:]):
        if b == a:
            continue
        r = exact(Q[None, :, a:b], K[None, :, a:b], V[None, :, a:b], U[None, :, a:b], causal,
                  scale, nthreads)
        for n in out:
            out[n][:, a:b] = r[n][0]
    return out


def rel_l2(approx, target) -> float:
    """100 * ||approx - target||_2 / ||target||_2 over the whole tensor (percent)."""
    a = np.asarray(approx, dtype=np.float64).ravel()
    t = np.asarray(target, dtype=np.float64).ravel()
    den = np.linalg.norm(t)
    num = np.linalg.norm(a - t)
    if den == 0.0:
        return float("inf") if num > 0 else 0.0
    return float(100.0 * num / den)
