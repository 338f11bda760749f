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
                        sequence its own attention problem; separate query
                        and key lengths with the causal diagonal aligned at
                        the end, empty rows).
  sampled               exact rows (O, LSE, dQ) and last keys (dK, dV) of one
                        long causal head, each from its own row softmaxes, for
                        sizes the full oracle cannot take.
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


def exact_varlen(q, k, v, do, cu_seqlens, causal: bool, scale: float, nthreads: int = 0,
                 cu_seqlens_k=None):
    """Exact FP64 attention over packed sequences.

    q, do: [Hq, total_q, d]; k, v: [Hkv, total_k, d] (Hkv dividing Hq).
    Sequence s holds queries cu_seqlens[s] .. cu_seqlens[s+1]-1 and keys
    cu_seqlens_k[s] .. cu_seqlens_k[s+1]-1 (the same offsets when
    cu_seqlens_k is None).  Attention never crosses a sequence boundary.  With
    causal, query i of a sequence with nq queries and nk keys sees key j iff
    j <= i + (nk - nq) (the causal diagonal aligned at the last query and key);
    a query that sees no key is empty: its O and dQ are 0 and its LSE is +inf.

    Each sequence is reduced to square problems of exact() (Section 3.2 with
    the support restricted to the visible keys): with causal, the queries are
    padded at the top with nk - nq rows of zero upstream gradient (or, when
    nq > nk, the first nq - nk rows are the empty ones); without, the queries
    are cut into chunks of nk rows (zero-gradient padding in the last).  Padding
    rows have u = 0, so they contribute exactly 0 to dK and dV.  Returns O, LSE
    ([Hq, total_q]), dQ, dK, dV shaped like the inputs.
    """
    Q, K, V, U = (as_f64(t) for t in (q, k, v, do))
    cq = [int(x) for x in np.asarray(cu_seqlens).ravel()]
    ck = cq if cu_seqlens_k is None else [int(x) for x in np.asarray(cu_seqlens_k).ravel()]
    Hq, tq, d = Q.shape
    Hkv, tk = K.shape[0], K.shape[1]
    if K.shape != (Hkv, tk, d) or V.shape != K.shape or U.shape != Q.shape or Hq % Hkv:
        raise ValueError("packed shapes: q, do [Hq, total_q, d]; k, v [Hkv, total_k, d]")
    for cu, tot in ((cq, tq), (ck, tk)):
        if cu[0] != 0 or cu[-1] != tot or any(b < a for a, b in zip(cu, cu[1:])):
            raise ValueError("offsets must start at 0, end at the total and be non-decreasing")
    if len(cq) != len(ck):
        raise ValueError("query and key offsets must describe the same number of sequences")
    out = dict(O=np.zeros_like(Q), LSE=np.full((Hq, tq), np.inf), dQ=np.zeros_like(Q),
               dK=np.zeros_like(K), dV=np.zeros_like(K))

    def square(qs, us, ks, vs, causal_):
        r = exact(qs[None], ks[None], vs[None], us[None], causal_, scale, nthreads)
        return {n: r[n][0] for n in r}

    for s in range(len(cq) - 1):
        a, b, ka, kb = cq[s], cq[s + 1], ck[s], ck[s + 1]
        nq, nk = b - a, kb - ka
        if nq == 0 or nk == 0:
            continue
        Qs, Us, Ks, Vs = Q[:, a:b], U[:, a:b], K[:, ka:kb], V[:, ka:kb]
        if causal:
            if nq <= nk:
                pad = nk - nq
                zq = np.zeros((Hq, pad, d))
                r = square(np.concatenate([zq, Qs], 1), np.concatenate([zq, Us], 1), Ks, Vs, True)
                rows = slice(pad, nk)
                out["O"][:, a:b], out["LSE"][:, a:b], out["dQ"][:, a:b] = (
                    r["O"][:, rows], r["LSE"][:, rows], r["dQ"][:, rows])
            else:
                first = a + (nq - nk)  # rows before it see no key
                r = square(Q[:, first:b], U[:, first:b], Ks, Vs, True)
                out["O"][:, first:b], out["LSE"][:, first:b], out["dQ"][:, first:b] = (
                    r["O"], r["LSE"], r["dQ"])
            out["dK"][:, ka:kb] += r["dK"]
            out["dV"][:, ka:kb] += r["dV"]
        else:
            for c0 in range(0, nq, nk):
                c1 = min(nq, c0 + nk)
                pad = nk - (c1 - c0)
                zq = np.zeros((Hq, pad, d))
                r = square(np.concatenate([Qs[:, c0:c1], zq], 1), np.concatenate([Us[:, c0:c1], zq], 1),
                           Ks, Vs, False)
                rows = slice(0, c1 - c0)
                out["O"][:, a + c0:a + c1], out["LSE"][:, a + c0:a + c1], out["dQ"][:, a + c0:a + c1] = (
                    r["O"][:, rows], r["LSE"][:, rows], r["dQ"][:, rows])
                out["dK"][:, ka:kb] += r["dK"]
                out["dV"][:, ka:kb] += r["dV"]
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
