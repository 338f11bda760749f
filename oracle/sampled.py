"""Exact FP64 attention outputs at sampled rows and keys of one long causal head.

TEST INFRASTRUCTURE ONLY (never imported by the product library).

Sequences too long for the full oracle are checked at outputs that each have a
self-contained definition (Section 3.2, support of row i restricted to the
keys j <= i):
  * query row i: O_i, LSE_i and dQ_i need only row i's softmax over its keys;
  * key j of the last few rows' reach: dK_j and dV_j sum over the rows i >= j
    that see key j, and each such row's P_ij, dP_ij - D_i come from that row's
    own softmax.
Scores and values are centered by the head's mean key and mean value (exact:
the softmax ignores a row-constant shift and O moves with a common value
shift, Proposition 3.1), as in the C oracle; the row's LSE adds the shift
alpha q_i . kbar back.  Keys are processed in chunks so memory stays bounded.
"""
from __future__ import annotations

import numpy as np

from . import as_f64

_CHUNK = 1 << 16


def _row(q_i, Kc, Vc, u_i, n, alpha):
    """Softmax and VJP pieces of one row over the first n centered keys:
    returns p (n,), c = u_i . (v_j - o_i) (n,), o_tilde (d_v,), M, log Z."""
    s = np.empty(n)
    for a in range(0, n, _CHUNK):
        b = min(n, a + _CHUNK)
        s[a:b] = alpha * (Kc[a:b] @ q_i)
    M = s.max()
    w = np.exp(s - M)
    Z = w.sum()
    p = w / Z
    ot = np.zeros(Vc.shape[1])
    for a in range(0, n, _CHUNK):
        b = min(n, a + _CHUNK)
        ot += p[a:b] @ Vc[a:b]
    c = np.empty(n)
    for a in range(0, n, _CHUNK):
        b = min(n, a + _CHUNK)
        c[a:b] = (Vc[a:b] - ot) @ u_i
    return p, c, ot, M, np.log(Z)


def exact_rows(q, k, v, do, rows, scale: float):
    """Causal head (q, k, v, do: [N, d], BF16 bits or floats).  For each query
    row in `rows`: O (d), LSE and dQ (d), float64."""
    Q, K, V, U = (as_f64(t) for t in (q, k, v, do))
    kbar, vbar = K.mean(axis=0), V.mean(axis=0)
    Kc, Vc = K - kbar, V - vbar
    out = {"O": [], "LSE": [], "dQ": []}
    for i in rows:
        n = int(i) + 1
        p, c, ot, M, logZ = _row(Q[i], Kc, Vc, U[i], n, scale)
        mu = np.zeros(Kc.shape[1])
        for a in range(0, n, _CHUNK):
            b = min(n, a + _CHUNK)
            mu += p[a:b] @ Kc[a:b]
        g = p * c
        dq = np.zeros(Kc.shape[1])
        for a in range(0, n, _CHUNK):
            b = min(n, a + _CHUNK)
            dq += g[a:b] @ (Kc[a:b] - mu)  # covariance form: sum_j p_j c_j (k_j - mu)
        out["O"].append(vbar + ot)
        out["LSE"].append(scale * float(Q[i] @ kbar) + M + logZ)
        out["dQ"].append(scale * dq)
    return {n: np.array(x) for n, x in out.items()}


def exact_last_keys(q, k, v, do, nkeys: int, scale: float):
    """Causal head: dK and dV ([nkeys, d], float64) of the last nkeys keys,
    summed over the rows i >= j that see key j."""
    Q, K, V, U = (as_f64(t) for t in (q, k, v, do))
    N = Q.shape[0]
    kbar, vbar = K.mean(axis=0), V.mean(axis=0)
    Kc, Vc = K - kbar, V - vbar
    j0 = N - nkeys
    dK = np.zeros((nkeys, Q.shape[1]))
    dV = np.zeros((nkeys, V.shape[1]))
    for i in range(j0, N):
        p, c, _, _, _ = _row(Q[i], Kc, Vc, U[i], i + 1, scale)
        g = p[j0:] * c[j0:]  # keys j0 .. i
        m = i + 1 - j0
        dK[:m] += scale * np.outer(g, Q[i])
        dV[:m] += np.outer(p[j0:], U[i])
    return {"dK": dK, "dV": dV}
