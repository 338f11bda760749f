"""Second, independent FP64 reference: explicit softmax-Jacobian VJP.

TEST INFRASTRUCTURE ONLY (never imported by the product library).

The paper cross-checks its centered VJP with "an independent FP64
implementation (explicit softmax Jacobian, 128-query chunks)" (appendix on
accuracy and cost, "Reference and metric"; synthetic-suite appendix,
"References").  This module is that second reference, written with different
algebra from the C oracle: scores and values are NOT centered, and each row's
score gradient is the softmax Jacobian applied to dP,
    J_i = diag(p_i) - p_i p_i^T,   ds_i = J_i (U_i V^T)
formed as an explicit matrix when the row support is small, and in the
equivalent factored form p*(dp - p.dp) otherwise.  Then
    dQ = alpha dS K,  dK = alpha dS^T Q,  dV = P^T U,  O = P V,
    LSE = max + log(sum exp(s - max)).
"""
from __future__ import annotations

import numpy as np


def jacobian_reference(q, k, v, u, causal: bool, alpha: float, chunk: int = 128,
                       explicit_max_support: int = 512):
    """One head; q, k, v, u float64 arrays (N, d).  Returns O, LSE, dQ, dK, dV."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    N, d = q.shape
    O = np.zeros((N, v.shape[1]))
    LSE = np.zeros(N)
    dQ = np.zeros((N, d))
    dK = np.zeros((N, d))
    dV = np.zeros((N, v.shape[1]))
    for r0 in range(0, N, chunk):
        r1 = min(N, r0 + chunk)
        S = alpha * (q[r0:r1] @ k.T)
        if causal:
            rows = np.arange(r0, r1)[:, None]
            cols = np.arange(N)[None, :]
            S = np.where(cols <= rows, S, -np.inf)
        m = S.max(axis=1, keepdims=True)
        E = np.exp(S - m)
        Z = E.sum(axis=1, keepdims=True)
        P = E / Z
        O[r0:r1] = P @ v
        LSE[r0:r1] = m[:, 0] + np.log(Z[:, 0])
        dP = u[r0:r1] @ v.T
        dS = np.zeros_like(P)
        for ii in range(r1 - r0):
            i = r0 + ii
            L = (i + 1) if causal else N
            p = P[ii, :L]
            dp = dP[ii, :L]
            if L <= explicit_max_support:
                J = np.diag(p) - np.outer(p, p)
                dS[ii, :L] = J @ dp
            else:
                dS[ii, :L] = p * dp - p * np.dot(p, dp)
        dQ[r0:r1] = alpha * (dS @ k)
        dK += alpha * (dS.T @ q[r0:r1])
        dV += P.T @ u[r0:r1]
    return O, LSE, dQ, dK, dV
