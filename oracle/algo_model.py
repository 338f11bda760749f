"""Scalar model of the paper's BF16 forward and backward (GProj and its ablations).

TEST INFRASTRUCTURE ONLY (never imported by the product library).

This follows the paper's Algorithm 1 (backward with the GProj additions) and
the implemented-arithmetic equations of the appendix "Implemented Arithmetic
and Rounding" step by step, in their notation, for one head:

  forward (eq. gproj-forward, FA3-SBS):
      x_ij  = computed unscaled logit q_i.k_j (FP32)
      z_ij  = exp2_32( fl32[ sub32(x_ij, x_i,max) * (alpha log2 e) ] )
      l_i   = sum_j z_ij,   O_i = BF16( sum_j BF16(z_ij) v_j / l_i )
      LSE_i = alpha x_i,max + ln l_i       (natural-log units)
  backward (Algorithm 1; eqs. gproj-row-mass, gproj-accumulators,
  gproj-query-implemented, gproj-key-implemented):
      D_i   = rowsum(dO_i * O_i)                              (FP32)
      P_ij  = exp(alpha x_ij - LSE_i)    (masked), computed as exp2
      r_ij  = BF16(P_ij)
      t_ij  = BF16( fl32[ P_ij (dP_ij - D_i) ] ),  dP = dO V^T
      rho_i = sum_j t_ij,   m_i = sum_j r_ij
      A_i   = sum_j t_ij k_j,   B_i = sum_j r_ij k_j          (FP32 accumulators)
      lambda_i = rho_i / m_i, or 0 where m_i = 0
      dq_i  = BF16( fl32[ alpha (A_i - lambda_i B_i) ] )     (gproj_q, gproj)
            = BF16( fl32[ alpha A_i ] )                       (plain)
      dV_j  = BF16( sum_i r_ij dO_i )
      dK^acc_j = sum_i t_ij q_i
      z_i   = BF16( lambda_i q_i ),   C_j = sum_i r_ij z_i
      dk_j  = BF16( fl32[ alpha (dK^acc_j - C_j) ] )          (gproj)
            = BF16( fl32[ alpha dK^acc_j ] )                  (plain, gproj_q)

Modelling choices (where the paper leaves freedom):
  * every FP32 accumulation (matrix products, row sums) is modelled as the
    exact sum rounded once to FP32 -- the paper calls m and rho "exact sums of
    the formed operands, which the kernel approximates in FP32";
  * the forward uses the final row maximum (a kernel's running maximum differs
    only by FP32 rounding of the rescale factors);
  * P uses one rounding of x*(alpha log2 e) - LSE*log2 e before exp2 (a fused
    multiply-add; the backward's probability formula is the native one and the
    paper fixes no rounding for it);
  * the key pass's r~ equals r and its lambda equals the query pass's lambda
    (the paper allows them to differ; here they are formed identically).
With rounding=False every cast is the identity and all arithmetic is FP64; the
model then equals the exact VJP (rho = 0 up to FP64 rounding).
"""
from __future__ import annotations

import numpy as np

LOG2E = 1.4426950408889634
MODES = ("plain", "gproj_q", "gproj")


def bf16_round(x):
    """Round float32 values to the nearest BF16 value (ties to even); float32 out."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    bits = x.view(np.uint32).astype(np.uint64)
    lsb = (bits >> np.uint64(16)) & np.uint64(1)
    r = ((bits + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    out = r.astype(np.uint32).view(np.float32).copy()
    nan = np.isnan(x)
    out[nan] = np.nan
    return out


class _Arith:
    """FP32/BF16 rounding helpers; identity in exact (rounding=False) mode."""

    def __init__(self, rounding: bool):
        self.rounding = rounding
        self.dt = np.float32 if rounding else np.float64

    def f32(self, x):
        return np.asarray(x, dtype=np.float64).astype(self.dt) if self.rounding else np.asarray(x, dtype=np.float64)

    def bf16(self, x):
        return bf16_round(x) if self.rounding else np.asarray(x, dtype=np.float64)

    def c(self, v):
        return self.dt(v)

    def exp2(self, x):
        return np.exp2(x.astype(self.dt))

    def log(self, x):
        return np.log(x.astype(self.dt))

    @staticmethod
    def wide(x):
        return np.asarray(x, dtype=np.float64)


def _mask(N: int, causal: bool):
    if not causal:
        return np.ones((N, N), dtype=bool)
    return np.tril(np.ones((N, N), dtype=bool))


def sbs_forward(q, k, v, causal: bool, alpha: float, rounding: bool = True):
    """FA3-SBS forward for one head (eq. gproj-forward).  Returns O, LSE, x."""
    ar = _Arith(rounding)
    W = ar.wide
    N = q.shape[0]
    a = ar.c(alpha)
    c = ar.c(a * ar.c(LOG2E))
    x = ar.f32(W(q) @ W(k).T)
    mask = _mask(N, causal)
    x = np.where(mask, x, -np.inf).astype(ar.dt)
    xmax = x.max(axis=1, keepdims=True)
    with np.errstate(invalid="ignore"):
        diff = (x - xmax).astype(ar.dt)             # sub32
        arg = (diff * c).astype(ar.dt)              # fl32[ . * (alpha log2 e)]
    z = np.where(mask, ar.exp2(arg), 0).astype(ar.dt)
    l = ar.f32(W(z).sum(axis=1))
    num = ar.f32(W(ar.bf16(z)) @ W(v))
    O = ar.bf16((num / l[:, None]).astype(ar.dt))
    LSE = (ar.c(a) * xmax[:, 0]).astype(ar.dt) + ar.log(l).astype(ar.dt)
    return O, LSE.astype(ar.dt), x


def backward(q, k, v, o, lse, u, causal: bool, alpha: float, mode: str,
             rounding: bool = True, x=None):
    """Algorithm 1 for one head.  Returns dQ, dK, dV and a dict of the row
    statistics and accumulators (rho, m, lam, A, B, dKacc, C, r, t, P)."""
    if mode not in MODES:
        raise ValueError(mode)
    ar = _Arith(rounding)
    W = ar.wide
    N = q.shape[0]
    a = ar.c(alpha)
    c = ar.c(a * ar.c(LOG2E))
    if x is None:
        x = ar.f32(W(q) @ W(k).T)
    mask = _mask(N, causal)
    lse2 = (np.asarray(lse).astype(ar.dt) * ar.c(LOG2E)).astype(ar.dt)
    arg = ar.f32(W(x) * float(c) - W(lse2)[:, None]) if rounding else (x * c - lse2[:, None])
    with np.errstate(invalid="ignore", over="ignore"):
        P = np.where(mask, ar.exp2(np.where(mask, arg, 0)), 0).astype(ar.dt)
    D = ar.f32((W(u) * W(o)).sum(axis=1))
    dP = ar.f32(W(u) @ W(v).T)
    r = ar.bf16(P)
    t = ar.bf16((P * (dP - D[:, None]).astype(ar.dt)).astype(ar.dt))
    t = np.where(mask, t, 0).astype(ar.dt)
    r = np.where(mask, r, 0).astype(ar.dt)
    rho = ar.f32(W(t).sum(axis=1))
    m = ar.f32(W(r).sum(axis=1))
    A = ar.f32(W(t) @ W(k))
    B = ar.f32(W(r) @ W(k))
    with np.errstate(invalid="ignore", divide="ignore"):
        lam = np.where(m != 0, (rho / np.where(m != 0, m, 1)).astype(ar.dt), 0).astype(ar.dt)
    if mode == "plain":
        dQ = ar.bf16((a * A).astype(ar.dt))
    else:
        corr = (lam[:, None] * B).astype(ar.dt)
        dQ = ar.bf16((a * (A - corr).astype(ar.dt)).astype(ar.dt))
    dKacc = ar.f32(W(t).T @ W(q))
    dV = ar.bf16(ar.f32(W(r).T @ W(u)))
    z = ar.bf16((lam[:, None] * np.asarray(q).astype(ar.dt)).astype(ar.dt))
    C = ar.f32(W(r).T @ W(z))
    if mode == "gproj":
        dK = ar.bf16((a * (dKacc - C).astype(ar.dt)).astype(ar.dt))
    else:
        dK = ar.bf16((a * dKacc).astype(ar.dt))
    stats = dict(rho=rho, m=m, lam=lam, A=A, B=B, dKacc=dKacc, C=C, r=r, t=t, P=P, D=D)
    return dQ, dK, dV, stats


def forward_backward(q, k, v, u, causal: bool, alpha: float, mode: str, rounding: bool = True):
    """Convenience: SBS forward then Algorithm 1 backward on one head."""
    O, LSE, x = sbs_forward(q, k, v, causal, alpha, rounding)
    dQ, dK, dV, st = backward(q, k, v, O, LSE, u, causal, alpha, mode, rounding, x=x)
    return O, LSE, dQ, dK, dV, st


def project_query_row(t, r, K, alpha):
    """GProj query contraction of one row (Section 4): alpha (t K - (rho/m) r K)."""
    t = np.asarray(t, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    rho = t.sum()
    m = r.sum()
    lam = rho / m if m != 0 else 0.0
    return alpha * (t @ K - lam * (r @ K))


# ------------------------------------------------------------------ diagnostic
def historical_fma_one_key(x, alpha, v):
    """Output row of a query with exactly one visible key under the historical
    FMA forward (appendix on the source of the saved-output error, eqs.
    historical-fma and historical-one-key), the scalar model the paper uses to
    explain the one-key violations:
        a = fl32(alpha log2 e),  r = fma(x, a, -fl32(x a)),  z = exp2_32(r),
        o = BF16( fl32[ BF16(z) v / z ] )
    x is the (FP32) unscaled logit of the single key, which is also the row
    maximum; v the key's value row (BF16 values).  The FMA rounds the exact
    x*a - fl32(x a) once to FP32 (computed exactly in FP64: the product of two
    FP32 values has at most 48 significant bits, and the difference is the
    rounding error of that product, exactly representable).  Returns float32.
    """
    a = np.float32(np.float32(alpha) * np.float32(LOG2E))
    x32 = np.float32(x)
    ma = np.float32(x32 * a)                           # fl32(m a)
    exact = np.float64(x32) * np.float64(a) - np.float64(ma)
    r = np.float32(exact)                              # the FMA's single rounding
    z = np.exp2(r, dtype=np.float32)
    zb = bf16_round(np.float32(z))
    acc = (np.asarray(v, dtype=np.float32) * np.float32(zb)).astype(np.float32)
    return bf16_round((acc / np.float32(z)).astype(np.float32))
