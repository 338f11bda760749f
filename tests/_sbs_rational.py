"""Exact-rational evaluation of the FA3-SBS forward for one query row (test
helper, not a test module).

Eq. gproj-forward (appendix "Implemented Arithmetic and Rounding") fixes the
order of the exponent argument: subtract the unscaled row maximum in FP32,
then multiply by the FP32 constant fl32(alpha) * fl32(log2 e), rounded once
more.  Here every FP32 operation is evaluated in exact rational arithmetic and
rounded to the nearest FP32 value (ties to even) by comparison of neighbours,
exp2 is evaluated to 60 decimal digits and rounded the same way, and the two
FP32 accumulations (the normaliser l and the value numerator) are exact sums
rounded once.  Alternative orders -- scale then subtract, and the historical
fused multiply-add -- are available so that a test can show the row tells them
apart.
"""
from __future__ import annotations

from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np

LOG2E = 1.4426950408889634


def rn32(x) -> np.float32:
    """Nearest FP32 value to the rational x (ties to the even significand)."""
    x = Fraction(x)
    f = np.float32(float(x))
    cands = (np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf)))
    return min(cands, key=lambda c: (abs(Fraction(float(c)) - x),
                                     int(np.array([c], np.float32).view(np.uint32)[0]) & 1))


def bf16_nearest(x) -> np.float32:
    """Nearest BF16 value to the FP32 value x (ties to even), by enumeration."""
    f = np.float32(x)
    bits = int(np.array([f], np.float32).view(np.uint32)[0]) & 0xFFFF0000
    cands = []
    for cb in (bits - 0x10000, bits, bits + 0x10000):
        if 0 <= cb <= 0xFFFFFFFF:
            c = np.array([cb], np.uint32).view(np.float32)[0]
            if np.isfinite(c):
                cands.append((abs(Fraction(float(c)) - Fraction(float(f))), (cb >> 16) & 1, c))
    cands.sort(key=lambda t: (t[0], t[1]))
    return np.float32(cands[0][2])


def exp2_rn32(a) -> np.float32:
    getcontext().prec = 60
    return rn32(Fraction(Decimal(2) ** Decimal(float(a))))


def ln_rn32(x) -> np.float32:
    getcontext().prec = 60
    return rn32(Fraction(Decimal(float(x)).ln()))


def _q(x) -> Fraction:
    return Fraction(float(x))


def sbs_row(x, v, alpha: float, order: str = "sbs"):
    """One row of the forward from its FP32 logits x (row maximum included)
    and the BF16 value rows v [len(x), dv].  order: "sbs" (subtract, then
    scale: eq. gproj-forward), "scale_then_subtract" or "fma" (the historical
    fma(x, a, -fl32(m a))).  Returns (o, lse, z): o BF16 values as float32,
    lse = fl32(fl32(alpha) x_max) + ln l rounded to FP32, z the FP32
    probabilities before normalisation."""
    a = np.float32(alpha)
    c = rn32(_q(a) * _q(np.float32(LOG2E)))
    xm = max(_q(t) for t in x)
    if order == "sbs":
        args = [rn32(_q(rn32(_q(t) - xm)) * _q(c)) for t in x]
    elif order == "scale_then_subtract":
        args = [rn32(_q(rn32(_q(t) * _q(c))) - _q(rn32(xm * _q(c)))) for t in x]
    elif order == "fma":
        args = [rn32(_q(t) * _q(c) - _q(rn32(xm * _q(c)))) for t in x]
    else:
        raise ValueError(order)
    z = [exp2_rn32(t) for t in args]
    l = rn32(sum(_q(t) for t in z))
    zb = [bf16_nearest(t) for t in z]
    v = np.asarray(v, np.float32)
    num = [rn32(sum(_q(zb[j]) * _q(v[j, c_]) for j in range(len(x)))) for c_ in range(v.shape[1])]
    o = np.array([bf16_nearest(rn32(_q(n) / _q(l))) for n in num], np.float32)
    lse = rn32(_q(rn32(_q(a) * xm)) + _q(ln_rn32(l)))
    return o, lse, np.array(z, np.float32)


def rounding_order_row(d: int = 64, n_keys: int = 4, seed: int = 3):
    """A row whose rounding orders give different outputs: every query is
    q = (2^12, 1, 0, ...), key j is k_j = (1032, delta_j, 0, ...) with
    delta = (0, -1, -3, -7.5, ...), so the unscaled logits are
    x_j = 4227072 + delta_j, exact in FP32 in any summation order.  At that
    magnitude fl32(x c) carries rounding errors of up to 1/32 while the
    differences x_j - x_max are exact, so subtract-then-scale, scale-then-
    subtract and the FMA give exponent arguments that differ by up to ~0.06.
    Returns q, k, v (float32 [n_keys, d], BF16 values) and x (FP32 logits)."""
    deltas = [0.0, -1.0, -3.0, -7.5, -0.5, -12.0, -2.5, -5.0][:n_keys]
    q = np.zeros((n_keys, d), np.float32)
    q[:, 0] = 2.0 ** 12
    q[:, 1] = 1.0
    k = np.zeros((n_keys, d), np.float32)
    k[:, 0] = 1032.0
    k[:, 1] = deltas
    rng = np.random.default_rng(seed)
    v = rng.standard_normal((n_keys, d)).astype(np.float32)
    v = np.array([[bf16_nearest(t) for t in row] for row in v], np.float32)
    x = [np.float32(4227072.0 + dl) for dl in deltas]
    return q, k, v, x


def bf16_ulps(a, b) -> np.ndarray:
    """Distance in BF16 units of the last place between BF16-valued float32
    arrays of the same sign pattern (for reporting)."""
    ai = np.asarray(a, np.float32).view(np.int32).astype(np.int64) >> 16
    bi = np.asarray(b, np.float32).view(np.int32).astype(np.int64) >> 16
    return np.abs(ai - bi)
