"""Pins of the BF16 algorithm model (oracle.algo_model) against the paper.

The model is the step-by-step statement of the paper's forward (eq.
gproj-forward) and Algorithm 1 backward with the implemented rounding points.
It is pinned by: an independent brute-force BF16 rounding check, the -24
witness values the paper prints, the exact-arithmetic limit (equals the exact
FP64 oracle), Proposition 4.1's algebraic properties, the two-key bound, and
the synthetic offset sweep floor the paper reports.
"""
import json
import os
import sys

import numpy as np
import pytest

import oracle
import synthetic as S
from oracle import algo_model as M

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _bf16_nearest_bruteforce(x: float) -> float:
    """Nearest BF16 value by enumeration of neighbours; ties to even mantissa."""
    f = np.float32(x)
    bits = int(np.array([f]).view(np.uint32)[0])
    base = bits & 0xFFFF0000
    cands = []
    for cb in (base - 0x10000, base, base + 0x10000):
        if cb < 0 or cb > 0xFFFFFFFF:
            continue
        val = float(np.array([cb], dtype=np.uint32).view(np.float32)[0])
        if np.isfinite(val):
            cands.append((abs(val - float(f)), (cb >> 16) & 1, val))
    cands.sort()
    best = [c for c in cands if c[0] == cands[0][0]]
    if len(best) > 1:
        best = [c for c in best if c[1] == 0]
    return best[0][2]


def test_bf16_round_against_bruteforce():
    rng = np.random.default_rng(1)
    xs = np.concatenate([rng.standard_normal(2000) * 10.0 ** rng.integers(-6, 6, 2000),
                         np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 3 / 1024, -0.125732421875,
                                   65536.0, 2 ** -126, 3.0e38])])
    got = M.bf16_round(xs.astype(np.float32))
    for x, g in zip(xs, got):
        assert g == _bf16_nearest_bruteforce(x), x
    # ties to even, and the paper's example: 1 + 3/1024 rounds to 1
    assert M.bf16_round(np.float32([1 + 2 ** -8]))[0] == 1.0
    assert M.bf16_round(np.float32([1 + 3 * 2 ** -8]))[0] == np.float32(1 + 2 ** -6)
    assert M.bf16_round(np.float32([1 + 3 / 1024]))[0] == 1.0


def _witness(golden_dir):
    with open(os.path.join(golden_dir, "witness_minus24.json")) as f:
        w = json.load(f)
    pb = w["printed_by_paper"]
    N, d = 4, 64
    q = np.zeros((N, d), np.float32); k = np.zeros((N, d), np.float32)
    v = np.zeros((N, d), np.float32); u = np.zeros((N, d), np.float32)
    k[:, :2] = pb["k"]; v[:, :2] = pb["v"]; u[3, :2] = pb["u"]
    return w, q, k, v, u


def _witness_from_printed(pb):
    """Witness-row dQ from the paper's printed values alone, in exact
    rationals: A = sum_j t_j k_j with the printed BF16 t, B = sum_j r_j k_j
    with r = BF16(p) = p (every printed p is 1/4, a BF16 value), lambda =
    rho / m with the printed rho and m = sum r = 1; plain dq = BF16(alpha A),
    GProj dq = BF16(fl32[alpha (A - lambda B)]) (every intermediate here is
    exact in FP32)."""
    from fractions import Fraction as F
    import _sbs_rational as R
    t = [F(x) for x in pb["t_bf16"]]
    r = [F(x) for x in pb["p"]]
    k = [[F(x) for x in row] for row in pb["k"]]
    alpha = F(pb["alpha"])
    A = [sum(t[j] * k[j][c] for j in range(4)) for c in range(2)]
    B = [sum(r[j] * k[j][c] for j in range(4)) for c in range(2)]
    lam = F(pb["rho"]) / sum(r)
    before = [alpha * (A[c] - lam * B[c]) for c in range(2)]
    assert all(R.rn32(x) == x for x in A + B + before)  # exact in FP32
    return {"A": [float(x) for x in A], "B": [float(x) for x in B], "lambda": float(lam),
            "gproj_dq_before_cast": [float(x) for x in before],
            "plain_dq_bf16": [float(R.bf16_nearest(R.rn32(alpha * A[c]))) for c in range(2)],
            "gproj_dq_bf16": [float(R.bf16_nearest(R.rn32(x))) for x in before]}


def test_witness_derived_values_match_the_fixture(golden_dir):
    """The fixture's oracle-written block (tests/golden/derive_witness.py)
    equals both what that script derives now and the exact-rational values
    computed from the printed quantities alone."""
    sys.path.insert(0, golden_dir)
    import derive_witness
    with open(os.path.join(golden_dir, "witness_minus24.json")) as f:
        w = json.load(f)
    stored = w["derived_by_oracle"]
    fresh = derive_witness.derive(w["printed_by_paper"])
    for key, val in fresh.items():
        assert stored[key] == val, key
    hand = _witness_from_printed(w["printed_by_paper"])
    for key, val in hand.items():
        assert stored[key] == val, key
    assert stored["exact_dq"][0] == w["printed_by_paper"]["exact_dq_first_coordinate"]


def test_witness_through_the_model(golden_dir):
    """Plain contracts the cast operand and returns -24; GProj returns exactly 0
    (Section 3.4, appendix A, Section 5.2 'on the four-key example ... exactly zero')."""
    w, q, k, v, u = _witness(golden_dir)
    pb, hand = w["printed_by_paper"], _witness_from_printed(w["printed_by_paper"])
    alpha = pb["alpha"]
    out = {}
    for mode in M.MODES:
        O, LSE, dQ, dK, dV, st = M.forward_backward(q, k, v, u, True, alpha, mode)
        out[mode] = (O, dQ, dK, dV, st)
    O, dQ, dK, dV, st = out["plain"]
    assert list(O[3, :2]) == pb["o"]
    assert list(st["t"][3, :4]) == pb["t_bf16"]
    assert st["rho"][3] == pb["rho"]
    assert np.float32(alpha) * st["A"][3, 0] == pb["plain_dq_first_coordinate"]
    assert list(dQ[3, :2]) == hand["plain_dq_bf16"]
    for mode in ("gproj_q", "gproj"):
        _, dQg, dKg, dVg, stg = out[mode]
        assert dQg[3, 0] == 0.0
        assert list(dQg[3, :2]) == hand["gproj_dq_bf16"]
        assert stg["lam"][3] == np.float32(-pb["eta"])
        assert np.abs(dKg).max() == 0.0
        assert np.all(dVg[:, :2] == 0.25)


def test_model_mode_identities():
    """gproj_q leaves dK, dV as plain; the key pass leaves dQ, dV as gproj_q
    (Section 5.2; appendix 'Backward-only comparison')."""
    w = S.WORKLOADS[1]
    x = S.make_inputs(w, 1001)
    q, k, v, u = (S.bf16_bits_to_f32(x[n][0, 0]) for n in ("q", "k", "v", "do"))
    res = {m: M.forward_backward(q, k, v, u, True, w.scale, m) for m in M.MODES}
    assert np.array_equal(res["plain"][3], res["gproj_q"][3])
    assert np.array_equal(res["plain"][4], res["gproj_q"][4])
    assert np.array_equal(res["gproj_q"][2], res["gproj"][2])
    assert np.array_equal(res["gproj_q"][4], res["gproj"][4])
    assert not np.array_equal(res["plain"][2], res["gproj"][2])


@pytest.mark.parametrize("causal", [True, False])
def test_model_exact_limit_equals_oracle(causal):
    """With every cast the identity and FP64 arithmetic, the model is the exact VJP."""
    rng = np.random.default_rng(2)
    N, d = 70, 16
    q = rng.standard_normal((N, d)); k = rng.standard_normal((N, d)) + 5 * rng.standard_normal(d)
    v = rng.standard_normal((N, d)); u = rng.standard_normal((N, d))
    ex = oracle.exact(q[None], k[None], v[None], u[None], causal, 0.3)
    for mode in M.MODES:
        O, LSE, dQ, dK, dV, st = M.forward_backward(q, k, v, u, causal, 0.3, mode, rounding=False)
        for n, a in zip(("O", "LSE", "dQ", "dK", "dV"), (O, LSE, dQ, dK, dV)):
            ref = ex[n][0]
            assert np.linalg.norm(a - ref) <= 1e-11 * max(1.0, np.linalg.norm(ref)), (mode, n)


def test_projection_properties():
    """Proposition 4.1: Pi_r idempotent, 1^T Pi_r = 0, t - lambda r has zero row
    sum, the query contraction equals alpha sum_j t_j (k_j - mu_r) and is
    unchanged by a common key translation at fixed t, r; t - lambda r is the
    minimum of sum (z - t)^2 / r over zero-sum z."""
    rng = np.random.default_rng(4)
    L, d, alpha = 50, 8, 0.7
    r = rng.random(L) + 0.01
    t = rng.standard_normal(L)
    K = rng.standard_normal((L, d))
    m = r.sum()
    Pi = np.eye(L) - np.outer(r, np.ones(L)) / m
    assert np.allclose(Pi @ Pi, Pi, atol=1e-13)
    assert np.allclose(np.ones(L) @ Pi, 0, atol=1e-13)
    tp = Pi @ t
    assert abs(tp.sum()) < 1e-12
    assert np.allclose(tp, t - (t.sum() / m) * r, atol=1e-13)
    G = M.project_query_row(t, r, K, alpha)
    mu_r = (r @ K) / m
    assert np.allclose(G, alpha * (t @ (K - mu_r)), atol=1e-12)
    b = rng.standard_normal(d) * 1e4
    assert np.allclose(M.project_query_row(t, r, K + b, alpha), G, rtol=0, atol=1e-8)
    # minimum r-weighted norm among zero-sum vectors: perturb along zero-sum directions
    base = np.sum((tp - t) ** 2 / r)
    for _ in range(20):
        e = rng.standard_normal(L); e -= e.mean()
        assert np.sum((tp + 1e-3 * e - t) ** 2 / r) >= base


def test_two_key_row_mass_bound():
    """Eq. two-key: |rho| <= 2 u_b eps(1-eps)|a1 - a2| for the BF16 cast t of g."""
    rng = np.random.default_rng(6)
    ub = 2.0 ** -8
    for _ in range(2000):
        eps = rng.random() * 0.5
        a1, a2 = rng.standard_normal(2) * 10.0 ** rng.integers(-3, 3)
        p = np.array([1 - eps, eps])
        a = np.array([a1, a2])
        g = p * (a - p @ a)
        t = M.bf16_round(g.astype(np.float32)).astype(np.float64)
        rho = t.sum()
        assert abs(rho) <= 2 * ub * eps * (1 - eps) * abs(a1 - a2) * (1 + 1e-6)


def _offset_sweep(std, offsets, rows, L=1024, d=64, seed=0):
    """Appendix D 'Synthetic offset sweep': exact FP64 forward and score gradient,
    t = BF16(g), r = BF16(p); per-row relative dq error, median over rows."""
    rng = np.random.default_rng(seed)
    out = {}
    for nb in offsets:
        eg, ef = [], []
        for _ in range(rows):
            z = rng.standard_normal((L, d))
            dirb = rng.standard_normal(d); dirb /= np.linalg.norm(dirb)
            K = z + nb * dirb
            q = rng.standard_normal(d); q *= std / np.linalg.norm(q)
            s = K @ q
            p = np.exp(s - s.max()); p /= p.sum()
            a = rng.standard_normal((L, d)) @ rng.standard_normal(d)
            g = p * (a - p @ a)
            G = g @ K
            t = M.bf16_round(g.astype(np.float32)).astype(np.float64)
            r = M.bf16_round(p.astype(np.float32)).astype(np.float64)
            Gf = t @ K
            Gp = M.project_query_row(t, r, K, 1.0)
            eg.append(np.linalg.norm(Gp - G) / np.linalg.norm(G))
            ef.append(np.linalg.norm(Gf - G) / np.linalg.norm(G))
        out[nb] = (100 * np.median(eg), 100 * np.median(ef))
    return out


def test_offset_sweep_floor():
    """Figure 1 panel 2: GProj stays at a floor of 0.12-0.17 % at logit std 3 for
    key offsets from 1 to 1e4, while contracting t directly grows with the offset."""
    res = _offset_sweep(3.0, [1.0, 100.0, 1e4], rows=256)
    for nb, (gp, fwd) in res.items():
        assert 0.12 <= gp <= 0.17, (nb, gp)
    assert res[1e4][1] > 100 * res[1e4][0]
    assert res[100.0][1] > 5 * res[100.0][0]
    assert res[1e4][1] > 20 * res[100.0][1]


def test_historical_fma_argument_is_the_rounding_error():
    """eq. historical-fma: with x = m, fma(x, a, -fl32(m a)) is exactly the
    rounding error x a - fl32(x a) (representable in FP32), checked with exact
    rational arithmetic; the model's one-key output then follows eq.
    historical-one-key, and equals v exactly when z is 1."""
    from fractions import Fraction
    a = np.float32(np.float32(0.125) * np.float32(M.LOG2E))
    for c in (3, 5, 7):
        for k in range(16):
            x = np.float32(64 * c * 2 ** k)
            prod = Fraction(float(x)) * Fraction(float(a))
            rounded = Fraction(float(np.float32(x * a)))
            err = prod - rounded
            assert Fraction(float(np.float32(float(err)))) == err  # exactly representable
            v = np.arange(-4, 4, dtype=np.float32)
            o = M.historical_fma_one_key(x, 0.125, v)
            z = np.exp2(np.float32(float(err)), dtype=np.float32)
            if z == np.float32(1.0):
                assert np.array_equal(o, v)
            want = M.bf16_round((v * M.bf16_round(z)) / z)
            assert np.array_equal(o, want)


# ------------------------------------------------ the SBS forward, pinned

def test_sbs_forward_single_key_rows_are_exact():
    """Appendix 'Prescribed FMA cases': query coordinates c * 2^k (c in
    {3, 5, 7}, k = 0..15), key coordinates 1, lengths 1 and 128.  The first
    causal row sees one key, so the subtract-before-scale forward must give
    z = 1 exactly and o_0 = v_0 bit for bit, and LSE_0 = fl32(alpha x_0), in
    all 96 cases."""
    rng = np.random.default_rng(0)
    d = 64
    for N in (1, 128):
        for cval in (3, 5, 7):
            for kexp in range(16):
                q = np.full((N, d), cval * 2.0 ** kexp, np.float32)
                k = np.ones((N, d), np.float32)
                v = rng.integers(-4, 5, (N, d)).astype(np.float32)
                O, LSE, x = M.sbs_forward(q, k, v, True, 0.125)
                assert np.array_equal(O[0], v[0]), (N, cval, kexp)
                x0 = np.float32(64 * cval * 2.0 ** kexp)
                assert x[0, 0] == x0
                assert LSE[0] == np.float32(np.float32(0.125) * x0), (N, cval, kexp)


def test_sbs_forward_rounding_order_against_exact_rationals():
    """Eq. gproj-forward evaluated in exact rational arithmetic (each FP32
    operation rounded to nearest once, exp2 and ln to 60 digits) on a row
    whose logits are ~4.2e6: the model's O and LSE equal the
    subtract-then-scale evaluation bit for bit, while the scale-then-subtract
    order and the historical FMA give different outputs on this row (so a
    model that swapped the order would fail here)."""
    import _sbs_rational as R
    q, k, v, x = R.rounding_order_row()
    for causal in (False, True):
        O, LSE, xm = M.sbs_forward(q, k, v, causal, 0.125)
        assert [np.float32(t) for t in xm[-1, :len(x)]] == x  # logits exact in FP32
        last = len(x) - 1
        o_ref, lse_ref, _ = R.sbs_row(x, v, 0.125, "sbs")
        assert np.array_equal(O[last], o_ref)
        assert LSE[last] == lse_ref
    o_sts, _, _ = R.sbs_row(x, v, 0.125, "scale_then_subtract")
    o_fma, _, _ = R.sbs_row(x, v, 0.125, "fma")
    assert np.count_nonzero(R.bf16_ulps(o_sts, o_ref) >= 2) >= 10
    assert np.count_nonzero(R.bf16_ulps(o_fma, o_ref) >= 2) >= 10
    # rows with a single visible key (causal row 0) are exact in every order
    O, _, _ = M.sbs_forward(q, k, v, True, 0.125)
    assert np.array_equal(O[0], v[0])


def test_historical_fma_one_key_outer_formula_in_rationals():
    """Eq. historical-one-key, o = BF16(fl32(BF16(z) v / z)), checked with the
    FP32 product and quotient evaluated exactly and rounded once each, for
    the 48 single-key logits 64 c 2^k and a spread of value rows."""
    import _sbs_rational as R
    from fractions import Fraction
    a = np.float32(np.float32(0.125) * np.float32(M.LOG2E))
    rng = np.random.default_rng(5)
    for c in (3, 5, 7):
        for kexp in range(16):
            x = np.float32(64 * c * 2 ** kexp)
            err = Fraction(float(x)) * Fraction(float(a)) - Fraction(float(np.float32(x * a)))
            z = R.exp2_rn32(R.rn32(err))
            zb = R.bf16_nearest(z)
            v = np.array([R.bf16_nearest(t) for t in rng.standard_normal(16) * 4], np.float32)
            want = np.array([R.bf16_nearest(R.rn32(Fraction(float(R.rn32(Fraction(float(zb)) *
                                                                        Fraction(float(vi)))))
                                                   / Fraction(float(z))))
                             for vi in v], np.float32)
            assert np.array_equal(M.historical_fma_one_key(x, 0.125, v), want), (c, kexp)


def test_row_and_tile_bounds_on_the_model_and_planted_defects():
    """The per-row / per-tile parity bounds used at full size: the BF16 model
    of Algorithm 1 meets them on the reference recipe (N = 1024, two heads),
    and a planted defect in its output -- one 64-row tile scaled by 1.07, or
    one row by 1.6 -- breaks them."""
    import _rowtile as RT
    w = S.WORKLOADS[2].with_shape(H=2, N=1024)
    x = S.make_inputs(w, 11)
    ex = oracle.exact(x["q"], x["k"], x["v"], x["do"], True, w.scale)
    outs = {}
    for h in range(2):
        q, k, v, u = (S.bf16_bits_to_f32(x[n][0, h]) for n in ("q", "k", "v", "do"))
        O, L, dq, dk, dv, st = M.forward_backward(q, k, v, u, True, w.scale, "gproj")
        for n, a in zip(("O", "dQ", "dK", "dV"), (O, dq, dk, dv)):
            outs.setdefault(n, []).append(a)
    for n, arrs in outs.items():
        got = np.stack(arrs)[None].astype(np.float64)
        RT.check(got, ex[n], n)
        bad = got.copy()
        bad[0, 1, 640:704] *= 1.07
        with pytest.raises(AssertionError):
            RT.check(bad, ex[n], n)
        bad = got.copy()
        bad[0, 0, 300] *= 1.6
        with pytest.raises(AssertionError):
            RT.check(bad, ex[n], n)
