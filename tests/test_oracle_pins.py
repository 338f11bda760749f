"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every check here is independent of the oracle's own formulas: brute force in
high-precision decimal arithmetic, central finite differences, closed forms,
conservation laws, invariances, values the paper prints, and an independent
second reference with different algebra.
"""
import decimal
import json
import os

import numpy as np
import pytest

import oracle
import synthetic as S

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _rand_case(rng, N, d, kbias=0.0, scale=1.0):
    q = rng.standard_normal((N, d)) * scale
    k = rng.standard_normal((N, d)) + kbias * rng.standard_normal(d)[None, :]
    v = rng.standard_normal((N, d))
    u = rng.standard_normal((N, d))
    return q, k, v, u


def _exact_head(q, k, v, u, causal, alpha):
    r = oracle.exact(q[None], k[None], v[None], u[None], causal, alpha)
    return {n: r[n][0] for n in r}


# ---------------------------------------------------------------- brute force

def _decimal_forward(q, k, v, u, causal, alpha, prec=50, dirs=None, h=None):
    """O, LSE and the scalar L = sum O*u by direct, unshifted softmax in
    50-digit decimal arithmetic (no max subtraction, no centering).
    With dirs=(dq, dk, dv) and a Decimal step h, the inputs are perturbed to
    x + h*dir inside the decimal arithmetic (no FP64 rounding of the step)."""
    ctx = decimal.Context(prec=prec)
    D = lambda x: ctx.create_decimal(repr(float(x)))  # noqa: E731
    N, d = q.shape

    def lift(x, dx):
        out = [[D(x[i, c]) for c in range(x.shape[1])] for i in range(x.shape[0])]
        if dx is not None:
            out = [[out[i][c] + h * D(dx[i, c]) for c in range(x.shape[1])]
                   for i in range(x.shape[0])]
        return out

    dq_, dk_, dv_ = dirs if dirs is not None else (None, None, None)
    Qd, Kd, Vd = lift(q, dq_), lift(k, dk_), lift(v, dv_)
    a = D(alpha)
    O = np.zeros((N, v.shape[1]))
    LSE = np.zeros(N)
    Ltot = D(0)
    for i in range(N):
        L = i + 1 if causal else N
        s = [a * sum((Qd[i][c] * Kd[j][c] for c in range(d)), D(0)) for j in range(L)]
        e = [ctx.exp(x) for x in s]
        Z = sum(e, D(0))
        LSE[i] = float(ctx.ln(Z))
        for c in range(v.shape[1]):
            oc = sum((e[j] * Vd[j][c] for j in range(L)), D(0)) / Z
            O[i, c] = float(oc)
            Ltot += oc * D(u[i, c])
    return O, LSE, Ltot


@pytest.mark.parametrize("causal", [True, False])
def test_forward_matches_decimal_brute_force(causal):
    rng = np.random.default_rng(7)
    q, k, v, u = _rand_case(rng, 5, 3, kbias=3.0, scale=2.0)
    ex = _exact_head(q, k, v, u, causal, 0.7)
    O, LSE, _ = _decimal_forward(q, k, v, u, causal, 0.7)
    assert np.allclose(ex["O"], O, rtol=0, atol=1e-13)
    assert np.allclose(ex["LSE"], LSE, rtol=0, atol=1e-13)


@pytest.mark.parametrize("causal", [True, False])
def test_vjp_matches_central_finite_differences(causal):
    """dQ, dK, dV are the gradients of L = sum(O * dO) (the VJP with u = dO)."""
    rng = np.random.default_rng(11)
    N, d, alpha = 6, 4, 0.6
    q, k, v, u = _rand_case(rng, N, d, kbias=2.0)
    ex = _exact_head(q, k, v, u, causal, alpha)
    h = 1e-5

    def L(qq, kk, vv):
        r = _exact_head(qq, kk, vv, u, causal, alpha)
        return float(np.sum(r["O"] * u))

    for name, arr, grad in (("q", q, ex["dQ"]), ("k", k, ex["dK"]), ("v", v, ex["dV"])):
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            ap = arr.copy(); ap[idx] += h
            am = arr.copy(); am[idx] -= h
            args_p = [q, k, v]; args_m = [q, k, v]
            pos = "qkv".index(name)
            args_p[pos] = ap; args_m[pos] = am
            fd[idx] = (L(*args_p) - L(*args_m)) / (2 * h)
        scale = np.abs(grad).max()
        assert np.abs(fd - grad).max() <= 1e-7 * max(scale, 1.0), name


def test_vjp_matches_decimal_finite_difference_direction():
    """Directional derivative of L from the 50-digit brute force (no FP64 at all)
    equals <grad, direction> from the oracle."""
    rng = np.random.default_rng(3)
    N, d, alpha = 4, 3, 0.9
    q, k, v, u = _rand_case(rng, N, d, kbias=1.5)
    ex = _exact_head(q, k, v, u, True, alpha)
    dq_dir, dk_dir, dv_dir = (rng.standard_normal((N, d)) for _ in range(3))
    h = decimal.Decimal("1e-15")
    dirs = (dq_dir, dk_dir, dv_dir)
    _, _, Lp = _decimal_forward(q, k, v, u, True, alpha, dirs=dirs, h=h)
    _, _, Lm = _decimal_forward(q, k, v, u, True, alpha, dirs=dirs, h=-h)
    fd = float((Lp - Lm) / (2 * h))
    an = float(np.sum(ex["dQ"] * dq_dir) + np.sum(ex["dK"] * dk_dir) + np.sum(ex["dV"] * dv_dir))
    assert abs(fd - an) <= 1e-12 * max(1.0, abs(an))


# -------------------------------------------------------- conservation laws

@pytest.mark.parametrize("causal", [True, False])
def test_conservation_laws(causal):
    """1^T g = 0 on every row (Proposition 3.1) implies sum_j dk_j = 0 per head;
    sum_j p_ij = 1 implies sum_j dv_j = sum_i u_i."""
    rng = np.random.default_rng(5)
    q, k, v, u = _rand_case(rng, 97, 16, kbias=6.0)
    ex = _exact_head(q, k, v, u, causal, 0.25)
    scale_k = np.abs(ex["dK"]).sum(axis=0).max()
    assert np.abs(ex["dK"].sum(axis=0)).max() <= 1e-13 * scale_k
    assert np.allclose(ex["dV"].sum(axis=0), u.sum(axis=0), rtol=0, atol=1e-12)


@pytest.mark.parametrize("causal", [True, False])
def test_translation_invariance(causal):
    """Common key and value translations leave the VJP unchanged at fixed u
    (Proposition 3.1); LSE shifts by alpha q.b and O by c."""
    rng = np.random.default_rng(9)
    q, k, v, u = _rand_case(rng, 64, 8, kbias=1.0)
    alpha = 0.35
    base = _exact_head(q, k, v, u, causal, alpha)
    b = rng.standard_normal(8) * 300.0
    c = rng.standard_normal(8) * 50.0
    shk = _exact_head(q, k + b[None, :], v, u, causal, alpha)
    shv = _exact_head(q, k, v + c[None, :], u, causal, alpha)
    big = np.zeros(8); big[0] = 65536.0
    shbig = _exact_head(q, k + big[None, :], v, u, causal, alpha)
    for n in ("dQ", "dK", "dV"):
        ref = np.linalg.norm(base[n])
        assert np.linalg.norm(shk[n] - base[n]) <= 1e-11 * ref, n
        assert np.linalg.norm(shv[n] - base[n]) <= 1e-11 * ref, n
        # k + 65536 is rounded in FP64 (ulp 1.5e-11): allow that much
        assert np.linalg.norm(shbig[n] - base[n]) <= 1e-9 * ref, n
    assert np.allclose(shk["LSE"], base["LSE"] + alpha * (q @ b), rtol=1e-12, atol=1e-9)
    assert np.allclose(shk["O"], base["O"], rtol=0, atol=1e-11)
    assert np.allclose(shv["O"], base["O"] + c[None, :], rtol=0, atol=1e-11)


# -------------------------------------------------------------- closed forms

def test_two_key_closed_form():
    """Eq. two-key: with weights (1-eps, eps), G_Q = alpha eps(1-eps)(a1-a2)(k1-k2)."""
    rng = np.random.default_rng(13)
    for _ in range(20):
        d = 8
        alpha = 0.3
        q = np.zeros((2, d)); u = np.zeros((2, d))
        q[1] = rng.standard_normal(d) * 2
        u[1] = rng.standard_normal(d)
        k = rng.standard_normal((2, d)) * 3
        v = rng.standard_normal((2, d))
        ex = _exact_head(q, k, v, u, False, alpha)
        s = alpha * (k @ q[1])
        eps = 1.0 / (1.0 + np.exp(s[0] - s[1]))   # weight of key 2
        a1, a2 = u[1] @ v[0], u[1] @ v[1]
        gq = alpha * eps * (1 - eps) * (a1 - a2) * (k[0] - k[1])
        assert np.allclose(ex["dQ"][1], gq, rtol=1e-12, atol=1e-15)


def _witness_inputs(golden_dir, d=64):
    with open(os.path.join(golden_dir, "witness_minus24.json")) as f:
        w = json.load(f)["printed_by_paper"]
    N = 4
    q = np.zeros((N, d)); k = np.zeros((N, d)); v = np.zeros((N, d)); u = np.zeros((N, d))
    k[:, :2] = np.array(w["k"])
    v[:, :2] = np.array(w["v"])
    u[3, :2] = np.array(w["u"])
    return w, q, k, v, u


def test_witness_exact_values(golden_dir):
    """The -24 witness (appendix A): exact dq has first coordinate 0."""
    w, q, k, v, u = _witness_inputs(golden_dir)
    ex = _exact_head(q, k, v, u, True, w["alpha"])
    assert ex["dQ"][3, 0] == pytest.approx(0.0, abs=1e-9)
    assert ex["dQ"][3, 1] == pytest.approx(-0.125732421875, abs=1e-15)
    assert np.abs(ex["dQ"][:3]).max() == 0.0
    assert np.abs(ex["dQ"][3, 2:]).max() == 0.0
    assert np.abs(ex["dK"]).max() == 0.0
    assert np.allclose(ex["dV"][:, :2], 0.25, rtol=0, atol=1e-15)
    assert np.allclose(ex["O"][3, :2], w["o"], rtol=0, atol=1e-15)


def test_special_cases():
    """Singleton row: O = v, dQ = dK = 0 exactly.  Constant V: dQ = dK = 0.
    Zero query, non-causal: uniform attention, O = mean(V), LSE = ln N."""
    rng = np.random.default_rng(17)
    q, k, v, u = _rand_case(rng, 1, 8)
    ex = _exact_head(q, k, v, u, True, 0.5)
    assert np.array_equal(ex["O"], v)
    assert np.abs(ex["dQ"]).max() == 0.0 and np.abs(ex["dK"]).max() == 0.0
    assert ex["LSE"][0] == pytest.approx(0.5 * q[0] @ k[0], rel=1e-14)
    q, k, v, u = _rand_case(rng, 33, 8, kbias=4.0)
    v[:] = rng.standard_normal(8)[None, :]
    ex = _exact_head(q, k, v, u, True, 0.5)
    assert np.abs(ex["dQ"]).max() < 1e-13 and np.abs(ex["dK"]).max() < 1e-13
    q = np.zeros_like(q)
    _, k, v, u = _rand_case(rng, 33, 8)
    ex = _exact_head(q, k, v, u, False, 0.5)
    assert np.allclose(ex["O"], v.mean(axis=0)[None, :], atol=1e-14)
    assert np.allclose(ex["LSE"], np.log(33), atol=1e-14)


# -------------------------------------------------- independent second reference

@pytest.mark.parametrize("N,d,causal,kbias", [(128, 64, True, 8.0), (77, 64, False, 4.0),
                                               (200, 128, True, 4.0), (1, 64, True, 0.0)])
def test_cross_reference_agreement(N, d, causal, kbias):
    """Centered VJP vs explicit softmax-Jacobian VJP agree within
    1e-10 + 1e-9 ||target|| (synthetic-suite appendix, 'References')."""
    rng = np.random.default_rng(N * 7 + d)
    q, k, v, u = _rand_case(rng, N, d, kbias=kbias)
    q, k, v, u = (oracle.widen_bf16(S.f32_to_bf16_bits(t)) for t in (q, k, v, u))
    alpha = 1 / np.sqrt(d)
    ex = _exact_head(q, k, v, u, causal, alpha)
    jr = oracle.jacobian_reference(q, k, v, u, causal, alpha)
    for n, ref in zip(("O", "LSE", "dQ", "dK", "dV"), jr):
        tol = 1e-10 + 1e-9 * np.linalg.norm(ex[n])
        assert np.linalg.norm(ex[n] - ref) <= tol, n


def test_oracle_batched_heads_match_single_heads():
    w = S.WORKLOADS[1].with_shape(B=2, H=3, N=40)
    x = S.make_inputs(w, 5)
    full = oracle.exact(x["q"], x["k"], x["v"], x["do"], True, w.scale)
    sub = S.make_inputs(w, 5, heads=[(1, 2)])
    one = oracle.exact(sub["q"], sub["k"], sub["v"], sub["do"], True, w.scale)
    for n in ("O", "LSE", "dQ", "dK", "dV"):
        assert np.array_equal(full[n][1, 2], one[n][0, 0])


def test_rel_l2_metric():
    t = np.array([3.0, 4.0])
    assert oracle.rel_l2(t * 1.01, t) == pytest.approx(1.0)
    assert oracle.rel_l2(t, t) == 0.0


# ------------------------------------------------------ grouped-query attention

def test_gqa_decimal_directional_derivative():
    """Grouped-query attention: L = sum over query heads of sum(O_h * dO_h) with
    the key/value head shared.  Its directional derivative from the 50-digit
    brute force equals <grad, direction> from the oracle, which pins the sum of
    every query head's contribution into the shared dK, dV (Section 3.2)."""
    rng = np.random.default_rng(21)
    Hq, N, d, alpha = 3, 4, 3, 0.8
    q = rng.standard_normal((Hq, N, d))
    k = rng.standard_normal((N, d)) + 1.5 * rng.standard_normal(d)[None, :]
    v = rng.standard_normal((N, d))
    u = rng.standard_normal((Hq, N, d))
    ex = oracle.exact(q[None], k[None, None], v[None, None], u[None], True, alpha)
    dq_dir = rng.standard_normal((Hq, N, d))
    dk_dir, dv_dir = rng.standard_normal((N, d)), rng.standard_normal((N, d))
    h = decimal.Decimal("1e-15")
    Lp = Lm = decimal.Decimal(0)
    for hh in range(Hq):
        dirs = (dq_dir[hh], dk_dir, dv_dir)
        Lp += _decimal_forward(q[hh], k, v, u[hh], True, alpha, dirs=dirs, h=h)[2]
        Lm += _decimal_forward(q[hh], k, v, u[hh], True, alpha, dirs=dirs, h=-h)[2]
    fd = float((Lp - Lm) / (2 * h))
    an = float(np.sum(ex["dQ"][0] * dq_dir) + np.sum(ex["dK"][0, 0] * dk_dir)
               + np.sum(ex["dV"][0, 0] * dv_dir))
    # FP64 rounding over three heads stays near 1e-12; a dropped head or a
    # wrong key/value head would be off by O(0.1).
    assert abs(fd - an) <= 1e-11 * max(1.0, abs(an))


def test_gqa_conservation_and_per_head_identity():
    """Per key/value head, sum_j dk_j = 0 (each query head's rows of dS sum to
    zero) and sum_j dv_j = sum over its query heads and rows of dO; each query
    head's O, LSE, dQ are those of multi-head attention against the shared K, V."""
    rng = np.random.default_rng(8)
    B, Hq, Hkv, N, d = 2, 4, 2, 11, 4
    q = rng.standard_normal((B, Hq, N, d))
    k = rng.standard_normal((B, Hkv, N, d)) + 3.0
    v = rng.standard_normal((B, Hkv, N, d))
    u = rng.standard_normal((B, Hq, N, d))
    for causal in (True, False):
        ex = oracle.exact(q, k, v, u, causal, 0.6)
        G = Hq // Hkv
        for b in range(B):
            for j in range(Hkv):
                assert np.abs(ex["dK"][b, j].sum(axis=0)).max() < 1e-12 * (1 + np.abs(ex["dK"][b, j]).max())
                want = u[b, j * G:(j + 1) * G].sum(axis=(0, 1))
                assert np.allclose(ex["dV"][b, j].sum(axis=0), want, rtol=0, atol=1e-12)
                for g in range(G):
                    h = j * G + g
                    one = _exact_head(q[b, h], k[b, j], v[b, j], u[b, h], causal, 0.6)
                    for n in ("O", "LSE", "dQ"):
                        assert np.array_equal(ex[n][b, h], one[n])


# ------------------------------------------------------- packed sequences

def _decimal_packed_loss(q, k, v, u, seg, causal, alpha, G, dirs=None, h=None, prec=40):
    """L = sum O*u over packed heads by direct softmax in decimal arithmetic,
    with the visibility written as a mask over the whole packed axis: key j is
    visible to query i iff seg[i] == seg[j] (and j <= i when causal).  Query
    head hq reads key/value head hq // G.  Returns (O, LSE, L)."""
    ctx = decimal.Context(prec=prec)
    D = lambda x: ctx.create_decimal(repr(float(x)))  # noqa: E731
    Hq, T, d = q.shape

    def lift(x, dx):
        out = [[[D(x[a, i, c]) for c in range(d)] for i in range(T)] for a in range(x.shape[0])]
        if dx is not None:
            out = [[[out[a][i][c] + h * D(dx[a, i, c]) for c in range(d)] for i in range(T)]
                   for a in range(x.shape[0])]
        return out

    dq_, dk_, dv_ = dirs if dirs is not None else (None, None, None)
    Qd, Kd, Vd = lift(q, dq_), lift(k, dk_), lift(v, dv_)
    a = D(alpha)
    O = np.zeros(q.shape)
    LSE = np.zeros((Hq, T))
    Ltot = D(0)
    for hq in range(Hq):
        hk = hq // G
        for i in range(T):
            vis = [j for j in range(T) if seg[j] == seg[i] and (not causal or j <= i)]
            s = [a * sum((Qd[hq][i][c] * Kd[hk][j][c] for c in range(d)), D(0)) for j in vis]
            e = [ctx.exp(x) for x in s]
            Z = sum(e, D(0))
            LSE[hq, i] = float(ctx.ln(Z))
            for c in range(d):
                oc = sum((e[n] * Vd[hk][j][c] for n, j in enumerate(vis)), D(0)) / Z
                O[hq, i, c] = float(oc)
                Ltot += oc * D(u[hq, i, c])
    return O, LSE, Ltot


@pytest.mark.parametrize("causal", [True, False])
def test_packed_oracle_matches_masked_brute_force(causal):
    """exact_varlen (per-sequence slices) against a brute force over the whole
    packed axis with a sequence mask: forward values and the directional
    derivative of L = sum O*dO, with grouped-query heads, empty and singleton
    sequences."""
    rng = np.random.default_rng(21)
    lens = [3, 0, 1, 4, 2]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    T, d, Hq, Hkv, alpha = int(cu[-1]), 3, 2, 1, 0.8
    seg = np.repeat(np.arange(len(lens)), lens)
    q = rng.standard_normal((Hq, T, d)) * 1.5
    k = rng.standard_normal((Hkv, T, d)) + 2.0 * rng.standard_normal(d)
    v = rng.standard_normal((Hkv, T, d))
    u = rng.standard_normal((Hq, T, d))
    ex = oracle.exact_varlen(q, k, v, u, cu, causal, alpha)
    O, LSE, _ = _decimal_packed_loss(q, k, v, u, seg, causal, alpha, Hq // Hkv)
    assert np.allclose(ex["O"], O, rtol=0, atol=1e-13)
    assert np.allclose(ex["LSE"], LSE, rtol=0, atol=1e-13)
    dirs = (rng.standard_normal(q.shape), rng.standard_normal(k.shape), rng.standard_normal(v.shape))
    h = decimal.Decimal("1e-15")
    _, _, Lp = _decimal_packed_loss(q, k, v, u, seg, causal, alpha, Hq // Hkv, dirs=dirs, h=h)
    _, _, Lm = _decimal_packed_loss(q, k, v, u, seg, causal, alpha, Hq // Hkv, dirs=dirs, h=-h)
    fd = float((Lp - Lm) / (2 * h))
    an = float(sum(np.sum(g * dd) for g, dd in zip((ex["dQ"], ex["dK"], ex["dV"]), dirs)))
    assert abs(fd - an) <= 1e-10 * max(1.0, abs(an))
    # a singleton sequence sees only itself: its output is its value row, its
    # query gradient is zero
    one = int(cu[2])
    assert np.array_equal(ex["O"][:, one], np.repeat(v[:, one], Hq // Hkv, axis=0))
    assert np.all(ex["dQ"][:, one] == 0.0)


def _decimal_packed_qk(q, k, v, u, segq, loc_q, segk, loc_k, nq_of, nk_of, causal, alpha, G,
                       dirs=None, h=None, prec=40):
    """Brute force over separate packed query and key axes: key j is visible to
    query i iff they belong to the same sequence s and (without causal) always,
    (with causal) loc_k[j] <= loc_q[i] + nk_s - nq_s.  A query with no visible
    key has O = 0 and LSE = +inf and adds nothing to L = sum O*u."""
    ctx = decimal.Context(prec=prec)
    D = lambda x: ctx.create_decimal(repr(float(x)))  # noqa: E731
    Hq, Tq, d = q.shape
    Tk = k.shape[1]

    def lift(x, dx):
        out = [[[D(x[a, i, c]) for c in range(d)] for i in range(x.shape[1])] for a in range(x.shape[0])]
        if dx is not None:
            out = [[[out[a][i][c] + h * D(dx[a, i, c]) for c in range(d)] for i in range(x.shape[1])]
                   for a in range(x.shape[0])]
        return out

    dq_, dk_, dv_ = dirs if dirs is not None else (None, None, None)
    Qd, Kd, Vd = lift(q, dq_), lift(k, dk_), lift(v, dv_)
    a = D(alpha)
    O = np.zeros(q.shape)
    LSE = np.full((Hq, Tq), np.inf)
    Ltot = D(0)
    for hq in range(Hq):
        hk = hq // G
        for i in range(Tq):
            s = segq[i]
            vis = [j for j in range(Tk) if segk[j] == s
                   and (not causal or loc_k[j] <= loc_q[i] + nk_of[s] - nq_of[s])]
            if not vis:
                continue
            sc = [a * sum((Qd[hq][i][c] * Kd[hk][j][c] for c in range(d)), D(0)) for j in vis]
            e = [ctx.exp(x) for x in sc]
            Z = sum(e, D(0))
            LSE[hq, i] = float(ctx.ln(Z))
            for c in range(d):
                oc = sum((e[n] * Vd[hk][j][c] for n, j in enumerate(vis)), D(0)) / Z
                O[hq, i, c] = float(oc)
                Ltot += oc * D(u[hq, i, c])
    return O, LSE, Ltot


@pytest.mark.parametrize("causal", [True, False])
def test_packed_oracle_separate_query_key_lengths(causal):
    """exact_varlen with separate query and key offsets (causal diagonal
    aligned at the end) against the masked brute force: sequences with more
    keys than queries, more queries than keys (empty causal rows), no keys,
    no queries, and equal lengths; values and the directional derivative of L."""
    rng = np.random.default_rng(33)
    lens = [(3, 5), (4, 2), (0, 3), (2, 0), (1, 1), (3, 3)]
    nq = [a for a, _ in lens]
    nk = [b for _, b in lens]
    cq = np.concatenate([[0], np.cumsum(nq)]).astype(np.int64)
    ck = np.concatenate([[0], np.cumsum(nk)]).astype(np.int64)
    segq = np.repeat(np.arange(len(lens)), nq)
    segk = np.repeat(np.arange(len(lens)), nk)
    loc_q = np.concatenate([np.arange(n) for n in nq])
    loc_k = np.concatenate([np.arange(n) for n in nk])
    Tq, Tk, d, Hq, Hkv, alpha = int(cq[-1]), int(ck[-1]), 3, 2, 1, 0.7
    q = rng.standard_normal((Hq, Tq, d)) * 1.5
    k = rng.standard_normal((Hkv, Tk, d)) + 1.5 * rng.standard_normal(d)
    v = rng.standard_normal((Hkv, Tk, d))
    u = rng.standard_normal((Hq, Tq, d))
    ex = oracle.exact_varlen(q, k, v, u, cq, causal, alpha, cu_seqlens_k=ck)
    G = Hq // Hkv
    O, LSE, _ = _decimal_packed_qk(q, k, v, u, segq, loc_q, segk, loc_k, nq, nk, causal, alpha, G)
    assert np.allclose(ex["O"], O, rtol=0, atol=1e-13)
    fin = np.isfinite(LSE)
    assert np.array_equal(np.isfinite(ex["LSE"]), fin)
    assert np.allclose(ex["LSE"][fin], LSE[fin], rtol=0, atol=1e-13)
    empty = ~fin[0]
    if causal:
        assert empty.any(), "the (4, 2) sequence has empty causal rows"
    assert np.all(ex["dQ"][:, empty] == 0.0) and np.all(ex["O"][:, empty] == 0.0)
    dirs = (rng.standard_normal(q.shape), rng.standard_normal(k.shape), rng.standard_normal(v.shape))
    hh = decimal.Decimal("1e-15")
    _, _, Lp = _decimal_packed_qk(q, k, v, u, segq, loc_q, segk, loc_k, nq, nk, causal, alpha, G,
                                  dirs=dirs, h=hh)
    _, _, Lm = _decimal_packed_qk(q, k, v, u, segq, loc_q, segk, loc_k, nq, nk, causal, alpha, G,
                                  dirs=dirs, h=-hh)
    fd = float((Lp - Lm) / (2 * hh))
    an = float(sum(np.sum(g * dd) for g, dd in zip((ex["dQ"], ex["dK"], ex["dV"]), dirs)))
    assert abs(fd - an) <= 1e-10 * max(1.0, abs(an))


@pytest.mark.parametrize("kbias", [0.0, 16.0])
def test_sampled_rows_and_keys_match_full_oracle(kbias):
    """oracle.sampled (numpy, per row / per key) against the full C oracle on a
    causal head of 300 tokens: rows at the start, tile edges and the end, and
    the last 9 keys."""
    from oracle import sampled
    rng = np.random.default_rng(31)
    N, d = 300, 64
    q = rng.standard_normal((N, d))
    k = rng.standard_normal((N, d)) + kbias * rng.standard_normal(d)
    v = rng.standard_normal((N, d))
    u = rng.standard_normal((N, d))
    alpha = 0.125
    ex = oracle.exact(q[None], k[None], v[None], u[None], True, alpha)
    rows = [0, 1, 63, 64, 150, 299]
    r = sampled.exact_rows(q, k, v, u, rows, alpha)
    for name in ("O", "dQ"):
        ref = ex[name][0][rows]
        assert np.abs(r[name] - ref).max() <= 1e-12 * max(1.0, np.abs(ref).max()), name
    assert np.abs(r["LSE"] - ex["LSE"][0][rows]).max() <= 1e-12 * max(1.0, np.abs(ex["LSE"]).max())
    kk = sampled.exact_last_keys(q, k, v, u, 9, alpha)
    for name in ("dK", "dV"):
        ref = ex[name][0][N - 9:]
        assert np.abs(kk[name] - ref).max() <= 1e-12 * max(1.0, np.abs(ref).max()), name
