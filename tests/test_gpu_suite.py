"""Synthetic numerical suite and packed variable-length sequences on the GPU,
through the C ABI (gpa_attn_fwd_varlen / gpa_attn_bwd_varlen for packed cases,
the dense *_gqa entry points for dense ones), against the FP64 oracle.

The suite's cases (synthetic/suite.py) follow the categories of the paper's
synthetic suite (appendix "Synthetic Numerical Suite").  Its outcome rule is
the paper's: a result fails if its relative L2 error exceeds 5 %, or, where the
exact target tensor is zero, if its absolute error exceeds 1e-6.  GProj must
pass every case; like the paper's it must also leave O and dV byte-identical to
the plain (FA3-SBS) backward and not increase the dK error.  Plain results are
reported, not gated (the paper's FA3-SBS fails its shifted cases).

Packed runs must also equal dense runs of each sequence alone bit for bit:
a sequence of a pack is the same attention problem, solved by the same kernels.
Sequences whose queries and keys differ in number are checked the same way
against the square problem they reduce to (queries padded at the top with
zero rows, or cut to the last nk queries when the leading ones see no key).
"""
import numpy as np
import pytest
import torch

import oracle
from synthetic import suite

import _gpu as G

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU"),
              pytest.mark.filterwarnings("ignore::RuntimeWarning")]

MODES = ("plain", "gproj_q", "gproj")
FAIL_REL_PCT = 5.0
ZERO_ABS = 1e-6


@pytest.fixture(scope="module")
def gpa():
    import paper_2609_34272_amd as gpa
    gpa.lib()
    return gpa


def _dense(a, B):
    """[H, B*N, d] packed axis -> [B, H, N, d]."""
    H, T, d = a.shape
    return np.ascontiguousarray(a.reshape(H, B, T // B, d).transpose(1, 0, 2, 3))


def _packed(t, B):
    """GPU [B, H, N, (d)] -> host float64 [H, B*N, (d)]."""
    a = G.to_host(t)
    if a.ndim == 4:
        return a.transpose(1, 0, 2, 3).reshape(a.shape[1], -1, a.shape[3])
    return a.transpose(1, 0, 2).reshape(a.shape[1], -1)


def key_offsets(case):
    """Keyword arguments for the key side of a packed case."""
    if not case.cross:
        return {}
    return dict(cu_seqlens_k=torch.tensor(case.cu_k, dtype=torch.int32, device="cuda:0"),
                max_seqlen_k=case.max_seqlen_k)


def run_case(gpa, case, x):
    """Forward and the three backward modes; host float64 results on the
    packed axis, plus BF16 bit patterns for the identity checks."""
    out = {}
    if case.packed:
        q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
        cu = torch.tensor(case.cu, dtype=torch.int32, device="cuda:0")
        kw = key_offsets(case)
        o, lse = gpa.attn_fwd_varlen(q, k, v, cu, case.max_seqlen, case.causal, case.scale, **kw)
        res = {m: gpa.attn_bwd_varlen(q, k, v, o, lse, u, cu, case.max_seqlen, m, case.causal,
                                      case.scale, return_stats=True, **kw) for m in MODES}
        torch.cuda.synchronize()
        host = G.to_host
    else:
        B = len(case.lens)
        q, k, v, u = (G.to_dev(_dense(x[n], B)) for n in ("q", "k", "v", "do"))
        o, lse = gpa.attn_fwd(q, k, v, case.causal, case.scale)
        res = {m: gpa.attn_bwd(q, k, v, o, lse, u, m, case.causal, case.scale, return_stats=True)
               for m in MODES}
        torch.cuda.synchronize()
        host = lambda t: _packed(t, B)  # noqa: E731
    out["O"], out["LSE"] = host(o), host(lse)
    out["O_bits"] = G.bits(o)
    for m, (dq, dk, dv, st) in res.items():
        out[m] = dict(dQ=host(dq), dK=host(dk), dV=host(dv), m=host(st["m"]),
                      lam=host(st["lambda"]), rho=host(st["rho"]),
                      bits={n: G.bits(t) for n, t in (("dQ", dq), ("dK", dk), ("dV", dv))})
    return out


def _err(a, t):
    """(relative L2 % or None for a zero target, absolute max error)."""
    den = np.linalg.norm(t)
    return (100.0 * np.linalg.norm(a - t) / den if den > 0 else None), float(np.abs(a - t).max())


def _passes(a, t):
    rel, ab = _err(a, t)
    return ab <= ZERO_ABS if rel is None else rel <= FAIL_REL_PCT


@pytest.mark.parametrize("case", suite.CASES, ids=lambda c: f"{c.index:03d}-{c.name.replace(' ', '_')}")
def test_suite_case(gpa, case):
    G.log(f"suite case {case.index:03d} {case.name}: lens={case.lens[:6]}{'...' if len(case.lens) > 6 else ''} "
          f"packed={case.packed} causal={case.causal} Hq={case.Hq} Hkv={case.Hkv} d={case.d}")
    check_case(gpa, case)


def random_packed_case(r: int) -> suite.SuiteCase:
    """Seeded random packed layout: 1-5 sequences of 0-259 queries, keys of
    the same or their own lengths, causal or not, d = 64 or 128, grouped or
    multi-head; lengths near tile edges are drawn often."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([424242, r])))
    nseq = int(rng.integers(1, 6))

    def lengths():
        edge = rng.choice([0, 1, 63, 64, 65, 127, 128, 129, 191, 192, 193], nseq)
        free = rng.integers(0, 260, nseq)
        return tuple(int(x) for x in np.where(rng.random(nseq) < 0.4, edge, free))

    lens = lengths()
    while max(lens) == 0:
        lens = lengths()
    lens_k = ()
    if rng.random() < 0.6:
        lens_k = lengths()
        while max(lens_k) == 0:
            lens_k = lengths()
    Hq, Hkv = [(4, 2), (2, 2), (4, 1), (8, 2)][int(rng.integers(0, 4))]
    return suite.SuiteCase(1000 + r, f"random packed {r}", "random", lens, packed=True,
                           causal=bool(rng.random() < 0.7), Hq=Hq, Hkv=Hkv,
                           d=128 if rng.random() < 0.25 else 64, lens_k=lens_k)


@pytest.mark.parametrize("r", range(16))
def test_random_packed_layout(gpa, r):
    """Seeded random packings (unequal query/key counts, empty sequences and
    rows, tile-edge lengths) checked like the suite's cases."""
    case = random_packed_case(r)
    G.log(f"random packed {r}: lens={case.lens} lens_k={case.lens_k} causal={case.causal} "
          f"Hq={case.Hq} Hkv={case.Hkv} d={case.d}")
    check_case(gpa, case)


def check_case(gpa, case):
    x = suite.make_case(case)
    ex = oracle.exact_varlen(x["q"], x["k"], x["v"], x["do"], case.cu, case.causal, case.scale,
                             cu_seqlens_k=case.cu_k)
    out = run_case(gpa, case, x)
    report = {}
    for m in ("plain", "gproj"):
        report[m] = {n: _err(out[m][n], ex[n]) for n in ("dQ", "dK", "dV")}
    report["O"] = _err(out["O"], ex["O"])
    G.log(f"  O {report['O']}  plain {report['plain']}  gproj {report['gproj']}")
    # the paper's outcome rule, for GProj
    assert _passes(out["O"], ex["O"]), ("O", report["O"])
    for n in ("dQ", "dK", "dV"):
        assert _passes(out["gproj"][n], ex[n]), ("gproj", n, report["gproj"][n])
    # O and dV byte-identical to the plain backward; mode identities
    b = lambda m, n: out[m]["bits"][n]  # noqa: E731
    assert np.array_equal(b("gproj", "dV"), b("plain", "dV"))
    assert np.array_equal(b("gproj_q", "dV"), b("plain", "dV"))
    assert np.array_equal(b("gproj_q", "dK"), b("plain", "dK"))
    assert np.array_equal(b("gproj", "dQ"), b("gproj_q", "dQ"))
    # the key correction does not increase the dK error
    pk, gk = report["plain"]["dK"], report["gproj"]["dK"]
    if pk[0] is not None:
        assert gk[0] <= 1.05 * pk[0] + 1e-3, (pk, gk)
    else:
        assert gk[1] <= max(1.05 * pk[1], ZERO_ABS), (pk, gk)
    # operand mass of every row that sees a key; a row that sees none is
    # empty: O = 0, LSE = +inf, and m = rho = lambda = 0, dQ = 0 in every mode
    empty = case.empty_rows()
    mass = out["gproj"]["m"][:, ~empty]
    assert np.all((mass > 0.99) & (mass < 1.01)), (mass.min(), mass.max())
    if empty.any():
        assert np.all(out["O"][:, empty] == 0.0)
        assert np.all(np.isposinf(out["LSE"][:, empty]))
        for m in MODES:
            assert np.all(out[m]["dQ"][:, empty] == 0.0), m
        for n in ("m", "rho", "lam"):
            assert np.all(out["gproj"][n][:, empty] == 0.0), n
    assert np.all(np.isfinite(out["LSE"][:, ~empty]))
    # keys no query sees get dK = dV = 0 exactly
    unseen = case.unseen_keys()
    if unseen.any():
        for m in MODES:
            assert np.all(out[m]["dK"][:, unseen] == 0.0) and np.all(out[m]["dV"][:, unseen] == 0.0), m
    if case.name == "singleton":
        assert np.all(out["gproj"]["dQ"] == 0.0)
        assert np.abs(out["gproj"]["dK"]).max() <= ZERO_ABS


def _slice_heads(a, lo, hi):
    return np.ascontiguousarray(a[:, lo:hi])[None]


@pytest.mark.parametrize("idx", [1, 3, 11, 14, 47, 48, 49])
def test_packed_equals_dense_per_sequence(gpa, idx):
    """Each sequence of a pack gives bitwise the results of a dense run on that
    sequence alone (same kernels, same per-problem arithmetic)."""
    case = suite.CASES[idx]
    assert case.packed
    x = suite.make_case(case)
    G.log(f"packed vs dense: case {idx:03d} {case.name}")
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    cu = torch.tensor(case.cu, dtype=torch.int32, device="cuda:0")
    o, lse = gpa.attn_fwd_varlen(q, k, v, cu, case.max_seqlen, case.causal, case.scale)
    pk = {m: gpa.attn_bwd_varlen(q, k, v, o, lse, u, cu, case.max_seqlen, m, case.causal,
                                 case.scale) for m in MODES}
    torch.cuda.synchronize()
    for lo, hi in zip(case.cu[:-1], case.cu[1:]):
        if hi == lo:
            continue
        qd, kd, vd, ud = (G.to_dev(_slice_heads(x[n], lo, hi)) for n in ("q", "k", "v", "do"))
        od, lsed = gpa.attn_fwd(qd, kd, vd, case.causal, case.scale)
        assert np.array_equal(G.bits(od)[0], G.bits(o)[:, lo:hi]), (lo, hi)
        assert torch.equal(lsed[0], lse[:, lo:hi]), (lo, hi)
        for m in MODES:
            dd = gpa.attn_bwd(qd, kd, vd, od, lsed, ud, m, case.causal, case.scale)
            for name, a, p in zip(("dQ", "dK", "dV"), dd, pk[m]):
                assert np.array_equal(G.bits(a)[0], G.bits(p)[:, lo:hi]), (m, name, lo, hi)


CROSS = [c.index for c in suite.CASES if c.cross and c.causal]


@pytest.mark.parametrize("idx", CROSS)
def test_unequal_query_key_equals_square(gpa, idx):
    """A causal sequence with nq queries and nk keys is the square problem on
    its keys with the queries aligned at the end: nq < nk pads the queries at
    the top with nk - nq zero rows of zero upstream gradient, nq > nk keeps
    the last nk queries (the others see no key).  Per-row results (O, LSE,
    dQ) match the square run bit for bit; dK and dV do too when nk - nq is a
    multiple of the 64-row tile (the padding rows add exact zeros, and the
    query tiles then line up)."""
    case = suite.CASES[idx]
    x = suite.make_case(case)
    G.log(f"unequal query/key vs square: case {idx:03d} {case.name}")
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    cu = torch.tensor(case.cu, dtype=torch.int32, device="cuda:0")
    kw = key_offsets(case)
    o, lse = gpa.attn_fwd_varlen(q, k, v, cu, case.max_seqlen, True, case.scale, **kw)
    pk = {m: gpa.attn_bwd_varlen(q, k, v, o, lse, u, cu, case.max_seqlen, m, True, case.scale,
                                 **kw) for m in MODES}
    torch.cuda.synchronize()
    ob, lh = G.bits(o), lse.cpu().numpy()
    pb = {m: [G.bits(t) for t in pk[m]] for m in MODES}
    Hq, d = case.Hq, case.d
    for s in range(len(case.lens)):
        a, b = int(case.cu[s]), int(case.cu[s + 1])
        ka, kb = int(case.cu_k[s]), int(case.cu_k[s + 1])
        nq, nk = b - a, kb - ka
        if nq == 0 or nk == 0:
            continue
        if nq <= nk:
            pad, first = nk - nq, a
            z = np.zeros((Hq, pad, d), np.uint16)
            qs = np.concatenate([z, x["q"][:, a:b]], 1)
            us = np.concatenate([z, x["do"][:, a:b]], 1)
            rows = slice(pad, nk)
        else:
            first = a + nq - nk
            qs, us = x["q"][:, first:b], x["do"][:, first:b]
            rows = slice(0, nk)
        qd, ud = G.to_dev(qs[None]), G.to_dev(us[None])
        kd, vd = G.to_dev(x["k"][None, :, ka:kb]), G.to_dev(x["v"][None, :, ka:kb])
        od, lsed = gpa.attn_fwd(qd, kd, vd, True, case.scale)
        assert np.array_equal(G.bits(od)[0][:, rows], ob[:, first:b]), s
        assert np.array_equal(lsed[0].cpu().numpy()[:, rows], lh[:, first:b]), s
        aligned = (nk - nq) % 64 == 0
        for m in MODES:
            dq, dk, dv = (G.bits(t)[0] for t in gpa.attn_bwd(qd, kd, vd, od, lsed, ud, m, True,
                                                             case.scale))
            assert np.array_equal(dq[:, rows], pb[m][0][:, first:b]), (m, s)
            if aligned:
                assert np.array_equal(dk, pb[m][1][:, ka:kb]), (m, s)
                assert np.array_equal(dv, pb[m][2][:, ka:kb]), (m, s)


def test_packed_reproducible(gpa):
    """Repeated runs of a packed case are bitwise identical."""
    case = suite.CASES[46]
    x = suite.make_case(case)
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    cu = torch.tensor(case.cu, dtype=torch.int32, device="cuda:0")
    runs = []
    for _ in range(2):
        o, lse = gpa.attn_fwd_varlen(q, k, v, cu, case.max_seqlen, case.causal, case.scale)
        g = gpa.attn_bwd_varlen(q, k, v, o, lse, u, cu, case.max_seqlen, "gproj", case.causal,
                                case.scale)
        torch.cuda.synchronize()
        runs.append([G.bits(t) for t in (o, *g)] + [lse.cpu().numpy()])
    for a, b in zip(*runs):
        assert np.array_equal(a, b)


def test_varlen_rejects_bad_arguments(gpa):
    """Validation happens on the host before any launch."""
    case = suite.CASES[1]
    x = suite.make_case(case)
    q, k, v = (G.to_dev(x[n]) for n in ("q", "k", "v"))
    cu = torch.tensor(case.cu, dtype=torch.int32, device="cuda:0")
    with pytest.raises(gpa.GpaError):
        gpa.attn_fwd_varlen(q, k, v, cu, case.total + 1, True, case.scale)  # max_seqlen > total
    with pytest.raises(gpa.GpaError):
        gpa.attn_fwd_varlen(q, k, v, cu, 0, True, case.scale)
    with pytest.raises(ValueError):
        gpa.attn_fwd_varlen(q, k, v, cu.to(torch.int64), case.max_seqlen, True, case.scale)
    with pytest.raises(ValueError):  # keys of their own length need their own offsets
        gpa.attn_fwd_varlen(q, k[:, :-1].contiguous(), v[:, :-1].contiguous(), cu,
                            case.max_seqlen, True, case.scale)
    with pytest.raises(gpa.GpaError):  # the key side's longest run exceeds its total
        gpa.attn_fwd_varlen(q, k, v, cu, case.max_seqlen, True, case.scale, cu_seqlens_k=cu,
                            max_seqlen_k=case.total + 1)
