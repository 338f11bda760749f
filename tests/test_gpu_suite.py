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


def run_case(gpa, case, x):
    """Forward and the three backward modes; host float64 results on the
    packed axis, plus BF16 bit patterns for the identity checks."""
    out = {}
    if case.packed:
        q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
        cu = torch.tensor(case.cu, dtype=torch.int32, device="cuda:0")
        o, lse = gpa.attn_fwd_varlen(q, k, v, cu, case.max_seqlen, case.causal, case.scale)
        res = {m: gpa.attn_bwd_varlen(q, k, v, o, lse, u, cu, case.max_seqlen, m, case.causal,
                                      case.scale, return_stats=True) for m in MODES}
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
    x = suite.make_case(case)
    ex = oracle.exact_varlen(x["q"], x["k"], x["v"], x["do"], case.cu, case.causal, case.scale)
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
    # operand mass of every row (every row here sees at least its own key)
    mass = out["gproj"]["m"]
    assert np.all((mass > 0.99) & (mass < 1.01)), (mass.min(), mass.max())
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
