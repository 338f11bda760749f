"""Failure and sanitizer-style tests of the HIP path (through the C ABI).

Guard regions: every input, output and the workspace lives inside a larger
buffer whose leading and trailing 4 KiB hold a sentinel byte.  After ragged,
non-causal, grouped-query and packed calls (unequal query/key counts, empty
sequences) the sentinels must be untouched (no write outside a buffer), the
inputs unchanged, the outputs free of the NaN pattern they were filled with
(every output element written), and the results bitwise those of ordinary
allocations with a zeroed workspace (a workspace full of NaN bytes on entry
changes nothing).

Non-finite inputs: a NaN or an infinity in one row of Q, K, V or dO must
reach every output row whose exact value depends on it (as a NaN or an
infinity), may also reach the rows that depend on the other rows of the same
64-row tile (the diagonal tile multiplies masked probabilities, exactly 0,
into the tile's operands, and 0 x NaN is NaN), and must leave every other row
bitwise equal to a run on clean inputs; the other head is untouched.
"""
import numpy as np
import pytest
import torch

import synthetic as S

import _gpu as G

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU"),
              pytest.mark.filterwarnings("ignore::RuntimeWarning")]

MODES = ("plain", "gproj_q", "gproj")
GUARD = 4096
SENTINEL = 0xA5


@pytest.fixture(scope="module")
def gpa():
    import paper_2609_34272_amd as gpa
    gpa.lib()
    return gpa


class Guarded:
    """A device buffer of nbytes between two sentinel-filled guard regions."""

    def __init__(self, nbytes, fill=0xFF, data=None):
        self.n = int(nbytes)
        self.buf = torch.full((2 * GUARD + max(self.n, 1),), SENTINEL, dtype=torch.uint8,
                              device="cuda:0")
        inner = self.buf[GUARD:GUARD + self.n]
        if data is not None:
            inner.copy_(data.contiguous().view(torch.uint8).reshape(-1))
        else:
            inner.fill_(fill)
        assert (self.ptr % 256) == 0

    @property
    def ptr(self):
        return self.buf.data_ptr() + GUARD

    def tensor(self, dtype, shape):
        return self.buf[GUARD:GUARD + self.n].view(dtype).view(shape)

    def guards_intact(self):
        return bool((self.buf[:GUARD] == SENTINEL).all()) and bool(
            (self.buf[GUARD + self.n:] == SENTINEL).all())


def _g(t):
    return Guarded(t.numel() * t.element_size(), data=t)


def _check_guards(bufs, tag):
    torch.cuda.synchronize()
    for name, b in bufs.items():
        assert b.guards_intact(), (tag, name, "wrote outside its buffer")


def _nan_free(t):
    return not bool(torch.isnan(t.float()).any())


@pytest.mark.parametrize("B,Hq,Hkv,N,d,causal", [
    (1, 3, 3, 200, 64, True), (2, 1, 1, 65, 128, False), (1, 6, 2, 129, 64, True),
    (1, 2, 2, 1, 128, True)])
def test_dense_calls_stay_inside_their_buffers(gpa, B, Hq, Hkv, N, d, causal):
    L = gpa.lib()
    w = S.Workload("guard", B, Hq, N, d, causal=causal, k_bias_std=4.0, do_std=1.0, Hkv=Hkv)
    x = S.make_inputs(w, 31 + N)
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    tag = f"dense {B}x{Hq}/{Hkv}x{N}x{d} causal={causal}"
    ins = {"q": _g(q), "k": _g(k), "v": _g(v), "do": _g(u)}
    o_ref, lse_ref = gpa.attn_fwd(q, k, v, causal, w.scale)
    out = {"o": Guarded(q.numel() * 2), "lse": Guarded(B * Hq * N * 4)}
    st = L.gpa_attn_fwd_gqa(ins["q"].ptr, ins["k"].ptr, ins["v"].ptr, out["o"].ptr,
                            out["lse"].ptr, B, Hq, Hkv, N, d, int(causal), w.scale, None)
    assert st == 0, L.gpa_last_error()
    _check_guards({**ins, **out}, tag + " fwd")
    o = out["o"].tensor(torch.bfloat16, q.shape)
    lse = out["lse"].tensor(torch.float32, lse_ref.shape)
    assert torch.equal(o, o_ref) and torch.equal(lse, lse_ref), tag
    ins.update({"o": _g(o_ref), "lse": _g(lse_ref)})
    for m, code in gpa.MODES.items():
        ref = gpa.attn_bwd(q, k, v, o_ref, lse_ref, u, m, causal, w.scale,
                           workspace=torch.zeros(gpa.attn_bwd_workspace_bytes(B, Hq, N, d, m, Hkv),
                                                 dtype=torch.uint8, device="cuda:0"))
        wsb = gpa.attn_bwd_workspace_bytes(B, Hq, N, d, m, Hkv)
        outs = {"dq": Guarded(q.numel() * 2), "dk": Guarded(k.numel() * 2),
                "dv": Guarded(v.numel() * 2), "ws": Guarded(wsb)}
        st = L.gpa_attn_bwd_gqa(ins["q"].ptr, ins["k"].ptr, ins["v"].ptr, ins["o"].ptr,
                                ins["lse"].ptr, ins["do"].ptr, outs["dq"].ptr, outs["dk"].ptr,
                                outs["dv"].ptr, B, Hq, Hkv, N, d, int(causal), w.scale, code,
                                outs["ws"].ptr, wsb, None)
        assert st == 0, L.gpa_last_error()
        _check_guards({**ins, **outs}, f"{tag} bwd {m}")
        for name, r, shape in (("dq", ref[0], q.shape), ("dk", ref[1], k.shape),
                               ("dv", ref[2], v.shape)):
            t = outs[name].tensor(torch.bfloat16, shape)
            assert _nan_free(t), (tag, m, name, "not fully written")
            assert torch.equal(t, r), (tag, m, name)
    for name, src in (("q", q), ("k", k), ("v", v), ("do", u), ("o", o_ref), ("lse", lse_ref)):
        assert torch.equal(ins[name].tensor(src.dtype, src.shape), src), (tag, name, "input changed")


@pytest.mark.parametrize("causal", [True, False])
def test_packed_calls_stay_inside_their_buffers(gpa, causal):
    """Packed sequences with their own key counts (more and fewer keys than
    queries, empty sequences on either side), grouped heads."""
    L = gpa.lib()
    nq = [0, 70, 1, 129, 64, 3]
    nk = [5, 70, 130, 129, 0, 3]
    Hq, Hkv, d = 4, 2, 64
    cq = np.concatenate([[0], np.cumsum(nq)]).astype(np.int32)
    ck = np.concatenate([[0], np.cumsum(nk)]).astype(np.int32)
    tq, tk = int(cq[-1]), int(ck[-1])
    rng = np.random.default_rng(8)
    mk = lambda H, T: G.to_dev(S.f32_to_bf16_bits(rng.standard_normal((H, T, d)).astype(np.float32)))  # noqa: E731
    q, u = mk(Hq, tq), mk(Hq, tq)
    k, v = mk(Hkv, tk), mk(Hkv, tk)
    cu_q = torch.from_numpy(cq).to("cuda:0")
    cu_k = torch.from_numpy(ck).to("cuda:0")
    scale = 0.125
    mq, mkk = max(nq), max(nk)
    o_ref, lse_ref = gpa.attn_fwd_varlen(q, k, v, cu_q, mq, causal, scale, cu_seqlens_k=cu_k,
                                         max_seqlen_k=mkk)
    ins = {"q": _g(q), "k": _g(k), "v": _g(v), "do": _g(u), "cu_q": _g(cu_q), "cu_k": _g(cu_k)}
    out = {"o": Guarded(q.numel() * 2), "lse": Guarded(Hq * tq * 4)}
    st = L.gpa_attn_fwd_varlen(ins["q"].ptr, ins["k"].ptr, ins["v"].ptr, out["o"].ptr,
                               out["lse"].ptr, ins["cu_q"].ptr, ins["cu_k"].ptr, len(nq), tq, tk,
                               Hq, Hkv, mq, mkk, d, int(causal), scale, None)
    assert st == 0, L.gpa_last_error()
    _check_guards({**ins, **out}, "packed fwd")
    o = out["o"].tensor(torch.bfloat16, q.shape)
    lse = out["lse"].tensor(torch.float32, lse_ref.shape)
    assert _nan_free(o) and _nan_free(lse)
    assert torch.equal(o, o_ref) and torch.equal(lse, lse_ref)
    ins.update({"o": _g(o_ref), "lse": _g(lse_ref)})
    for m, code in gpa.MODES.items():
        wsb = gpa.attn_bwd_varlen_workspace_bytes(len(nq), tq, Hq, Hkv, mq, d, m, tk, mkk)
        ref = gpa.attn_bwd_varlen(q, k, v, o_ref, lse_ref, u, cu_q, mq, m, causal, scale,
                                  workspace=torch.zeros(wsb, dtype=torch.uint8, device="cuda:0"),
                                  cu_seqlens_k=cu_k, max_seqlen_k=mkk)
        outs = {"dq": Guarded(q.numel() * 2), "dk": Guarded(k.numel() * 2),
                "dv": Guarded(v.numel() * 2), "ws": Guarded(wsb)}
        st = L.gpa_attn_bwd_varlen(ins["q"].ptr, ins["k"].ptr, ins["v"].ptr, ins["o"].ptr,
                                   ins["lse"].ptr, ins["do"].ptr, outs["dq"].ptr, outs["dk"].ptr,
                                   outs["dv"].ptr, ins["cu_q"].ptr, ins["cu_k"].ptr, len(nq), tq,
                                   tk, Hq, Hkv, mq, mkk, d, int(causal), scale, code,
                                   outs["ws"].ptr, wsb, None)
        assert st == 0, L.gpa_last_error()
        _check_guards({**ins, **outs}, f"packed bwd {m}")
        for name, r, t in (("dq", ref[0], q), ("dk", ref[1], k), ("dv", ref[2], v)):
            got = outs[name].tensor(torch.bfloat16, t.shape)
            assert _nan_free(got), (m, name, "not fully written")
            assert torch.equal(got, r), (m, name)
    for name, src in (("q", q), ("k", k), ("v", v), ("do", u), ("o", o_ref), ("lse", lse_ref),
                      ("cu_q", cu_q), ("cu_k", cu_k)):
        assert torch.equal(ins[name].tensor(src.dtype, src.shape), src), (name, "input changed")


# ------------------------------------------------------- non-finite inputs

def _deps(src, r, N):
    """Rows of each output whose exact value depends on row r of input src
    (one causal head of N tokens)."""
    every, ge, le = set(range(N)), set(range(r, N)), set(range(r + 1))
    return {"Q": {"O": {r}, "LSE": {r}, "dQ": {r}, "dK": le, "dV": le},
            "K": {"O": ge, "LSE": ge, "dQ": ge, "dK": every, "dV": every},
            "V": {"O": ge, "LSE": set(), "dQ": ge, "dK": every, "dV": set()},
            "dO": {"O": set(), "LSE": set(), "dQ": {r}, "dK": le, "dV": le}}[src]


def _bad_rows(t):
    t = t.float()
    bad = ~torch.isfinite(t)
    if bad.dim() == 4:  # [B, H, N, d] -> rows; LSE is already [B, H, N]
        bad = bad.any(dim=-1)
    return bad.cpu().numpy()


@pytest.mark.parametrize("src,row,value", [
    ("Q", 100, float("nan")), ("K", 150, float("nan")), ("V", 70, float("nan")),
    ("V", 70, float("inf")), ("dO", 200, float("nan")), ("dO", 200, float("-inf"))])
def test_non_finite_input_propagation(gpa, src, row, value):
    N, d = 300, 64
    w = S.Workload("nonfinite", 1, 2, N, d, k_bias_std=4.0, do_std=1.0)
    x = S.make_inputs(w, 404)
    clean = {n: G.to_dev(x[n]) for n in ("q", "k", "v", "do")}
    dirty = {n: t.clone() for n, t in clean.items()}
    key = {"Q": "q", "K": "k", "V": "v", "dO": "do"}[src]
    dirty[key][0, 1, row, 5] = value

    def run(t):
        o, lse = gpa.attn_fwd(t["q"], t["k"], t["v"], True, w.scale)
        res = {"O": o, "LSE": lse}
        for m in MODES:
            res[m] = gpa.attn_bwd(t["q"], t["k"], t["v"], o, lse, t["do"], m, True, w.scale)
        torch.cuda.synchronize()
        return res

    a, b = run(clean), run(dirty)
    dep = _deps(src, row, N)
    t0 = row // 64 * 64
    spill = {}
    for r2 in range(t0, min(t0 + 64, N)):
        for n, rows in _deps(src, r2, N).items():
            spill.setdefault(n, set()).update(rows)
    summary = []
    for n, ta, tb in [("O", a["O"], b["O"]), ("LSE", a["LSE"], b["LSE"])] + [
            (f"{m}.{nm}", a[m][i], b[m][i]) for m in MODES for i, nm in enumerate(("dQ", "dK", "dV"))]:
        base = n.split(".")[-1]
        assert not _bad_rows(ta).any(), (n, "clean run not finite")
        bad = _bad_rows(tb)
        assert not bad[0, 0].any(), (src, n, "the other head was reached")
        got = set(np.flatnonzero(bad[0, 1]).tolist())
        assert dep[base] <= got, (src, n, "dependent rows stayed finite", sorted(dep[base] - got)[:8])
        assert got <= spill[base], (src, n, "reached rows outside the tile rule",
                                    sorted(got - spill[base])[:8])
        keep = np.array([i not in got for i in range(N)])
        ba, bb = ta[0, 1][torch.from_numpy(keep).to(ta.device)], tb[0, 1][torch.from_numpy(keep).to(tb.device)]
        assert torch.equal(ba, bb), (src, n, "a row outside the affected set changed")
        assert torch.equal(ta[0, 0], tb[0, 0]), (src, n, "the other head changed")
        summary.append(f"{n} {len(got)} (exact {len(dep[base])})")
    G.log(f"[non-finite {src} row {row} = {value}] rows reached: " + ", ".join(summary))
