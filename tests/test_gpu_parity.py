"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

Accuracy gates (the hot-path contract): in gproj mode each of dQ, dK, dV has
full-tensor relative L2 error <= 1.0 % against the exact FP64 VJP and at most
2x the error of the FP32 attention baseline run on the same inputs; plain mode
shows the blow-up on biased-key inputs.  Semantics gates: the -24 witness, the
single-key identities, bitwise mode identities and bitwise reproducibility.
Agreement with the step-by-step BF16 model of Algorithm 1 is checked with
tolerances derived from where the two may legitimately differ (FP32
accumulation order).
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import synthetic as S
from oracle import algo_model as M

import _gpu as G

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU"),
              pytest.mark.filterwarnings("ignore::RuntimeWarning")]

MODES = ("plain", "gproj_q", "gproj")
NAMES = ("dQ", "dK", "dV")


@pytest.fixture(scope="module")
def gpa():
    import paper_2609_34272_amd as gpa
    gpa.lib()
    return gpa


def run_all(gpa, x, causal, scale):
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    o, lse = gpa.attn_fwd(q, k, v, causal, scale)
    out = {"O": o, "LSE": lse}
    for m in MODES:
        dq, dk, dv, st = gpa.attn_bwd(q, k, v, o, lse, u, m, causal, scale, return_stats=True)
        out[m] = dict(dQ=dq, dK=dk, dV=dv, stats={n: t.clone() for n, t in st.items()})
    fo, flse, fdq, fdk, fdv = gpa.fp32_attn(q, k, v, u, causal, scale)
    out["fp32"] = dict(O=fo, LSE=flse, dQ=fdq, dK=fdk, dV=fdv)
    torch.cuda.synchronize()
    return out


def errors_vs_exact(out, ex):
    e = {"O": G.rel_l2(G.to_host(out["O"]), ex["O"])}
    for m in MODES + ("fp32",):
        e[m] = {n: G.rel_l2(G.to_host(out[m][n]), ex[n]) for n in NAMES}
    e["fp32"]["O"] = G.rel_l2(G.to_host(out["fp32"]["O"]), ex["O"])
    lse_scale = max(1.0, float(np.abs(ex["LSE"]).max()))
    e["fp32"]["LSE"] = float(np.abs(G.to_host(out["fp32"]["LSE"]) - ex["LSE"]).max()) / lse_scale
    return e


# The FP32 baseline's own error.  Its only BF16 step is the final cast of each
# output, whose relative error is at most 2^-9 (0.195 %) per element and hence
# over a whole tensor; 0.25 % leaves 0.055 % for its FP32 arithmetic on these
# workloads (logits of moderate size).  Its LSE is FP32 throughout.
FP32_MAX_PCT = 0.25
FP32_LSE_REL = 1e-5


def check_accuracy_gates(e, tag, blowup_ratio=3.0, fp32_not_worse=False):
    G.log(f"[{tag}] O {e['O']:.4f}% | " + " | ".join(
        f"{m}: " + "/".join(f"{e[m][n]:.4f}" for n in NAMES) for m in MODES + ("fp32",))
        + f" | fp32 O {e['fp32']['O']:.4f}% LSE rel {e['fp32']['LSE']:.2e}")
    for n in NAMES:
        assert e["gproj"][n] <= 1.0, (tag, "gproj", n, e["gproj"][n])
        assert e["gproj"][n] <= 2.0 * e["fp32"][n], (tag, "gproj vs fp32", n)
    # the FP32 baseline is gated on its own, so the 2x rule cannot pass vacuously
    for n in ("O",) + NAMES:
        assert e["fp32"][n] <= FP32_MAX_PCT, (tag, "fp32", n, e["fp32"][n])
    assert e["fp32"]["LSE"] <= FP32_LSE_REL, (tag, "fp32 LSE", e["fp32"]["LSE"])
    if fp32_not_worse:
        for n in NAMES:
            assert e["fp32"][n] <= e["gproj"][n], (tag, "fp32 worse than gproj", n)
        assert e["fp32"]["O"] <= e["O"], (tag, "fp32 O worse than the BF16 forward")
    assert e["gproj_q"]["dQ"] <= 1.0
    assert e["O"] <= 0.5
    if blowup_ratio:
        assert e["plain"]["dQ"] >= blowup_ratio * e["gproj"]["dQ"], (tag, "no blow-up")


def check_mode_identities(out):
    b = lambda m, n: G.bits(out[m][n])  # noqa: E731
    assert np.array_equal(b("plain", "dK"), b("gproj_q", "dK"))
    assert np.array_equal(b("plain", "dV"), b("gproj_q", "dV"))
    assert np.array_equal(b("gproj_q", "dQ"), b("gproj", "dQ"))
    assert np.array_equal(b("gproj_q", "dV"), b("gproj", "dV"))
    for n in ("rho", "m", "lambda"):
        assert torch.equal(out["gproj_q"]["stats"][n], out["gproj"]["stats"][n])


# ------------------------------------------------------------------ witness

def test_witness_minus24(gpa, golden_dir):
    """Section 3.4 / appendix A: plain returns -24 in the zero coordinate,
    GProj returns exactly 0 (Section 5.2)."""
    with open(os.path.join(golden_dir, "witness_minus24.json")) as f:
        w = json.load(f)
    pb, hand = w["printed_by_paper"], w["derived_by_oracle"]
    N, d = 4, 64
    q = np.zeros((1, 1, N, d), np.float32); k = np.zeros_like(q); v = np.zeros_like(q); u = np.zeros_like(q)
    k[0, 0, :, :2] = pb["k"]; v[0, 0, :, :2] = pb["v"]; u[0, 0, 3, :2] = pb["u"]
    x = {n: S.f32_to_bf16_bits(a) for n, a in zip(("q", "k", "v", "do"), (q, k, v, u))}
    out = run_all(gpa, x, True, pb["alpha"])
    O = G.to_host(out["O"])[0, 0]
    assert list(O[3, :2]) == pb["o"]
    plain = G.to_host(out["plain"]["dQ"])[0, 0]
    assert plain[3, 0] == pb["plain_dq_first_coordinate"]
    assert list(plain[3, :2]) == hand["plain_dq_bf16"]
    for m in ("gproj_q", "gproj"):
        dq = G.to_host(out[m]["dQ"])[0, 0]
        assert dq[3, 0] == 0.0
        assert list(dq[3, :2]) == hand["gproj_dq_bf16"]
        assert out[m]["stats"]["lambda"][0, 0, 3].item() == -pb["eta"]
    for m in MODES:
        assert np.abs(G.to_host(out[m]["dK"])).max() == 0.0
        assert np.all(G.to_host(out[m]["dV"])[0, 0, :, :2] == 0.25)
    G.log(f"[witness] plain dq3={plain[3, :2]} gproj dq3={G.to_host(out['gproj']['dQ'])[0, 0, 3, :2]}")


# ----------------------------------------------------- single-key identities

def test_single_key_rows(gpa):
    """Appendix 'Prescribed FMA cases': all 64 query coordinates c*2^k
    (c in {3,5,7}, k = 0..15), all key coordinates 1, lengths 1 and 128.  The
    first causal row has one legal key, so o_0 = v_0 and dq_0 = 0 exactly; the
    subtract-before-scale forward must restore both in all 96 cases.  Values and
    upstream derivatives are small integers, so u.v is exact in FP32 whatever the
    summation order (D and dP then agree exactly)."""
    rng = np.random.default_rng(0)
    d = 64
    for N in (1, 128):
        for cval in (3, 5, 7):
            for kexp in range(16):
                q = np.full((1, 1, N, d), cval * 2.0 ** kexp, np.float32)
                k = np.ones((1, 1, N, d), np.float32)
                v = rng.integers(-4, 5, (1, 1, N, d)).astype(np.float32)
                u = np.zeros((1, 1, N, d), np.float32)
                u[0, 0, 0] = rng.integers(-3, 4, d)
                x = {n: S.f32_to_bf16_bits(a) for n, a in zip(("q", "k", "v", "do"), (q, k, v, u))}
                qd, kd, vd, ud = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
                o, lse = gpa.attn_fwd(qd, kd, vd, True, 0.125)
                assert np.array_equal(G.bits(o)[0, 0, 0], x["v"][0, 0, 0]), (N, cval, kexp)
                for m in MODES:
                    dq, dk, dv = gpa.attn_bwd(qd, kd, vd, o, lse, ud, m, True, 0.125)
                    assert np.abs(G.to_host(dq)[0, 0, 0]).max() == 0.0, (N, cval, kexp, m)


def test_historical_fma_forward_one_key_rows(gpa):
    """Diagnostic (not the GProj path): the historical FMA exponent rounding
    (eq. historical-fma) on the same 96 single-key constructions.  The first
    row's output must equal the paper's scalar model BF16(BF16(z) v / z) (eq.
    historical-one-key) bit for bit in every case, some cases must violate
    o0 = v0, and the FA3-SBS forward on the same inputs must not."""
    rng = np.random.default_rng(0)
    d = 64
    viol = 0
    mism = []
    for N in (1, 128):
        for cval in (3, 5, 7):
            for kexp in range(16):
                q = np.full((1, 1, N, d), cval * 2.0 ** kexp, np.float32)
                k = np.ones((1, 1, N, d), np.float32)
                v = rng.integers(-4, 5, (1, 1, N, d)).astype(np.float32)
                x = {n: S.f32_to_bf16_bits(a) for n, a in zip(("q", "k", "v"), (q, k, v))}
                qd, kd, vd = (G.to_dev(x[n]) for n in ("q", "k", "v"))
                o, _ = gpa.attn_fwd_fma(qd, kd, vd, True, 0.125)
                o0 = G.to_host(o)[0, 0, 0].astype(np.float32)
                want = M.historical_fma_one_key(64 * cval * 2 ** kexp, 0.125, v[0, 0, 0])
                if not np.array_equal(o0, want):
                    mism.append((N, cval, kexp))
                viol += int(not np.array_equal(o0, v[0, 0, 0]))
                osbs, _ = gpa.attn_fwd(qd, kd, vd, True, 0.125)
                assert np.array_equal(G.bits(osbs)[0, 0, 0], x["v"][0, 0, 0])
    G.log(f"[historical FMA forward] one-key violations {viol}/96, model mismatches {mism}")
    assert not mism
    assert viol > 0


# ---------------------------------------------------- tiny workload (cfg 1)

@pytest.mark.parametrize("seed", S.seeds_for(1, 8))
def test_tiny_workload(gpa, seed):
    w = S.WORKLOADS[1]
    x = S.make_inputs(w, seed)
    out = run_all(gpa, x, w.causal, w.scale)
    ex = oracle.exact(x["q"], x["k"], x["v"], x["do"], w.causal, w.scale)
    e = errors_vs_exact(out, ex)
    check_accuracy_gates(e, f"tiny seed {seed}", fp32_not_worse=True)
    record_seed(w.name, seed, e)
    check_mode_identities(out)
    lse_err = np.abs(G.to_host(out["LSE"]) - ex["LSE"]).max()
    assert lse_err <= 1e-4 * max(1.0, np.abs(ex["LSE"]).max())
    # against the BF16 model of Algorithm 1, fed the GPU's own O and LSE
    q, k, v, u = (S.bf16_bits_to_f32(x[n][0, 0]) for n in ("q", "k", "v", "do"))
    o = G.to_host(out["O"])[0, 0].astype(np.float32)
    lse = G.to_host(out["LSE"])[0, 0].astype(np.float32)
    Om, Lm, _ = M.sbs_forward(q, k, v, w.causal, w.scale)
    dO = G.rel_l2(o, Om)
    msg = [f"O {dO:.4f}"]
    assert dO <= 0.3
    for m in MODES:
        mq, mk, mv, st = M.backward(q, k, v, o, lse, u, w.causal, w.scale, m)
        for n, ref in zip(NAMES, (mq, mk, mv)):
            r = G.rel_l2(G.to_host(out[m][n])[0, 0], ref)
            msg.append(f"{m}.{n} {r:.4f}")
            # the plain dQ is dominated by the leak alpha*rho*mu_k, whose rho
            # is a sum of cast errors; a few order-dependent flips move it.
            assert r <= (0.25 * e["plain"]["dQ"] if (m == "plain" and n == "dQ") else 0.1), (m, n, r)
        gm = out[m]["stats"]
        if m != "plain":
            assert np.allclose(gm["m"].cpu().numpy()[0, 0], st["m"], rtol=0, atol=2e-3)
    G.log(f"[tiny seed {seed}] vs model: " + " ".join(msg))
    mass = out["gproj"]["stats"]["m"].cpu().numpy()
    assert mass.min() > 0.99 and mass.max() < 1.01


# ------------------------------------- long heads, sampled exact outputs

@pytest.mark.parametrize("N,d", [(262144, 64), (131035, 128)])
def test_long_head_sampled_outputs(gpa, N, d):
    """One causal head of 2^18 tokens (d = 64) and of 2^17 - 37 tokens
    (d = 128), far beyond the full oracle: O, LSE and dQ at sampled rows and
    dK, dV at the last 8 keys against oracle.sampled, to the same gates; mode
    identities on the whole tensors."""
    from oracle import sampled
    w = S.Workload("long head", 1, 1, N, d, k_bias_std=8.0, do_std=0.01)
    x = S.make_inputs(w, 9100 + d)
    G.log(f"long head N={N} d={d}")
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    o, lse = gpa.attn_fwd(q, k, v, True, w.scale)
    res = {m: gpa.attn_bwd(q, k, v, o, lse, u, m, True, w.scale) for m in MODES}
    torch.cuda.synchronize()
    assert torch.equal(res["gproj"][0], res["gproj_q"][0])
    assert torch.equal(res["gproj_q"][1], res["plain"][1])
    assert torch.equal(res["gproj"][2], res["plain"][2])
    rows = [0, 1, 63, 64, 4095, N // 2, N - 65, N - 1]
    h = lambda n: x[n][0, 0]  # noqa: E731
    ref = sampled.exact_rows(h("q"), h("k"), h("v"), h("do"), rows, w.scale)
    keys = sampled.exact_last_keys(h("q"), h("k"), h("v"), h("do"), 8, w.scale)
    idx = torch.tensor(rows, device=q.device)
    e = {"O": G.rel_l2(G.to_host(o[0, 0, idx]), ref["O"])}
    lse_err = float(np.abs(G.to_host(lse[0, 0, idx]) - ref["LSE"]).max())
    for m in MODES:
        dq, dk, dv = res[m]
        e[m] = (G.rel_l2(G.to_host(dq[0, 0, idx]), ref["dQ"]),
                G.rel_l2(G.to_host(dk[0, 0, N - 8:]), keys["dK"]),
                G.rel_l2(G.to_host(dv[0, 0, N - 8:]), keys["dV"]))
    G.log(f"[long head N={N} d={d}] O {e['O']:.4f}% LSE abs {lse_err:.2e} " +
          " ".join(f"{m} dQ/dK/dV {a:.3f}/{b:.3f}/{c:.3f}" for m, (a, b, c) in
                   ((m, e[m]) for m in MODES)))
    assert e["O"] <= 0.5
    assert lse_err <= 1e-4 * max(1.0, float(np.abs(ref["LSE"]).max()))
    assert all(x_ <= 1.0 for x_ in e["gproj"]), e["gproj"]


# --------------------------------------- FA3 / FA3-SBS / GProj ordering

def _sharp_errors(gpa, q_std):
    w = S.Workload("sharp", 1, 2, 1024, 64, q_std=q_std, k_bias_std=64.0, do_std=1.0)
    x = S.make_inputs(w, 777)
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    ex = oracle.exact(x["q"], x["k"], x["v"], x["do"], True, w.scale)
    e = {}
    for fwd_name, fwd in (("sbs", gpa.attn_fwd), ("fma", gpa.attn_fwd_fma)):
        o, lse = fwd(q, k, v, True, w.scale)
        for m in ("plain", "gproj"):
            dq, dk, dv = gpa.attn_bwd(q, k, v, o, lse, u, m, True, w.scale)
            torch.cuda.synchronize()
            e[fwd_name, m] = {n: G.rel_l2(G.to_host(t), ex[n])
                              for n, t in (("O", o), ("dQ", dq), ("dK", dk), ("dV", dv))}
    fo, _, fdq, fdk, fdv = gpa.fp32_attn(q, k, v, u, True, w.scale)
    torch.cuda.synchronize()
    e["fp32", "-"] = {n: G.rel_l2(G.to_host(t), ex[n])
                      for n, t in (("O", fo), ("dQ", fdq), ("dK", fdk), ("dV", fdv))}
    G.log(f"[sharp regime, query spread {q_std:g}, max |scaled logit| "
          f"{float(np.abs(ex['LSE']).max()):.3g}] " + " | ".join(
              f"{f}+{m}: " + "/".join(f"{e[f, m][n]:.3f}" for n in ("O", "dQ", "dK", "dV"))
              for f, m in e))
    return e


def test_fa3_ordering_in_the_sharp_regime(gpa):
    """The paper's accuracy ordering (Results, accuracy table, Table 1): with the
    historical FMA exponent rounding in the forward (FA3), the plain backward's
    dQ and dK errors are far above those with the subtract-before-scale forward
    (FA3-SBS), which are far above GProj's.  It shows in the regime the paper
    measures in (near one-hot rows, a large common key offset).

    At the paper's logit scale (~10^4: query spread 300, key bias spread 64,
    N = 1024, two heads) GProj meets the contract's rule against the fused FP32
    baseline.  At ten times that scale (query spread 3000) the ordering is
    starker; there the backward's P = exp(s - LSE) (FA3's formula, which GProj
    keeps) carries the FP32 resolution of an LSE of ~2e5, while the fused FP32
    baseline rebuilds P from the row maximum and inverse normaliser, so GProj
    sits at up to 3x its error there (still within 1 %)."""
    paper = _sharp_errors(gpa, 300.0)
    gp, f32 = paper["sbs", "gproj"], paper["fp32", "-"]
    for n in ("dQ", "dK", "dV"):
        assert gp[n] <= 1.0 and gp[n] <= 2.0 * f32[n], (n, gp[n], f32[n])
    assert paper["sbs", "plain"]["dQ"] > 10.0 * gp["dQ"]
    e = _sharp_errors(gpa, 3000.0)
    fa3, sbs, gp, f32 = e["fma", "plain"], e["sbs", "plain"], e["sbs", "gproj"], e["fp32", "-"]
    assert gp["dQ"] <= 3.0 * f32["dQ"] and gp["dK"] <= 3.0 * f32["dK"]
    assert fa3["O"] > 2.0 * sbs["O"]
    assert fa3["dQ"] > 2.0 * sbs["dQ"] and sbs["dQ"] > 10.0 * gp["dQ"]
    assert fa3["dK"] > 2.0 * sbs["dK"] and sbs["dK"] > gp["dK"]
    assert max(gp["dQ"], gp["dK"], gp["dV"]) <= 1.0


# ------------------------------------------------------- key-bias sweep

def test_key_bias_sweep(gpa):
    """The theorem on forward repair versus projection (Section 4): the plain
    backward's dQ error grows linearly in the common key offset relative to
    the key spread, while GProj's does not move.  Sweep the per-channel key
    bias spread 0, 4, 16, 64 at N = 1024 (two heads)."""
    errs = {}
    for kb in (0.0, 4.0, 16.0, 64.0):
        w = S.Workload("bias sweep", 1, 2, 1024, 64, k_bias_std=kb, do_std=1.0)
        x = S.make_inputs(w, 5150)
        out = run_all(gpa, x, True, w.scale)
        ex = oracle.exact(x["q"], x["k"], x["v"], x["do"], True, w.scale)
        e = errors_vs_exact(out, ex)
        check_accuracy_gates(e, f"key bias {kb}", blowup_ratio=0)
        errs[kb] = (e["plain"]["dQ"], e["gproj"]["dQ"])
    G.log("[key bias sweep] plain / gproj dQ %: " +
          ", ".join(f"{kb:g}: {p:.3f} / {g:.3f}" for kb, (p, g) in errs.items()))
    plain = [errs[kb][0] for kb in (0.0, 4.0, 16.0, 64.0)]
    assert all(a < b for a, b in zip(plain, plain[1:])), plain
    assert 3.0 <= plain[3] / plain[2] <= 6.0, plain          # linear: 64 / 16 = 4
    assert all(g <= 0.5 for _, g in errs.values())
    assert max(g for _, g in errs.values()) <= 1.2 * min(g for _, g in errs.values())


# --------------------------------------------------------- ragged shapes

RAGGED = [(1, 1, 1, 64, True), (1, 2, 17, 64, True), (2, 1, 65, 128, True),
          (1, 1, 127, 64, False), (1, 3, 200, 128, True), (1, 1, 64, 64, False),
          (2, 2, 129, 64, True)]


@pytest.mark.parametrize("B,H,N,d,causal", RAGGED)
def test_ragged_shapes(gpa, B, H, N, d, causal):
    w = S.Workload("ragged", B, H, N, d, causal=causal, k_bias_std=4.0, do_std=1.0)
    x = S.make_inputs(w, 77 + N)
    out = run_all(gpa, x, causal, w.scale)
    ex = oracle.exact(x["q"], x["k"], x["v"], x["do"], causal, w.scale)
    check_mode_identities(out)
    if N == 1:
        # singleton rows: exact dQ = dK = 0; GProj's dQ is exactly zero
        assert np.abs(G.to_host(out["gproj"]["dQ"])).max() == 0.0
        for m in MODES:
            assert np.abs(G.to_host(out[m]["dQ"])).max() <= 1e-6
            assert np.abs(G.to_host(out[m]["dK"])).max() <= 1e-6
        assert np.array_equal(G.bits(out["O"]), x["v"])
        return
    e = errors_vs_exact(out, ex)
    check_accuracy_gates(e, f"ragged {B}x{H}x{N}x{d} causal={causal}", blowup_ratio=0)


def test_determinism(gpa):
    w = S.WORKLOADS[1].with_shape(H=2, N=300)
    x = S.make_inputs(w, 5)
    a = run_all(gpa, x, True, w.scale)
    b = run_all(gpa, x, True, w.scale)
    assert torch.equal(a["O"], b["O"]) and torch.equal(a["LSE"], b["LSE"])
    for m in MODES:
        for n in NAMES:
            assert torch.equal(a[m][n], b[m][n]), (m, n)


# ------------------------------------------------------- full-size workloads

# Per-seed errors of the workloads run under the eight-seed protocol (seeds
# 1000 k + s, s = 0..7; the paper reports medians over its eight captures).
SEED_LOG = {}


def record_seed(workload, seed, e):
    SEED_LOG.setdefault(workload, {})[seed] = e


def _full(gpa, index, seed, heads=None):
    import _rowtile as RT
    w = S.WORKLOADS[index]
    G.log(f"[workload {w.name} seed {seed}] generating inputs")
    x = S.make_inputs(w, seed, heads=None, workers=16)
    G.log(f"[workload {w.name} seed {seed}] running GPU")
    out = run_all(gpa, x, w.causal, w.scale)
    if heads is None:
        sel = lambda a: a  # noqa: E731
        xs = x
    else:
        idx = tuple(np.array(h) for h in zip(*heads))
        sel = lambda a: a[idx][:, None]  # noqa: E731
        xs = {n: sel(a) for n, a in x.items()}
    G.log(f"[workload {w.name} seed {seed}] running oracle on "
          f"{'all' if heads is None else len(heads)} heads")
    ex = oracle.exact(xs["q"], xs["k"], xs["v"], xs["do"], w.causal, w.scale)
    host = {"O": sel(G.to_host(out["O"]))}
    for m in MODES + ("fp32",):
        host[m] = {n: sel(G.to_host(out[m][n])) for n in NAMES}
    host["fp32"]["O"] = sel(G.to_host(out["fp32"]["O"]))
    host["fp32"]["LSE"] = sel(G.to_host(out["fp32"]["LSE"])[..., None])[..., 0]
    e = {"O": G.rel_l2(host["O"], ex["O"])}
    for m in MODES + ("fp32",):
        e[m] = {n: G.rel_l2(host[m][n], ex[n]) for n in NAMES}
    e["fp32"]["O"] = G.rel_l2(host["fp32"]["O"], ex["O"])
    e["fp32"]["LSE"] = float(np.abs(host["fp32"]["LSE"] - ex["LSE"]).max()) / max(
        1.0, float(np.abs(ex["LSE"]).max()))
    check_accuracy_gates(e, f"{w.name} seed {seed}", fp32_not_worse=heads is None)
    check_mode_identities(out)
    # localised defects: every row and every 64-row tile against the median
    rt = {"O": RT.check(host["O"], ex["O"], "O")}
    for m in MODES + ("fp32",):
        for n in NAMES:
            rt[f"{m}.{n}"] = RT.check(host[m][n], ex[n], f"{w.name} {m}.{n}",
                                      rows=f"{m}.{n}" not in RT.UNCORRECTED)
    rt["fp32.O"] = RT.check(host["fp32"]["O"], ex["O"], "fp32.O")
    G.log(f"[{w.name} seed {seed}] max/median error ratios, rows (bound {RT.K_ROW:g}; "
          f"not bounded for {', '.join(sorted(RT.UNCORRECTED))}) / 64-row tiles "
          f"(bound {RT.K_TILE:g}): " + ", ".join(f"{k_} {r:.1f}/{t:.2f}" for k_, (r, t) in rt.items()))
    mass = out["gproj"]["stats"]["m"].cpu().numpy()
    assert mass.min() > 0.99 and mass.max() < 1.01
    G.log(f"[{w.name}] operand mass m in [{mass.min():.6f}, {mass.max():.6f}]")
    return e


@pytest.mark.parametrize("seed", S.seeds_for(2, 8))
def test_full_h16_n4096_d64(gpa, seed):
    record_seed("h16_n4096_d64", seed, _full(gpa, 2, seed))


@pytest.mark.parametrize("seed", S.seeds_for(3, 8))
def test_full_h16_n4096_d128(gpa, seed):
    record_seed("h16_n4096_d128", seed, _full(gpa, 3, seed))


def test_full_h16_n16384_d64_head_subset(gpa):
    _full(gpa, 4, 4000, heads=[(0, 0), (0, 15)])


def test_full_b8_h32_n8192_d128_head_subset(gpa):
    _full(gpa, 5, 5000, heads=[(0, 0), (7, 31)])


def test_seed_protocol_medians():
    """Per-seed and median errors of the eight-seed workloads (logged); every
    seed has passed its gates in the tests above.  Skipped when those tests
    were not all run in this session."""
    want = {"tiny": S.seeds_for(1, 8), "h16_n4096_d64": S.seeds_for(2, 8),
            "h16_n4096_d128": S.seeds_for(3, 8)}
    if any(sorted(SEED_LOG.get(k, {})) != v for k, v in want.items()):
        pytest.skip("the eight-seed tests did not all run in this session")
    for wl, seeds in want.items():
        for m in MODES + ("fp32",):
            rows = []
            for n in (("O",) if m == "fp32" else ()) + NAMES:
                vals = [SEED_LOG[wl][s][m][n] for s in seeds]
                rows.append(f"{n} median {np.median(vals):.4f} per seed "
                            + " ".join(f"{v:.4f}" for v in vals))
            G.log(f"[seed protocol {wl}] {m}: " + "; ".join(rows))
        o = [SEED_LOG[wl][s]["O"] for s in seeds]
        G.log(f"[seed protocol {wl}] O median {np.median(o):.4f} per seed "
              + " ".join(f"{v:.4f}" for v in o))
        med = {n: np.median([SEED_LOG[wl][s]["gproj"][n] for s in seeds]) for n in NAMES}
        assert all(v <= 1.0 for v in med.values()), (wl, med)


# ------------------------------------ both passes form the same t and r

@pytest.mark.parametrize("causal", [True, False])
def test_both_passes_form_the_same_t_and_r(gpa, causal):
    """The query-major and key-major passes rebuild P, t and r independently.
    With d = 128, N = 64, Q = [I | X] and K = [Y | I] the logits q_i.k_j =
    y_j[i] + x_i[j] are arbitrary, yet every product the kernels form reads
    single values of t and r exactly: A_i (query pass) holds t_ij at column
    64 + j, dK^acc_j (key pass) holds t_ij at column i, and with dO = [I | 0]
    dV_j holds r_ij at column i.  With alpha = 1/8 every cast is exact, so
    plain dQ and dK must give the same t bit for bit, and gproj_q's dQ =
    BF16(fl32[alpha (t - lambda r)]) must match the key pass's r."""
    N, d, alpha = 64, 128, 0.125
    rng = np.random.default_rng(12)
    eye = np.eye(N, dtype=np.float32)
    X = S.bf16_bits_to_f32(S.f32_to_bf16_bits(rng.standard_normal((N, N)).astype(np.float32)))
    Y = S.bf16_bits_to_f32(S.f32_to_bf16_bits(rng.standard_normal((N, N)).astype(np.float32)))
    q = np.concatenate([eye, X], axis=1)[None, None]
    k = np.concatenate([Y, eye], axis=1)[None, None]
    v = rng.standard_normal((1, 1, N, d)).astype(np.float32)
    u = np.concatenate([eye, np.zeros((N, N), np.float32)], axis=1)[None, None]
    x = {n: S.f32_to_bf16_bits(a) for n, a in zip(("q", "k", "v", "do"), (q, k, v, u))}
    qd, kd, vd, ud = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    o, lse = gpa.attn_fwd(qd, kd, vd, causal, alpha)
    dq, dk, dv = gpa.attn_bwd(qd, kd, vd, o, lse, ud, "plain", causal, alpha)
    dq_g, _, dv_g, st = gpa.attn_bwd(qd, kd, vd, o, lse, ud, "gproj_q", causal, alpha,
                                     return_stats=True)
    torch.cuda.synchronize()
    DQ, DK, DV = (G.to_host(t)[0, 0].astype(np.float32) for t in (dq, dk, dv))
    t_query = DQ[:, N:] / np.float32(alpha)          # t_ij from the query pass
    t_key = DK[:, :N].T / np.float32(alpha)          # t_ij from the key pass
    r_key = DV[:, :N].T                              # r_ij from the key pass
    assert np.array_equal(t_query, t_key)
    assert np.count_nonzero(t_query) > N              # a non-trivial pattern
    lam = st["lambda"][0, 0].cpu().numpy().astype(np.float32)
    a32 = np.float32(alpha)
    corr = (lam[:, None] * r_key).astype(np.float32)
    want = (a32 * (t_query - corr).astype(np.float32)).astype(np.float32)
    want_bits = S.f32_to_bf16_bits(want)
    got_bits = G.bits(dq_g)[0, 0][:, N:]
    assert np.array_equal(got_bits, want_bits)
    assert np.array_equal(G.bits(dv_g), G.bits(dv))
    G.log(f"[t and r across passes, causal={causal}] {np.count_nonzero(t_query)} nonzero t, "
          f"{np.count_nonzero(r_key)} nonzero r: identical in both passes")


# ------------------------------------------------------------ maximum size

def test_maximum_size_sampled_heads(gpa):
    """The largest shape the boundary accepts at d = 64: B*H*N*d just under
    2^31 (B = 1, H = 511, N = 65536; 4.3 GB per tensor, ~39 GB on the GPU),
    so every head, row and tile offset of every kernel is exercised near its
    limit.  Heads are independent, so all heads but the first and the last
    are filled with device-side random values and those two with the seeded
    recipe; they are checked at sampled rows (O, LSE, dQ) and at the last 8
    keys (dK, dV) against oracle.sampled, to the same gates as the long-head
    test, and the mode identities hold on the whole tensors."""
    from oracle import sampled
    B, H, N, d = 1, 511, 65536, 64
    assert B * H * N * d < 2 ** 31
    w = S.Workload("maximum size", B, H, N, d, k_bias_std=4.0, do_std=0.01)
    picks = [(0, 0), (0, H - 1)]
    x = S.make_inputs(w, 9600, heads=picks)
    G.log(f"[maximum size] B={B} H={H} N={N} d={d}: filling {B * H * N * d} elements per tensor")
    gen = torch.Generator(device="cuda:0")
    gen.manual_seed(9600)
    t = {}
    for n, sd in (("q", 1.0), ("k", 1.0), ("v", 1.0), ("do", 0.01)):
        a = torch.randn((B, H, N, d), generator=gen, device="cuda:0", dtype=torch.bfloat16)
        if sd != 1.0:
            a.mul_(sd)
        for i, (b, h) in enumerate(picks):
            a[b, h].copy_(G.to_dev(x[n][i, 0]))
        t[n] = a
    o, lse = gpa.attn_fwd(t["q"], t["k"], t["v"], True, w.scale)
    res = {}
    for m in MODES:
        res[m] = gpa.attn_bwd(t["q"], t["k"], t["v"], o, lse, t["do"], m, True, w.scale)
        torch.cuda.synchronize()
        G.log(f"[maximum size] {m} backward done")
    assert torch.equal(res["gproj"][0], res["gproj_q"][0])
    assert torch.equal(res["gproj_q"][1], res["plain"][1])
    assert torch.equal(res["gproj"][2], res["plain"][2])
    rows = [0, 1, 4095, N // 2, N - 65, N - 1]
    idx = torch.tensor(rows, device="cuda:0")
    for i, (b, h) in enumerate(picks):
        hx = lambda n: x[n][i, 0]  # noqa: E731
        ref = sampled.exact_rows(hx("q"), hx("k"), hx("v"), hx("do"), rows, w.scale)
        keys = sampled.exact_last_keys(hx("q"), hx("k"), hx("v"), hx("do"), 8, w.scale)
        e = {"O": G.rel_l2(G.to_host(o[b, h, idx]), ref["O"])}
        lse_err = float(np.abs(G.to_host(lse[b, h, idx]) - ref["LSE"]).max())
        for m in MODES:
            dq, dk, dv = res[m]
            e[m] = (G.rel_l2(G.to_host(dq[b, h, idx]), ref["dQ"]),
                    G.rel_l2(G.to_host(dk[b, h, N - 8:]), keys["dK"]),
                    G.rel_l2(G.to_host(dv[b, h, N - 8:]), keys["dV"]))
        G.log(f"[maximum size head {h}] O {e['O']:.4f}% LSE abs {lse_err:.2e} " +
              " ".join(f"{m} dQ/dK/dV {a:.3f}/{b_:.3f}/{c:.3f}" for m, (a, b_, c) in
                       ((m, e[m]) for m in MODES)))
        assert e["O"] <= 0.5
        assert lse_err <= 1e-4 * max(1.0, float(np.abs(ref["LSE"]).max()))
        assert all(v_ <= 1.0 for v_ in e["gproj"]), e["gproj"]
    del t, o, lse, res
    torch.cuda.empty_cache()
