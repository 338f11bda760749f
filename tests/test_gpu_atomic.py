"""The backward with Algorithm 1's own schedule (gpa_attn_bwd_atomic: one
key-major pass with FP32 atomic accumulation of the query-side sums, then in
gproj mode the key-correction pass) against the two-pass backward
(gpa_attn_bwd) and the FP64 oracle, in every mode.

The key-major pass runs the key pass's own code for dV (and, in plain and
gproj_q mode, for dK) with D and the tile statistics formed by the query
pass's code, so those outputs must equal gpa_attn_bwd's bit for bit.  The
atomic sums (A, and in the GProj modes B, rho, m) hold the same BF16 products
as the two-pass schedule's register sums, in an order that varies between
runs; the gproj dK takes dK^acc and C from two separate FP32 accumulators
where the two-pass schedule folds them into one.  Those outputs must meet the
two-pass accuracy against the FP64 oracle (within 2 %) and differ from the
two-pass outputs by at most a tenth of that error.
"""
import numpy as np
import pytest
import torch

import oracle
import synthetic as S

import _gpu as G

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


@pytest.fixture(scope="module")
def gpa():
    import paper_2609_34272_amd as gpa
    gpa.lib()
    return gpa


@pytest.mark.parametrize("mode", ["plain", "gproj_q", "gproj"])
@pytest.mark.parametrize("B,H,N,d,causal", [
    (1, 2, 200, 64, True), (1, 1, 1, 64, True), (2, 1, 65, 128, True), (1, 2, 130, 64, False),
    (1, 1, 100, 128, False), (1, 2, 64, 64, False), (1, 16, 4096, 64, True)])
def test_atomic_schedule_matches_two_pass(gpa, B, H, N, d, causal, mode):
    w = S.Workload("atomic", B, H, N, d, causal=causal, k_bias_std=4.0,
                   do_std=0.01 if N == 4096 else 1.0)
    x = S.make_inputs(w, 2000 if N == 4096 else 60 + N, workers=16)
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    tag = f"{mode} {B}x{H}x{N}x{d} causal={causal}"
    print(f"[atomic] {tag}", flush=True)
    o, lse = gpa.attn_fwd(q, k, v, causal, w.scale)
    ref = gpa.attn_bwd(q, k, v, o, lse, u, mode, causal, w.scale)
    got = gpa.attn_bwd_atomic(q, k, v, o, lse, u, mode, causal, w.scale)
    torch.cuda.synchronize()
    assert torch.equal(got[2], ref[2]), (tag, "dV")
    exact = ["dK"] if mode != "gproj" else []
    for name in exact:
        assert torch.equal(got[1], ref[1]), (tag, name)
    ex = oracle.exact(x["q"], x["k"], x["v"], x["do"], causal, w.scale)
    if N == 1:
        assert np.abs(G.to_host(got[0])).max() <= 1e-6
        assert np.abs(G.to_host(got[1])).max() <= 1e-6
        return
    for i, name in ((0, "dQ"), (1, "dK")):
        if name in exact:
            continue
        e_ref = G.rel_l2(G.to_host(ref[i]), ex[name])
        e_got = G.rel_l2(G.to_host(got[i]), ex[name])
        e_order = G.rel_l2(G.to_host(got[i]), G.to_host(ref[i]))
        G.log(f"[atomic {tag}] {name} rel-L2 {e_got:.4f}% (two-pass {e_ref:.4f}%), "
              f"between the two {e_order:.4f}%")
        assert e_order <= 0.1 * e_ref, (tag, name, e_order, e_ref)
        assert e_got <= 1.02 * e_ref + 1e-3, (tag, name, e_got, e_ref)
