"""The plain backward as one key-major pass with FP32 atomic dQ
(gpa_attn_bwd_atomic) against the two-pass plain backward and the FP64 oracle.

It runs the key pass's own code for dK and dV with D and the tile statistics
formed by the query pass's code, so dK and dV must equal gpa_attn_bwd's plain
outputs bit for bit.  dQ = BF16(alpha A) with A summed by atomics in an order
that varies between runs: it must meet the plain backward's accuracy (same
error against the FP64 oracle within 2 %, since both contract the same BF16
t with the same FP32 accumulator, only in another order) and differ from the
two-pass dQ by at most a tenth of that error.
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


@pytest.mark.parametrize("B,H,N,d,causal", [
    (1, 2, 200, 64, True), (1, 1, 1, 64, True), (2, 1, 65, 128, True), (1, 2, 130, 64, False),
    (1, 16, 4096, 64, True)])
def test_atomic_plain_matches_two_pass_plain(gpa, B, H, N, d, causal):
    w = S.Workload("atomic", B, H, N, d, causal=causal, k_bias_std=4.0,
                   do_std=0.01 if N == 4096 else 1.0)
    x = S.make_inputs(w, 2000 if N == 4096 else 60 + N, workers=16)
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    o, lse = gpa.attn_fwd(q, k, v, causal, w.scale)
    ref = gpa.attn_bwd(q, k, v, o, lse, u, "plain", causal, w.scale)
    got = gpa.attn_bwd_atomic(q, k, v, o, lse, u, causal, w.scale)
    torch.cuda.synchronize()
    tag = f"{B}x{H}x{N}x{d} causal={causal}"
    assert torch.equal(got[1], ref[1]), (tag, "dK")
    assert torch.equal(got[2], ref[2]), (tag, "dV")
    ex = oracle.exact(x["q"], x["k"], x["v"], x["do"], causal, w.scale)
    if N == 1:
        assert np.abs(G.to_host(got[0])).max() <= 1e-6
        return
    e_ref = G.rel_l2(G.to_host(ref[0]), ex["dQ"])
    e_got = G.rel_l2(G.to_host(got[0]), ex["dQ"])
    # the two summation orders differ by FP32 rounding of A, a small fraction
    # of the plain dQ's own error (its uncorrected row-mass leak)
    e_order = G.rel_l2(G.to_host(got[0]), G.to_host(ref[0]))
    G.log(f"[atomic plain {tag}] dQ rel-L2 {e_got:.4f}% (two-pass {e_ref:.4f}%), "
          f"between the two {e_order:.4f}%")
    assert e_order <= 0.1 * e_ref, (tag, e_order, e_ref)
    assert e_got <= 1.02 * e_ref + 1e-3, (tag, e_got, e_ref)
