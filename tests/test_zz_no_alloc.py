"""gpa_attn_bwd_noalloc: the backward with the library's own per-GPU scratch
array instead of a caller workspace, for callers that cannot allocate.

Called through the C ABI with preallocated outputs, it must return bitwise
what gpa_attn_bwd returns with a workspace (the same kernels), on two calls in
a row with the second one smaller (the scratch keeps the first call's
contents, which the second must not depend on), in every mode; a shape whose
workspace exceeds the scratch is rejected before anything is launched.
"""
import ctypes

import pytest
import torch

import synthetic as S

import _gpu as G

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def test_noalloc_matches_workspace_backward_on_consecutive_calls():
    import paper_2609_34272_amd as gpa
    L = gpa.lib()
    cap = L.gpa_attn_bwd_noalloc_max_bytes()
    assert cap >= gpa.attn_bwd_workspace_bytes(1, 16, 4096, 64, "gproj")
    for m, code in gpa.MODES.items():
        for (B, H, N, d, causal) in ((1, 4, 1000, 64, True), (1, 2, 130, 128, False),
                                     (2, 1, 65, 64, True)):
            w = S.Workload("noalloc", B, H, N, d, causal=causal, k_bias_std=4.0, do_std=1.0)
            x = S.make_inputs(w, 900 + N)
            q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
            o, lse = gpa.attn_fwd(q, k, v, causal, w.scale)
            ref = gpa.attn_bwd(q, k, v, o, lse, u, m, causal, w.scale)
            dq, dk, dv = (torch.full_like(q, float("nan")) for _ in range(3))
            G.log(f"[noalloc] mode {m} shape {B}x{H}x{N}x{d} causal={causal}")
            st = L.gpa_attn_bwd_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                        lse.data_ptr(), u.data_ptr(), dq.data_ptr(),
                                        dk.data_ptr(), dv.data_ptr(), B, H, N, d, int(causal),
                                        w.scale, code, torch.cuda.current_stream().cuda_stream)
            assert st == 0, L.gpa_last_error()
            torch.cuda.synchronize()
            for name, a, b in (("dQ", dq, ref[0]), ("dK", dk, ref[1]), ("dV", dv, ref[2])):
                assert torch.equal(a, b), (m, (B, H, N, d), name)


def test_noalloc_rejects_shapes_beyond_its_scratch():
    import paper_2609_34272_amd as gpa
    L = gpa.lib()
    cap = L.gpa_attn_bwd_noalloc_max_bytes()
    B, H, N, d = 1, 64, 65536, 128
    assert gpa.attn_bwd_workspace_bytes(B, H, N, d, "gproj") > cap
    p = ctypes.c_void_p(256)  # never dereferenced: the size check comes first
    st = L.gpa_attn_bwd_noalloc(p, p, p, p, p, p, p, p, p, B, H, N, d, 1, 0.1, 2, None)
    assert st == 3, st  # GPA_EWORKSPACE
    assert b"at most" in L.gpa_last_error()
