"""The library's kernel timing (gpa_profile_enable / gpa_profile_read) records
each kernel between events that its own launch places at the kernel's start
and end.  Over a run of back-to-back backward calls, the per-kernel durations
therefore sum to at most the wall time of the run on the stream, and to most
of it (with the timing events the gap between dependent launches is ~6 us,
against ~130 us per call at 16 heads of 4096 tokens); every launch is
counted once per call."""
import numpy as np
import pytest
import torch

import synthetic as S

import _gpu as G

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


@pytest.mark.parametrize("mode,kernels", [("plain", ("bwd_dq", "bwd_dkdv")),
                                          ("gproj", ("bwd_dq", "bwd_dkdv"))])
def test_kernel_times_add_up_to_the_call(mode, kernels):
    import paper_2609_34272_amd as gpa
    w = S.Workload("timing", 1, 16, 4096, 64, causal=True, k_bias_std=4.0, do_std=0.01)
    x = S.make_inputs(w, 77, workers=16)
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    o, lse = gpa.attn_fwd(q, k, v, True, w.scale)
    ws = torch.empty(gpa.attn_bwd_workspace_bytes(1, 16, 4096, 64, mode), dtype=torch.uint8,
                     device=q.device)
    fn = lambda: gpa.attn_bwd(q, k, v, o, lse, u, mode, True, w.scale, workspace=ws)  # noqa: E731
    for _ in range(5):
        fn()
    torch.cuda.synchronize()
    calls = 50
    gpa.profile_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(calls):
        fn()
    e1.record()
    torch.cuda.synchronize()
    prof = gpa.profile_read()
    gpa.profile_enable(False)
    wall = e0.elapsed_time(e1)
    for name in kernels:
        assert prof[name][1] == calls, (name, prof[name])
    busy = sum(prof[name][0] for name in kernels)
    G.log(f"[timing {mode}] kernels {busy:.3f} ms of {wall:.3f} ms on the stream "
          f"({100 * busy / wall:.1f} %)")
    assert busy <= wall * 1.001, (busy, wall)
    assert busy >= 0.75 * wall, (busy, wall)
