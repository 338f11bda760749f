"""The library's calls can be captured in a HIP graph (torch.cuda.CUDAGraph):
they only enqueue kernels on the caller's stream, with no allocation, memset
or synchronisation of their own.  A captured forward + backward, replayed
several times with other eager work and synchronisations between replays,
gives bitwise the eager results on every replay (dense grouped-query and
packed layouts, all three backward modes)."""
import numpy as np
import pytest
import torch

import synthetic as S
from synthetic import suite

import _gpu as G

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

MODES = ("plain", "gproj_q", "gproj")


@pytest.fixture(scope="module")
def gpa():
    import paper_2609_34272_amd as gpa
    gpa.lib()
    return gpa


def _capture_and_check(step, eager_noise):
    """Capture step() (which reads only preallocated inputs and workspaces),
    replay it 3 times with eager work in between, compare with eager runs."""
    ref = [t.clone() for t in step()]
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(2):
            step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = step()
    torch.cuda.synchronize()
    for rep in range(3):
        eager_noise()
        torch.cuda.synchronize()
        for t in out:
            t.zero_()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(out, ref):
            assert np.array_equal(G.bits(a) if a.dtype == torch.bfloat16 else a.cpu().numpy(),
                                  G.bits(b) if b.dtype == torch.bfloat16 else b.cpu().numpy()), rep


def test_graph_dense_gqa(gpa):
    w = S.WORKLOADS[6].with_shape(N=777)
    x = S.make_inputs(w, 31)
    G.log(f"graph capture dense: {w.name} N=777")
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    B, H, N, d = q.shape
    Hkv = k.shape[1]
    ws = {m: torch.empty(gpa.attn_bwd_workspace_bytes(B, H, N, d, m, Hkv), dtype=torch.uint8,
                         device=q.device) for m in MODES}
    noise_in = torch.randn(1 << 20, device=q.device)

    def step():
        o, lse = gpa.attn_fwd(q, k, v, True, w.scale)
        outs = [o, lse]
        for m in MODES:
            outs += list(gpa.attn_bwd(q, k, v, o, lse, u, m, True, w.scale, workspace=ws[m]))
        return outs

    _capture_and_check(step, lambda: noise_in.mul_(1.0001).sum())


def test_graph_packed(gpa):
    case = next(c for c in suite.CASES if c.name == "fewer queries than keys")
    x = suite.make_case(case)
    G.log(f"graph capture packed: case {case.index:03d} {case.name}")
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    cu = torch.tensor(case.cu, dtype=torch.int32, device="cuda:0")
    cu_k = torch.tensor(case.cu_k, dtype=torch.int32, device="cuda:0")
    kw = dict(cu_seqlens_k=cu_k, max_seqlen_k=case.max_seqlen_k)
    ws = torch.empty(gpa.attn_bwd_varlen_workspace_bytes(
        len(case.lens), case.total, case.Hq, case.Hkv, case.max_seqlen, case.d, "gproj",
        case.total_k, case.max_seqlen_k), dtype=torch.uint8, device="cuda:0")
    noise_in = torch.randn(1 << 18, device="cuda:0")

    def step():
        o, lse = gpa.attn_fwd_varlen(q, k, v, cu, case.max_seqlen, True, case.scale, **kw)
        return [o, lse, *gpa.attn_bwd_varlen(q, k, v, o, lse, u, cu, case.max_seqlen, "gproj",
                                             True, case.scale, workspace=ws, **kw)]

    _capture_and_check(step, lambda: noise_in.mul_(0.9999).sum())
