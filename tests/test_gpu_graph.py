"""The library's calls can be captured in a HIP graph (torch.cuda.CUDAGraph):
they only enqueue kernels on the caller's stream, with no allocation, memset
or synchronisation of their own.  A captured forward + backward, replayed
several times with other eager work and synchronisations between replays,
gives bitwise the eager results on every replay (dense grouped-query and
packed layouts, all three backward modes).  Calls on concurrent side streams
give the default stream's results."""
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


def test_calls_on_side_streams(gpa):
    """Every call is enqueued on the caller's current stream: two problems run
    concurrently on two side streams (each with its own workspace) give
    bitwise the results of the same calls on the default stream."""
    w = S.WORKLOADS[2].with_shape(H=2, N=1500)
    xs = [S.make_inputs(w, s) for s in (71, 72)]
    G.log("side streams: h2 N=1500, two problems")
    dev = torch.device("cuda:0")
    ins = [[G.to_dev(x[n]) for n in ("q", "k", "v", "do")] for x in xs]
    B, H, N, d = ins[0][0].shape

    def run(q, k, v, u, ws):
        o, lse = gpa.attn_fwd(q, k, v, True, w.scale)
        return [o, lse, *gpa.attn_bwd(q, k, v, o, lse, u, "gproj", True, w.scale, workspace=ws)]

    wss = [torch.empty(gpa.attn_bwd_workspace_bytes(B, H, N, d, "gproj"), dtype=torch.uint8,
                       device=dev) for _ in range(2)]
    ref = [run(*ins[i], wss[i]) for i in range(2)]
    ref = [[t.clone() for t in r] for r in ref]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(2)]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    outs = []
    for i, s in enumerate(streams):
        with torch.cuda.stream(s):
            outs.append(run(*ins[i], wss[i]))
    for s in streams:
        torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for r, o in zip(ref, outs):
        for a, b in zip(r, o):
            assert torch.equal(a, b)
