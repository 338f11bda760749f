"""torch.autograd integration: gradients through gpa.attention /
gpa.attention_varlen are bitwise those of the C-ABI backward called directly
(same kernels), in every mode, and a small model trains through it."""
import numpy as np
import pytest
import torch

import synthetic as S
from synthetic import suite

import _gpu as G

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


@pytest.fixture(scope="module")
def gpa():
    import paper_2609_34272_amd as gpa
    gpa.lib()
    return gpa


@pytest.mark.parametrize("mode", ["plain", "gproj_q", "gproj"])
def test_autograd_matches_direct_calls(gpa, mode):
    w = S.WORKLOADS[6].with_shape(N=300)
    x = S.make_inputs(w, 11)
    G.log(f"autograd dense {mode}: {w.name} N=300")
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    o_ref, lse = gpa.attn_fwd(q, k, v, True, w.scale)
    ref = gpa.attn_bwd(q, k, v, o_ref, lse, u, mode, True, w.scale)
    qa, ka, va = (t.clone().requires_grad_(True) for t in (q, k, v))
    o = gpa.attention(qa, ka, va, True, w.scale, mode)
    o.backward(u)
    torch.cuda.synchronize()
    assert np.array_equal(G.bits(o.detach()), G.bits(o_ref))
    for a, b in zip((qa.grad, ka.grad, va.grad), ref):
        assert np.array_equal(G.bits(a), G.bits(b))


@pytest.mark.parametrize("name", ["unequal lengths mixed", "more queries than keys"])
def test_autograd_varlen_matches_direct_calls(gpa, name):
    case = next(c for c in suite.CASES if c.name == name)
    x = suite.make_case(case)
    G.log(f"autograd varlen: case {case.index:03d} {case.name}")
    q, k, v, u = (G.to_dev(x[n]) for n in ("q", "k", "v", "do"))
    cu = torch.tensor(case.cu, dtype=torch.int32, device="cuda:0")
    kw = {}
    if case.cross:
        kw = dict(cu_seqlens_k=torch.tensor(case.cu_k, dtype=torch.int32, device="cuda:0"),
                  max_seqlen_k=case.max_seqlen_k)
    o_ref, lse = gpa.attn_fwd_varlen(q, k, v, cu, case.max_seqlen, True, case.scale, **kw)
    ref = gpa.attn_bwd_varlen(q, k, v, o_ref, lse, u, cu, case.max_seqlen, "gproj", True,
                              case.scale, **kw)
    qa, ka, va = (t.clone().requires_grad_(True) for t in (q, k, v))
    o = gpa.attention_varlen(qa, ka, va, cu, case.max_seqlen, True, case.scale, "gproj", **kw)
    o.backward(u)
    torch.cuda.synchronize()
    assert np.array_equal(G.bits(o.detach()), G.bits(o_ref))
    for a, b in zip((qa.grad, ka.grad, va.grad), ref):
        assert np.array_equal(G.bits(a), G.bits(b))


def test_small_model_trains(gpa):
    """A two-layer attention model's loss goes down over a few AdamW steps."""
    torch.manual_seed(0)
    dm, H, dh, N = 128, 2, 64, 256
    proj = torch.nn.Linear(dm, 3 * H * dh, bias=False).cuda()
    out = torch.nn.Linear(H * dh, dm, bias=False).cuda()
    opt = torch.optim.AdamW(list(proj.parameters()) + list(out.parameters()), lr=3e-3)
    x = torch.randn(N, dm, device="cuda")
    y = torch.randn(N, dm, device="cuda")
    losses = []
    for _ in range(20):
        with torch.autocast("cuda", dtype=torch.bfloat16):
            qkv = proj(x).view(N, 3, H, dh).permute(1, 2, 0, 3)
            q, k, v = (qkv[i].unsqueeze(0).contiguous() for i in range(3))
            o = gpa.attention(q, k, v, True, dh ** -0.5, "gproj")
            pred = out(o[0].transpose(0, 1).reshape(N, H * dh))
        loss = torch.nn.functional.mse_loss(pred.float(), y)
        loss.backward()
        opt.step()
        opt.zero_grad()
        losses.append(float(loss))
    assert all(np.isfinite(losses))
    assert losses[-1] < losses[0]
