"""torch.autograd integration of the attention forward and backward.

attention(q, k, v, causal, scale, mode) returns O from the FA3-SBS forward and
routes its gradient through the library's backward in the chosen mode
(plain | gproj_q | gproj); attention_varlen does the same for packed
variable-length sequences.  The forward saves Q, K, V, O and the FP32 LSE for
the backward (the state Algorithm 1 takes as input); nothing else is kept.
Both directions run in libgpa's HIP kernels.
"""
from __future__ import annotations

import torch

from . import attn_bwd, attn_bwd_varlen, attn_fwd, attn_fwd_varlen

__all__ = ["attention", "attention_varlen"]


class _Attention(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, causal, scale, mode):
        o, lse = attn_fwd(q, k, v, causal, scale)
        ctx.save_for_backward(q, k, v, o, lse)
        ctx.causal, ctx.scale, ctx.mode = causal, scale, mode
        return o

    @staticmethod
    def backward(ctx, do):
        q, k, v, o, lse = ctx.saved_tensors
        dq, dk, dv = attn_bwd(q, k, v, o, lse, do.contiguous(), ctx.mode, ctx.causal, ctx.scale)
        return dq, dk, dv, None, None, None


class _AttentionVarlen(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, cu_seqlens, max_seqlen, causal, scale, mode, cu_seqlens_k,
                max_seqlen_k):
        o, lse = attn_fwd_varlen(q, k, v, cu_seqlens, max_seqlen, causal, scale, cu_seqlens_k,
                                 max_seqlen_k)
        cu_k = cu_seqlens if cu_seqlens_k is None else cu_seqlens_k
        ctx.save_for_backward(q, k, v, o, lse, cu_seqlens, cu_k)
        ctx.max_seqlen, ctx.causal, ctx.scale, ctx.mode = max_seqlen, causal, scale, mode
        ctx.max_seqlen_k = max_seqlen if cu_seqlens_k is None else max_seqlen_k
        return o

    @staticmethod
    def backward(ctx, do):
        q, k, v, o, lse, cu, cu_k = ctx.saved_tensors
        dq, dk, dv = attn_bwd_varlen(q, k, v, o, lse, do.contiguous(), cu, ctx.max_seqlen,
                                     ctx.mode, ctx.causal, ctx.scale, cu_seqlens_k=cu_k,
                                     max_seqlen_k=ctx.max_seqlen_k)
        return dq, dk, dv, None, None, None, None, None, None, None


def attention(q, k, v, causal: bool = True, scale=None, mode: str = "gproj"):
    """Differentiable attention: q [B, Hq, N, d], k, v [B, Hkv, N, d] (bf16,
    contiguous, on the GPU) -> O [B, Hq, N, d]."""
    return _Attention.apply(q, k, v, bool(causal), scale, mode)


def attention_varlen(q, k, v, cu_seqlens, max_seqlen: int, causal: bool = True, scale=None,
                     mode: str = "gproj", cu_seqlens_k=None, max_seqlen_k=None):
    """Differentiable attention over packed sequences: q [Hq, total_q, d], k, v
    [Hkv, total_k, d], int32 query offsets cu_seqlens [nseq + 1] (key offsets
    cu_seqlens_k, default the same) -> O [Hq, total_q, d]."""
    mk = None if max_seqlen_k is None else int(max_seqlen_k)
    return _AttentionVarlen.apply(q, k, v, cu_seqlens, int(max_seqlen), bool(causal), scale, mode,
                                  cu_seqlens_k, mk)
