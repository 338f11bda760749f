"""BF16 attention with the GProj gradient correction on AMD MI355X (gfx950).

Thin Python binding of libgpa.so (C ABI in include/gpa.h).  It only marshals
arguments: it checks tensor properties, allocates outputs and the workspace
with torch, and passes raw device pointers and the current HIP stream.  Every
step of the forward and backward runs in the library's HIP kernels; there is no
fallback path.

Python names mirror the C entry points:
  gpa_attn_fwd / attn_fwd                 -> O, LSE
  gpa_attn_bwd / attn_bwd                 -> dQ, dK, dV   (mode plain|gproj_q|gproj)
  gpa_attn_bwd_workspace_bytes / attn_bwd_workspace_bytes
  gpa_bwd_stats_offsets / bwd_stats_offsets
  gpa_fp32_attn / fp32_attn               -> O, LSE, dQ, dK, dV (FP32 baseline)
Grouped-query attention (k, v with fewer heads than q) goes through
gpa_attn_fwd_gqa / gpa_attn_bwd_gqa / gpa_attn_bwd_gqa_workspace_bytes; the
same Python functions pick them from the tensor shapes.  Packed
variable-length sequences ([H, total, d] tensors with int32 sequence offsets)
go through gpa_attn_fwd_varlen / gpa_attn_bwd_varlen
(attn_fwd_varlen / attn_bwd_varlen).
"""
from __future__ import annotations

import ctypes
import math
import os

import torch  # noqa: F401  (load torch's HIP runtime first; libgpa binds to it)

__all__ = [
    "MODES", "lib", "attn_fwd", "attn_fwd_fma", "attn_bwd", "attn_bwd_workspace_bytes", "bwd_stats_offsets",
    "attn_fwd_varlen", "attn_bwd_varlen", "attn_bwd_varlen_workspace_bytes",
    "fp32_attn", "fp32_attn_workspace_bytes", "profile_enable", "profile_read", "GpaError",
    "LIB_PATH", "attention", "attention_varlen", "attn_bwd_noalloc", "attn_bwd_atomic",
    "attn_bwd_atomic_workspace_bytes",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgpa.so")
MODES = {"plain": 0, "gproj_q": 1, "gproj": 2}
_STATUS = {0: "GPA_OK", 1: "GPA_EINVAL", 2: "GPA_ENOTSUP", 3: "GPA_EWORKSPACE", 4: "GPA_EHIP"}

_lib = None


class GpaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


def lib():
    """The loaded libgpa (ctypes).  Builds it in-tree first if it is missing;
    raises if it cannot be built or loaded."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from . import build as _build
        _build.build()
    L = ctypes.CDLL(LIB_PATH)
    P, I64, INT, F32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    L.gpa_version.restype = ctypes.c_char_p
    L.gpa_status_str.restype = ctypes.c_char_p
    L.gpa_status_str.argtypes = [INT]
    L.gpa_last_error.restype = ctypes.c_char_p
    L.gpa_attn_fwd.restype = INT
    L.gpa_attn_fwd.argtypes = [P, P, P, P, P, I64, I64, I64, I64, INT, F32, P]
    L.gpa_attn_bwd_workspace_bytes.restype = SZ
    L.gpa_attn_bwd_workspace_bytes.argtypes = [I64, I64, I64, I64, INT]
    L.gpa_attn_bwd.restype = INT
    L.gpa_attn_bwd.argtypes = [P, P, P, P, P, P, P, P, P, I64, I64, I64, I64, INT, F32, INT, P, SZ, P]
    L.gpa_attn_fwd_fma.restype = INT
    L.gpa_attn_fwd_fma.argtypes = [P, P, P, P, P, I64, I64, I64, I64, INT, F32, P]
    L.gpa_attn_fwd_gqa.restype = INT
    L.gpa_attn_fwd_gqa.argtypes = [P, P, P, P, P, I64, I64, I64, I64, I64, INT, F32, P]
    L.gpa_attn_bwd_gqa_workspace_bytes.restype = SZ
    L.gpa_attn_bwd_gqa_workspace_bytes.argtypes = [I64, I64, I64, I64, I64, INT]
    L.gpa_attn_bwd_gqa.restype = INT
    L.gpa_attn_bwd_gqa.argtypes = [P, P, P, P, P, P, P, P, P, I64, I64, I64, I64, I64, INT, F32,
                                   INT, P, SZ, P]
    L.gpa_attn_fwd_varlen.restype = INT
    L.gpa_attn_fwd_varlen.argtypes = [P] * 7 + [I64] * 8 + [INT, F32, P]
    L.gpa_attn_bwd_varlen_workspace_bytes.restype = SZ
    L.gpa_attn_bwd_varlen_workspace_bytes.argtypes = [I64] * 8 + [INT]
    L.gpa_attn_bwd_varlen.restype = INT
    L.gpa_attn_bwd_varlen.argtypes = [P] * 11 + [I64] * 8 + [INT, F32, INT, P, SZ, P]
    L.gpa_bwd_stats_offsets.restype = INT
    L.gpa_bwd_stats_offsets.argtypes = [I64, I64, I64, I64, INT] + [ctypes.POINTER(SZ)] * 4
    L.gpa_fp32_attn_workspace_bytes.restype = SZ
    L.gpa_fp32_attn_workspace_bytes.argtypes = [I64, I64, I64, I64]
    L.gpa_fp32_attn.restype = INT
    L.gpa_fp32_attn.argtypes = [P, P, P, P, P, P, P, P, P, I64, I64, I64, I64, INT, F32, P, SZ, P]
    L.gpa_profile_enable.restype = None
    L.gpa_profile_enable.argtypes = [INT]
    L.gpa_attn_bwd_noalloc_max_bytes.restype = SZ
    L.gpa_attn_bwd_noalloc_max_bytes.argtypes = []
    L.gpa_attn_bwd_noalloc.restype = INT
    L.gpa_attn_bwd_noalloc.argtypes = [P, P, P, P, P, P, P, P, P, I64, I64, I64, I64, INT, F32,
                                       INT, P]
    L.gpa_attn_bwd_atomic_workspace_bytes.restype = SZ
    L.gpa_attn_bwd_atomic_workspace_bytes.argtypes = [I64, I64, I64, I64, INT]
    L.gpa_attn_bwd_atomic.restype = INT
    L.gpa_attn_bwd_atomic.argtypes = [P, P, P, P, P, P, P, P, P, I64, I64, I64, I64, INT, F32, INT,
                                      P, SZ, P]
    L.gpa_profile_read.restype = INT
    L.gpa_profile_read.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(I64), INT]
    L.gpa_kernel_name.restype = ctypes.c_char_p
    L.gpa_kernel_name.argtypes = [INT]
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        raise GpaError(status, lib().gpa_last_error().decode())


def _stream(t: torch.Tensor) -> int:
    return torch.cuda.current_stream(t.device).cuda_stream


def _shape(q: torch.Tensor, name="q"):
    if q.dim() != 4:
        raise ValueError(f"{name} must be [B, H, N, d], got {tuple(q.shape)}")
    return tuple(int(x) for x in q.shape)


def _need(t: torch.Tensor, name: str, shape, dtype):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _scale(d: int, scale):
    return 1.0 / math.sqrt(d) if scale is None else float(scale)


def _kv_heads(q, k, name="k"):
    B, Hq, N, d = _shape(q)
    if k.dim() != 4 or k.shape[0] != B or k.shape[2] != N or k.shape[3] != d:
        raise ValueError(f"{name} must be [B, Hkv, N, d] matching q, got {tuple(k.shape)}")
    Hkv = int(k.shape[1])
    if Hkv < 1 or Hq % Hkv:
        raise ValueError(f"query heads {Hq} must be a multiple of key/value heads {Hkv}")
    return Hkv


def attn_fwd(q, k, v, causal: bool = True, scale=None):
    """FA3-SBS forward.  q: bf16 [B, Hq, N, d]; k, v: bf16 [B, Hkv, N, d] on the
    GPU (Hkv == Hq: multi-head; Hkv < Hq: grouped-query).
    Returns O (bf16, shaped like q) and LSE (float32 [B, Hq, N])."""
    B, H, N, d = _shape(q)
    Hkv = _kv_heads(q, k)
    _need(q, "q", (B, H, N, d), torch.bfloat16)
    for t, n in ((k, "k"), (v, "v")):
        _need(t, n, (B, Hkv, N, d), torch.bfloat16)
    o = torch.empty_like(q)
    lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    if Hkv == H:
        _check(lib().gpa_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                  lse.data_ptr(), B, H, N, d, int(bool(causal)), _scale(d, scale),
                                  _stream(q)))
    else:
        _check(lib().gpa_attn_fwd_gqa(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                      lse.data_ptr(), B, H, Hkv, N, d, int(bool(causal)),
                                      _scale(d, scale), _stream(q)))
    return o, lse


def attn_fwd_fma(q, k, v, causal: bool = True, scale=None):
    """Diagnostic forward with the historical FMA exponent rounding (not the
    GProj path).  Multi-head only.  Returns O, LSE like attn_fwd."""
    B, H, N, d = _shape(q)
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _need(t, n, (B, H, N, d), torch.bfloat16)
    o = torch.empty_like(q)
    lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    _check(lib().gpa_attn_fwd_fma(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                  lse.data_ptr(), B, H, N, d, int(bool(causal)), _scale(d, scale),
                                  _stream(q)))
    return o, lse


def attn_bwd_workspace_bytes(B: int, H: int, N: int, d: int, mode="gproj", Hkv=None) -> int:
    m = MODES[mode] if isinstance(mode, str) else int(mode)
    if Hkv is None or Hkv == H:
        return int(lib().gpa_attn_bwd_workspace_bytes(B, H, N, d, m))
    return int(lib().gpa_attn_bwd_gqa_workspace_bytes(B, H, Hkv, N, d, m))


def bwd_stats_offsets(B: int, H: int, N: int, d: int, mode="gproj"):
    """Byte offsets of D, rho, m, lambda inside the backward workspace."""
    offs = [ctypes.c_size_t() for _ in range(4)]
    m = MODES[mode] if isinstance(mode, str) else int(mode)
    _check(lib().gpa_bwd_stats_offsets(B, H, N, d, m, *[ctypes.byref(o) for o in offs]))
    return dict(zip(("D", "rho", "m", "lambda"), (o.value for o in offs)))


def attn_bwd(q, k, v, o, lse, do, mode: str = "gproj", causal: bool = True, scale=None,
             workspace=None, return_stats: bool = False):
    """Backward (plain | gproj_q | gproj).  q, o, do: bf16 [B, Hq, N, d];
    k, v: bf16 [B, Hkv, N, d].  Returns dQ, dK, dV (bf16, shaped like q, k, v);
    with return_stats=True also a dict of FP32 [B, Hq, N] tensors D, rho, m,
    lambda (views into the workspace)."""
    B, H, N, d = _shape(q)
    Hkv = _kv_heads(q, k)
    for t, n in ((q, "q"), (o, "o"), (do, "do")):
        _need(t, n, (B, H, N, d), torch.bfloat16)
    for t, n in ((k, "k"), (v, "v")):
        _need(t, n, (B, Hkv, N, d), torch.bfloat16)
    _need(lse, "lse", (B, H, N), torch.float32)
    mcode = MODES[mode] if isinstance(mode, str) else int(mode)
    nbytes = attn_bwd_workspace_bytes(B, H, N, d, mcode, Hkv)
    if workspace is None:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    dq = torch.empty_like(q)
    dk = torch.empty_like(k)
    dv = torch.empty_like(v)
    wsz = workspace.numel() * workspace.element_size()
    if Hkv == H:
        _check(lib().gpa_attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                  lse.data_ptr(), do.data_ptr(), dq.data_ptr(), dk.data_ptr(),
                                  dv.data_ptr(), B, H, N, d, int(bool(causal)), _scale(d, scale),
                                  mcode, workspace.data_ptr(), wsz, _stream(q)))
    else:
        _check(lib().gpa_attn_bwd_gqa(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                      lse.data_ptr(), do.data_ptr(), dq.data_ptr(), dk.data_ptr(),
                                      dv.data_ptr(), B, H, Hkv, N, d, int(bool(causal)),
                                      _scale(d, scale), mcode, workspace.data_ptr(), wsz,
                                      _stream(q)))
    if not return_stats:
        return dq, dk, dv
    offs = bwd_stats_offsets(B, H, N, d, mcode)
    n = B * H * N
    stats = {name: workspace[off:off + 4 * n].view(torch.float32).view(B, H, N)
             for name, off in offs.items()}
    return dq, dk, dv, stats


def attn_bwd_atomic(q, k, v, o, lse, do, mode: str = "plain", causal: bool = True, scale=None,
                    workspace=None):
    """The backward with Algorithm 1's schedule: one key-major pass with FP32
    atomic accumulation of the query-side sums, then (gproj) the key
    correction pass (gpa_attn_bwd_atomic; dense multi-head).  dV bitwise that
    of attn_bwd(mode=mode); plain and gproj_q dK too; dQ the same sums in
    another order."""
    B, H, N, d = _shape(q)
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (o, "o"), (do, "do")):
        _need(t, n, (B, H, N, d), torch.bfloat16)
    _need(lse, "lse", (B, H, N), torch.float32)
    mi = MODES[mode] if isinstance(mode, str) else int(mode)
    nbytes = int(lib().gpa_attn_bwd_atomic_workspace_bytes(B, H, N, d, mi))
    if workspace is None:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    _check(lib().gpa_attn_bwd_atomic(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                     lse.data_ptr(), do.data_ptr(), dq.data_ptr(), dk.data_ptr(),
                                     dv.data_ptr(), B, H, N, d, int(bool(causal)), _scale(d, scale),
                                     mi, workspace.data_ptr(), workspace.numel(), _stream(q)))
    return dq, dk, dv


def attn_bwd_atomic_workspace_bytes(B: int, H: int, N: int, d: int, mode: str = "plain") -> int:
    mi = MODES[mode] if isinstance(mode, str) else int(mode)
    return int(lib().gpa_attn_bwd_atomic_workspace_bytes(B, H, N, d, mi))


def attn_bwd_noalloc(q, k, v, o, lse, do, mode: str = "gproj", causal: bool = True, scale=None,
                     out=None):
    """attn_bwd without a workspace: the library uses its own per-GPU scratch
    array (gpa_attn_bwd_noalloc; multi-head only, shapes whose workspace fits
    gpa_attn_bwd_noalloc_max_bytes()).  out: optional preallocated (dq, dk,
    dv); otherwise they are allocated here.  Calls that overlap on one GPU
    share the scratch and race."""
    B, H, N, d = _shape(q)
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (o, "o"), (do, "do")):
        _need(t, n, (B, H, N, d), torch.bfloat16)
    _need(lse, "lse", (B, H, N), torch.float32)
    mcode = MODES[mode] if isinstance(mode, str) else int(mode)
    if out is None:
        out = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v))
    dq, dk, dv = out
    for t, n in ((dq, "dq"), (dk, "dk"), (dv, "dv")):
        _need(t, n, (B, H, N, d), torch.bfloat16)
    _check(lib().gpa_attn_bwd_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                      lse.data_ptr(), do.data_ptr(), dq.data_ptr(), dk.data_ptr(),
                                      dv.data_ptr(), B, H, N, d, int(bool(causal)),
                                      _scale(d, scale), mcode, _stream(q)))
    return dq, dk, dv


def _offsets(cu, name):
    if (not cu.is_cuda or cu.dtype != torch.int32 or cu.dim() != 1 or cu.numel() < 2
            or not cu.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous 1-D int32 GPU tensor of nseq + 1 offsets")


class _Packed:
    """Checked packed layout: q [Hq, total_q, d], k [Hkv, total_k, d], int32
    offsets on the GPU for each side (the key side defaults to the query
    side's offsets and longest run)."""

    def __init__(self, q, k, cu_seqlens, max_seqlen, cu_seqlens_k, max_seqlen_k):
        if q.dim() != 3 or k.dim() != 3 or k.shape[2] != q.shape[2]:
            raise ValueError(f"packed q [Hq, total_q, d] and k [Hkv, total_k, d] expected, got "
                             f"{tuple(q.shape)}, {tuple(k.shape)}")
        self.Hq, self.total_q, self.d = (int(x) for x in q.shape)
        self.Hkv, self.total_k = int(k.shape[0]), int(k.shape[1])
        if self.Hkv < 1 or self.Hq % self.Hkv:
            raise ValueError(f"query heads {self.Hq} must be a multiple of key/value heads {self.Hkv}")
        _offsets(cu_seqlens, "cu_seqlens")
        self.cu_q = cu_seqlens
        self.max_q = int(max_seqlen)
        if cu_seqlens_k is None:
            if self.total_k != self.total_q:
                raise ValueError("k has its own token count: pass cu_seqlens_k and max_seqlen_k")
            self.cu_k, self.max_k = cu_seqlens, self.max_q
        else:
            _offsets(cu_seqlens_k, "cu_seqlens_k")
            if cu_seqlens_k.numel() != cu_seqlens.numel():
                raise ValueError("cu_seqlens and cu_seqlens_k must describe the same number of sequences")
            if max_seqlen_k is None:
                raise ValueError("cu_seqlens_k needs max_seqlen_k")
            self.cu_k, self.max_k = cu_seqlens_k, int(max_seqlen_k)
        self.nseq = cu_seqlens.numel() - 1

    def offsets(self):
        """The C arguments from the offsets through max_seqlen_k."""
        return (self.cu_q.data_ptr(), self.cu_k.data_ptr(), self.nseq, self.total_q, self.total_k,
                self.Hq, self.Hkv, self.max_q, self.max_k, self.d)


def attn_fwd_varlen(q, k, v, cu_seqlens, max_seqlen: int, causal: bool = True, scale=None,
                    cu_seqlens_k=None, max_seqlen_k=None):
    """FA3-SBS forward over packed sequences.  q: bf16 [Hq, total_q, d]; k, v:
    bf16 [Hkv, total_k, d]; cu_seqlens: int32 [nseq + 1] query offsets on the
    GPU (sequence s = queries cu[s] .. cu[s+1]-1); max_seqlen: the longest
    query run.  cu_seqlens_k / max_seqlen_k give the key side (default: the
    same as the queries); with causal the diagonal is aligned at the last
    query and key, and a query that sees no key gets O = 0, LSE = +inf.
    Returns O (bf16 [Hq, total_q, d]) and LSE (float32 [Hq, total_q])."""
    pk = _Packed(q, k, cu_seqlens, max_seqlen, cu_seqlens_k, max_seqlen_k)
    _need(q, "q", (pk.Hq, pk.total_q, pk.d), torch.bfloat16)
    for t, n in ((k, "k"), (v, "v")):
        _need(t, n, (pk.Hkv, pk.total_k, pk.d), torch.bfloat16)
    o = torch.empty_like(q)
    lse = torch.empty((pk.Hq, pk.total_q), dtype=torch.float32, device=q.device)
    _check(lib().gpa_attn_fwd_varlen(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                     lse.data_ptr(), *pk.offsets(), int(bool(causal)),
                                     _scale(pk.d, scale), _stream(q)))
    return o, lse


def attn_bwd_varlen_workspace_bytes(nseq: int, total: int, Hq: int, Hkv: int, max_seqlen: int,
                                    d: int, mode="gproj", total_k=None, max_seqlen_k=None) -> int:
    m = MODES[mode] if isinstance(mode, str) else int(mode)
    tk = total if total_k is None else int(total_k)
    mk = max_seqlen if max_seqlen_k is None else int(max_seqlen_k)
    return int(lib().gpa_attn_bwd_varlen_workspace_bytes(nseq, total, tk, Hq, Hkv, max_seqlen, mk,
                                                         d, m))


def attn_bwd_varlen(q, k, v, o, lse, do, cu_seqlens, max_seqlen: int, mode: str = "gproj",
                    causal: bool = True, scale=None, workspace=None, return_stats: bool = False,
                    cu_seqlens_k=None, max_seqlen_k=None):
    """Backward over packed sequences (layouts as attn_fwd_varlen).  Returns
    dQ, dK, dV; with return_stats=True also FP32 [Hq, total_q] views D, rho,
    m, lambda into the workspace."""
    pk = _Packed(q, k, cu_seqlens, max_seqlen, cu_seqlens_k, max_seqlen_k)
    for t, n in ((q, "q"), (o, "o"), (do, "do")):
        _need(t, n, (pk.Hq, pk.total_q, pk.d), torch.bfloat16)
    for t, n in ((k, "k"), (v, "v")):
        _need(t, n, (pk.Hkv, pk.total_k, pk.d), torch.bfloat16)
    _need(lse, "lse", (pk.Hq, pk.total_q), torch.float32)
    mcode = MODES[mode] if isinstance(mode, str) else int(mode)
    nbytes = attn_bwd_varlen_workspace_bytes(pk.nseq, pk.total_q, pk.Hq, pk.Hkv, pk.max_q, pk.d,
                                             mcode, pk.total_k, pk.max_k)
    if workspace is None:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=q.device)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    wsz = workspace.numel() * workspace.element_size()
    _check(lib().gpa_attn_bwd_varlen(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                     lse.data_ptr(), do.data_ptr(), dq.data_ptr(), dk.data_ptr(),
                                     dv.data_ptr(), *pk.offsets(), int(bool(causal)),
                                     _scale(pk.d, scale), mcode, workspace.data_ptr(), wsz,
                                     _stream(q)))
    if not return_stats:
        return dq, dk, dv
    offs = bwd_stats_offsets(1, pk.Hq, pk.total_q, pk.d, mcode)
    n = pk.Hq * pk.total_q
    stats = {name: workspace[off:off + 4 * n].view(torch.float32).view(pk.Hq, pk.total_q)
             for name, off in offs.items()}
    return dq, dk, dv, stats


def fp32_attn_workspace_bytes(B: int, H: int, N: int, d: int) -> int:
    return int(lib().gpa_fp32_attn_workspace_bytes(B, H, N, d))


def fp32_attn(q, k, v, do, causal: bool = True, scale=None):
    """FP32-arithmetic attention forward + backward with BF16 I/O (baseline).
    Returns O, LSE, dQ, dK, dV."""
    B, H, N, d = _shape(q)
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (do, "do")):
        _need(t, n, (B, H, N, d), torch.bfloat16)
    nbytes = fp32_attn_workspace_bytes(B, H, N, d)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    o = torch.empty_like(q)
    lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)
    _check(lib().gpa_fp32_attn(q.data_ptr(), k.data_ptr(), v.data_ptr(), do.data_ptr(), o.data_ptr(),
                               lse.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                               B, H, N, d, int(bool(causal)), _scale(d, scale), ws.data_ptr(),
                               nbytes, _stream(q)))
    return o, lse, dq, dk, dv


def profile_enable(on: bool = True):
    lib().gpa_profile_enable(int(bool(on)))


def profile_read():
    """{kernel name: (total ms, launches)} since the last read; synchronises."""
    n = 16
    ms = (ctypes.c_double * n)()
    cnt = (ctypes.c_int64 * n)()
    k = lib().gpa_profile_read(ms, cnt, n)
    return {lib().gpa_kernel_name(i).decode(): (ms[i], cnt[i]) for i in range(k)}


from .autograd import attention, attention_varlen  # noqa: E402

# Raw C entry points under their C names (argument marshalling is the caller's).
def __getattr__(name):
    if name.startswith("gpa_"):
        return getattr(lib(), name)
    raise AttributeError(name)
