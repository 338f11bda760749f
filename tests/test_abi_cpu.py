"""The C-ABI library loads, exports every declared symbol, and rejects bad
arguments before launching anything (no GPU needed: every call here fails
validation, so no HIP call is made)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_symbols():
    with open(os.path.join(ROOT, "include", "gpa.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(gpa_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2609_34272_amd as gpa
    return gpa.lib()


def test_header_declares_the_boundary():
    syms = _declared_symbols()
    for s in ("gpa_attn_fwd", "gpa_attn_bwd", "gpa_attn_bwd_workspace_bytes",
              "gpa_bwd_stats_offsets", "gpa_fp32_attn"):
        assert s in syms


def test_library_exports_every_declared_symbol(lib):
    for s in _declared_symbols():
        assert hasattr(lib, s), s


def test_version_and_status_strings(lib):
    assert b"gfx950" in lib.gpa_version()
    for code in range(5):
        assert lib.gpa_status_str(code).startswith(b"GPA_")


def test_workspace_sizes(lib):
    import paper_2609_34272_amd as gpa
    n = gpa.attn_bwd_workspace_bytes(1, 16, 4096, 64, "gproj")
    assert n >= 4 * 16 * 4096 * 4
    assert gpa.attn_bwd_workspace_bytes(1, 1, 1, 64, "plain") > 0
    assert gpa.attn_bwd_workspace_bytes(1, 1, 1, 96, "plain") == 0
    assert gpa.attn_bwd_workspace_bytes(0, 1, 1, 64, "plain") == 0
    assert lib.gpa_attn_bwd_workspace_bytes(1, 1, 8, 64, 7) == 0
    offs = gpa.bwd_stats_offsets(2, 3, 100, 128, "gproj")
    vals = sorted(offs.values())
    assert vals[0] == 0 and all(v % 256 == 0 for v in vals)
    assert vals[-1] + 2 * 3 * 100 * 4 <= gpa.attn_bwd_workspace_bytes(2, 3, 100, 128, "gproj")
    assert gpa.fp32_attn_workspace_bytes(1, 2, 10, 64) >= 2 * 10 * 64 * 4 + 2 * 10 * 4


FAKE = 0x7F0000000000  # never dereferenced: validation fails first


def _fwd(lib, Q=FAKE, K=FAKE + 0x10000000, V=FAKE + 0x20000000, O=FAKE + 0x30000000,
         L=FAKE + 0x40000000, B=1, H=1, N=128, d=64, causal=1, scale=0.125):
    return lib.gpa_attn_fwd(Q, K, V, O, L, B, H, N, d, causal, scale, None)


def test_fwd_validation(lib):
    assert _fwd(lib, Q=None) == 1
    assert b"Q is NULL" in lib.gpa_last_error()
    assert _fwd(lib, K=FAKE + 0x10000008) == 1
    assert b"aligned" in lib.gpa_last_error()
    assert _fwd(lib, d=96) == 2
    assert _fwd(lib, N=0) == 1
    assert _fwd(lib, scale=float("nan")) == 1
    assert _fwd(lib, scale=-1.0) == 1
    assert _fwd(lib, B=1 << 20, H=1 << 10, N=1 << 10) == 1     # too many elements
    assert _fwd(lib, O=FAKE + 0x100) == 1                       # O overlaps Q
    assert b"overlaps" in lib.gpa_last_error()


def _bwd(lib, mode=2, ws=FAKE + 0x90000000, ws_bytes=None, dQ=FAKE + 0x60000000, N=128, d=64):
    if ws_bytes is None:
        ws_bytes = lib.gpa_attn_bwd_workspace_bytes(1, 1, N, 64, mode) or 1 << 20
    base = [FAKE + i * 0x10000000 for i in range(9)]
    base[6] = dQ
    return lib.gpa_attn_bwd(*base, 1, 1, N, d, 1, 0.125, mode, ws, ws_bytes, None)


def test_bwd_validation(lib):
    assert _bwd(lib, mode=3) == 1
    assert _bwd(lib, ws=None) == 3
    assert _bwd(lib, ws_bytes=16) == 3
    assert _bwd(lib, ws=FAKE + 0x90000010) == 3                 # not 256-byte aligned
    assert _bwd(lib, dQ=FAKE + 0x10000000) == 1                 # dQ aliases K
    assert _bwd(lib, d=80) == 2


def test_atomic_schedule_workspace_and_validation(lib):
    import paper_2609_34272_amd as gpa
    B, H, N, d = 1, 16, 4096, 64
    big = B * H * N * d * 4
    plain = gpa.attn_bwd_atomic_workspace_bytes(B, H, N, d, "plain")
    gq = gpa.attn_bwd_atomic_workspace_bytes(B, H, N, d, "gproj_q")
    gp = gpa.attn_bwd_atomic_workspace_bytes(B, H, N, d, "gproj")
    # A; then B, rho, m; then dK^acc (FP32) and -z (BF16)
    assert plain >= big
    assert gq - plain >= big + 2 * B * H * N * 4
    assert gp - gq >= big + big // 2
    assert all(v % 256 == 0 for v in (plain, gq, gp))
    assert lib.gpa_attn_bwd_atomic_workspace_bytes(1, 1, 8, 64, 3) == 0
    assert lib.gpa_attn_bwd_atomic_workspace_bytes(1, 1, 8, 80, 0) == 0
    args = [FAKE + i * 0x10000000 for i in range(9)]
    ws = FAKE + 0x90000000
    need = lib.gpa_attn_bwd_atomic_workspace_bytes(1, 1, 128, 64, 2)
    assert lib.gpa_attn_bwd_atomic(*args, 1, 1, 128, 64, 1, 0.125, 3, ws, need, None) == 1
    assert lib.gpa_attn_bwd_atomic(*args, 1, 1, 128, 64, 1, 0.125, 2, ws, need - 256, None) == 3
    assert lib.gpa_attn_bwd_atomic(*args, 1, 1, 128, 64, 1, 0.125, 2, None, need, None) == 3


def test_fp32_validation(lib):
    args = [FAKE + i * 0x10000000 for i in range(9)]
    assert lib.gpa_fp32_attn(*args, 1, 1, 64, 64, 1, 0.125, None, 0, None) == 3
    args[4] = None
    assert lib.gpa_fp32_attn(*args, 1, 1, 64, 64, 1, 0.125, FAKE + 0xA0000000, 1 << 30, None) == 1


def test_python_binding_rejects_cpu_tensors():
    import torch
    import paper_2609_34272_amd as gpa
    q = torch.zeros(1, 1, 8, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        gpa.attn_fwd(q, q, q)


def test_gqa_validation(lib):
    P = FAKE
    # Hq not a multiple of Hkv
    assert lib.gpa_attn_fwd_gqa(P, P + 0x10000000, P + 0x20000000, P + 0x30000000, P + 0x40000000,
                                1, 6, 4, 128, 64, 1, 0.125, None) == 1
    assert b"multiple" in lib.gpa_last_error()
    assert lib.gpa_attn_bwd_gqa_workspace_bytes(1, 6, 4, 128, 64, 2) == 0
    # grouped workspace adds the per-head FP32 contributions
    mha = lib.gpa_attn_bwd_gqa_workspace_bytes(1, 16, 16, 4096, 64, 2)
    gqa = lib.gpa_attn_bwd_gqa_workspace_bytes(1, 16, 4, 4096, 64, 2)
    assert mha == lib.gpa_attn_bwd_workspace_bytes(1, 16, 4096, 64, 2)
    assert gqa == mha + 2 * 16 * 4096 * 64 * 4


def _fwd_varlen(lib, cu=FAKE + 0x50000000, cu_k=None, nseq=3, total=300, total_k=300, Hq=4,
                Hkv=2, ms=128, ms_k=128, d=64, O=FAKE + 0x30000000):
    P = FAKE
    return lib.gpa_attn_fwd_varlen(P, P + 0x10000000, P + 0x20000000, O, P + 0x40000000, cu,
                                   cu_k, nseq, total, total_k, Hq, Hkv, ms, ms_k, d, 1, 0.125, None)


def test_varlen_validation(lib):
    assert _fwd_varlen(lib, cu=None) == 1
    assert b"cu_seqlens_q is NULL" in lib.gpa_last_error()
    assert _fwd_varlen(lib, cu=FAKE + 0x50000002) == 1                 # not 4-byte aligned
    assert _fwd_varlen(lib, cu_k=FAKE + 0x60000002) == 1
    assert _fwd_varlen(lib, ms=301) == 1                               # longer than total
    assert _fwd_varlen(lib, ms=0) == 1
    assert _fwd_varlen(lib, nseq=0) == 1
    assert _fwd_varlen(lib, Hq=6, Hkv=4) == 1
    assert _fwd_varlen(lib, d=96) == 2
    assert _fwd_varlen(lib, O=FAKE + 0x50000000) == 1                  # O overlaps cu_seqlens_q
    assert b"overlaps" in lib.gpa_last_error()
    # the key side: its own total and longest run, checked on their own
    assert _fwd_varlen(lib, cu_k=FAKE + 0x60000000, total_k=200, ms_k=201) == 1
    assert _fwd_varlen(lib, cu_k=FAKE + 0x60000000, total_k=0, ms_k=0) == 1
    assert _fwd_varlen(lib, cu_k=FAKE + 0x60000000, O=FAKE + 0x60000000) == 1
    assert b"cu_seqlens_k" in lib.gpa_last_error()
    # shared offsets (cu_seqlens_k NULL) need matching totals and runs
    assert _fwd_varlen(lib, total_k=200) == 1
    assert _fwd_varlen(lib, ms_k=64) == 1
    assert b"shared offsets" in lib.gpa_last_error()
    # workspace: row statistics over [Hq, total_q], tile blocks per (sequence,
    # head) and 64 query rows, z over the queries, grouped partials over the keys
    ws = lib.gpa_attn_bwd_varlen_workspace_bytes(3, 300, 300, 4, 2, 128, 128, 64, 2)
    assert ws >= 4 * 4 * 300 * 4 + 3 * 4 * 2 * 512 + 4 * 300 * 64 * 2 + 2 * 4 * 300 * 64 * 4
    ws_k = lib.gpa_attn_bwd_varlen_workspace_bytes(3, 300, 500, 4, 2, 128, 256, 64, 2)
    assert ws_k - ws == 2 * 4 * 200 * 64 * 4
    assert lib.gpa_attn_bwd_varlen_workspace_bytes(3, 300, 300, 4, 2, 301, 128, 64, 2) == 0
    assert lib.gpa_attn_bwd_varlen_workspace_bytes(3, 300, 300, 4, 2, 128, 301, 64, 2) == 0
    assert lib.gpa_attn_bwd_varlen_workspace_bytes(3, 300, 300, 4, 2, 128, 128, 64, 3) == 0
    # the backward rejects a short workspace before launching anything
    P = FAKE
    args = [P + i * 0x10000000 for i in range(9)]
    assert lib.gpa_attn_bwd_varlen(*args, P + 0x90000000, None, 3, 300, 300, 4, 2, 128, 128, 64,
                                   1, 0.125, 2, P + 0xA0000000, 16, None) == 3
