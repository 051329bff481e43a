"""The C-ABI library loads, exports every entry point include/moe.h declares, and rejects invalid
arguments on the host before launching anything (no GPU needed: no compute call reaches HIP)."""
import ctypes
import os
import re

import pytest

from paper_2606_26453_amd import moe
from paper_2606_26453_amd.build import LIB_PATH

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "moe.h")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB_PATH), reason="library not built")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z_0-9]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = _declared()
    assert len(names) >= 11
    L = ctypes.CDLL(LIB_PATH)
    for n in names:
        assert hasattr(L, n), f"{n} declared in moe.h but not exported"
    assert set(names) == set(moe._SIG), "binding and header disagree"


def test_status_strings():
    L = moe.lib()
    for code in range(5):
        assert L.moe_status_string(code)
    assert L.moe_status_string(99) == b"unknown status"


FAKE = 1 << 20        # a 16-byte-aligned non-NULL address that is never dereferenced
BAD = FAKE + 2        # misaligned


def test_route_permute_rejects():
    L = moe.lib()
    args = lambda T=10, d=64, E=4, k=2, norm=1, x=FAKE, ws=FAKE, wsb=1 << 20: (
        FAKE, x, T, d, E, k, norm, FAKE, FAKE, FAKE, FAKE, FAKE, x, ws, wsb, None)
    assert L.moe_route_permute(*args(k=5)) == 1            # k > E
    assert L.moe_route_permute(*args(k=0)) == 1
    assert L.moe_route_permute(*args(E=300, k=2)) == 2     # E > 256
    assert L.moe_route_permute(*args(d=100)) == 2          # d % 64
    assert L.moe_route_permute(*args(T=-1)) == 1
    assert L.moe_route_permute(*args(norm=2)) == 1
    assert L.moe_route_permute(*args(x=BAD)) == 1          # misaligned
    assert L.moe_route_permute(*args(wsb=0)) == 3          # workspace too small
    assert b"workspace" in L.moe_last_error()
    assert L.moe_route_permute(*args(T=1 << 30, k=4)) == 2  # R >= 2^31
    assert L.moe_route_permute_workspace_bytes(0, 4, 2) == 0
    assert L.moe_route_permute_workspace_bytes(1000, 64, 6) > 0


def test_gemm_rejects():
    L = moe.lib()
    fwd = lambda G=4, R=100, K=128, N=128, A=FAKE, B2=None, C2=None, act=None: L.moe_grouped_gemm_fwd(
        A, FAKE, B2, FAKE, G, R, K, N, FAKE, C2, act, None)
    assert fwd(G=0) == 2 and fwd(G=257) == 2
    assert fwd(K=100) == 2 and fwd(N=96) == 2
    assert fwd(R=-1) == 1
    assert fwd(A=BAD) == 1
    assert fwd(B2=FAKE) == 1                 # B2 without C2
    assert fwd(act=FAKE) == 1                # act without B2
    assert fwd(A=None) == 1
    assert fwd(R=0) == 0                     # empty: successful no-op
    dx = lambda G=4, R=100, K=128, N=128, dC2=None, B2=None: L.moe_grouped_gemm_dx(
        FAKE, FAKE, dC2, B2, FAKE, G, R, K, N, FAKE, None)
    assert dx(K=65) == 2 and dx(dC2=FAKE) == 1 and dx(R=0) == 0
    dw = lambda G=4, R=100, K=128, N=128, dC2=None, dB2=None, dB=FAKE: L.moe_grouped_gemm_dw(
        FAKE, FAKE, dC2, FAKE, G, R, K, N, dB, dB2, None)
    assert dw(N=32) == 2 and dw(dC2=FAKE) == 1 and dw(dB=None) == 1 and dw(dB=BAD) == 1
    dw16 = lambda G=4, R=100, K=128, N=128, dC2=None, dB2=None, dB=FAKE: L.moe_grouped_gemm_dw_bf16(
        FAKE, FAKE, dC2, FAKE, G, R, K, N, dB, dB2, None)
    assert dw16(G=257) == 2 and dw16(K=2880 + 32) == 2 and dw16(dC2=FAKE) == 1 and dw16(dB=None) == 1
    assert dw16(dB=BAD) == 1 and dw16(R=-1) == 1
    dwp = lambda G=4, R=100, K=128, N=128, cnt=FAKE, dB=FAKE: L.moe_grouped_gemm_dw_persistent(
        FAKE, FAKE, None, FAKE, G, R, K, N, dB, None, cnt, None)
    assert dwp(cnt=None) == 1 and dwp(cnt=BAD) == 1 and dwp(N=32) == 2 and dwp(dB=None) == 1
    dwp16 = lambda G=4, R=100, K=128, N=128, cnt=FAKE: L.moe_grouped_gemm_dw_bf16_persistent(
        FAKE, FAKE, None, FAKE, G, R, K, N, FAKE, None, cnt, None)
    assert dwp16(cnt=None) == 1 and dwp16(cnt=BAD) == 1 and dwp16(G=0) == 2
    dxs = lambda G=4, R=100, K=128, N=128, hg=FAKE: L.moe_grouped_gemm_dx_swiglu_bwd(
        FAKE, FAKE, FAKE, G, R, K, N, hg, FAKE, FAKE, FAKE, None)
    assert dxs(N=100) == 2 and dxs(hg=None) == 1 and dxs(hg=BAD) == 1 and dxs(R=0) == 0


def test_split_rejects():
    """The split-tail dX entries need a workspace of the queried size: missing or short -> 3."""
    L = moe.lib()
    need = L.moe_grouped_gemm_split_workspace_bytes()
    assert need >= 256 * 256 * 256 * 4
    dx = lambda ws=FAKE, n=need, K=128: L.moe_grouped_gemm_dx_split(
        FAKE, FAKE, None, None, FAKE, 4, 100, K, 128, FAKE, ws, n, None)
    assert dx(ws=None) == 3 and dx(n=need - 1) == 3 and dx(ws=BAD) == 3 and dx(K=65) == 2
    dxs = lambda ws=FAKE, n=need: L.moe_grouped_gemm_dx_swiglu_bwd_split(
        FAKE, FAKE, FAKE, 4, 100, 128, 128, FAKE, FAKE, FAKE, FAKE, ws, n, None)
    assert dxs(ws=None) == 3 and dxs(n=16) == 3
    fwd = lambda ws=FAKE, n=need, N=128: L.moe_grouped_gemm_fwd_split(
        FAKE, FAKE, None, FAKE, 4, 100, 128, N, FAKE, None, None, ws, n, None)
    assert fwd(ws=None) == 3 and fwd(n=need // 2) == 3 and fwd(N=96) == 2
    # the split dW: counters first, then a given workspace must be whole and aligned (NULL: no split)
    dws = lambda cnt=FAKE, ws=FAKE, n=need, K=128: L.moe_grouped_gemm_dw_split(
        FAKE, FAKE, None, FAKE, 1, 100, K, 128, FAKE, None, cnt, ws, n, None)
    assert dws(cnt=None) == 1 and dws(cnt=BAD) == 1 and dws(n=need - 1) == 3 and dws(ws=BAD) == 3
    assert dws(K=65) == 2


def test_fp8_rejects():
    L = moe.lib()
    qz = lambda M=10, K=64, x=FAKE, q=FAKE: L.moe_quantize_fp8_rows(x, M, K, q, FAKE, None)
    assert qz(K=24) == 2 and qz(x=None) == 1 and qz(x=BAD) == 1 and qz(q=FAKE + 4) == 1 and qz(M=0) == 0
    f8 = lambda G=4, R=100, K=128, N=128, A=FAKE, sa=FAKE, ws=None, n=0: L.moe_grouped_gemm_fwd_fp8(
        A, sa, FAKE, FAKE, FAKE, G, R, K, N, FAKE, ws, n, None)
    assert f8(K=96) == 2 and f8(N=100) == 2 and f8(G=0) == 2 and f8(A=None) == 1 and f8(sa=None) == 1
    assert f8(A=BAD) == 1 and f8(R=0) == 0 and f8(ws=FAKE, n=16) == 3
    gu = lambda F=128, K=128, act=FAKE, hg=FAKE: L.moe_grouped_gemm_fwd_fp8_gate_up(
        FAKE, FAKE, FAKE, FAKE, FAKE, 4, 100, K, F, hg, FAKE, act, None, 0, None)
    assert gu(F=64) == 2 and gu(K=96) == 2 and gu(hg=None) == 1 and gu(act=BAD) == 1
    qw = lambda G=2, K=64, N=128, w=FAKE, w2=None, q=FAKE: L.moe_quantize_fp8_weight(w, w2, G, K, N, q, FAKE, None)
    assert qw(K=24) == 2 and qw(N=96) == 2 and qw(N=192, w2=FAKE) == 2 and qw(G=-1) == 1
    assert qw(w=None) == 1 and qw(w=BAD) == 1 and qw(q=FAKE + 8) == 1 and qw(w2=BAD) == 1 and qw(G=0) == 0


def test_mx_rejects():
    L = moe.lib()
    assert L.moe_mx_scale_bytes(10, 64) == 40 and L.moe_mx_scale_bytes(10, 2880) == 23 * 40
    assert L.moe_mx_scale_bytes(0, 64) == 0 and L.moe_mx_scale_bytes(10, 0) == 0
    assert L.moe_mx_tokens_cols_bound(100, 4) == 640 and L.moe_mx_tokens_cols_bound(0, 1) == 128
    qr = lambda M=10, K=64, x=FAKE, x2=None, q=FAKE: L.moe_quantize_mx_rows(x, x2, M, K, q, FAKE, None)
    assert qr(K=48) == 2 and qr(x=None) == 1 and qr(x=BAD) == 1 and qr(x2=BAD) == 1 and qr(q=FAKE + 4) == 1
    assert qr(M=-1) == 1 and qr(M=0) == 0
    qw = lambda G=2, K=64, N=128, w=FAKE, w2=None, qt=FAKE, st=FAKE, q_r=FAKE, sr=FAKE: L.moe_quantize_mx_weight(
        w, w2, G, K, N, qt, st, q_r, sr, None)
    assert qw(K=48) == 2 and qw(N=96) == 2 and qw(N=192, w2=FAKE) == 2
    assert qw(st=None) == 1 and qw(sr=None) == 1 and qw(qt=None, st=None, q_r=None, sr=None) == 1
    assert qw(w=None) == 1 and qw(w=BAD) == 1 and qw(qt=FAKE + 8) == 1 and qw(q_r=FAKE + 4) == 1 and qw(G=0) == 0
    mx = lambda G=4, R=100, K=128, N=128, A=FAKE, sa=FAKE, sw=FAKE, ws=None, n=0: L.moe_grouped_gemm_fwd_mx(
        A, sa, FAKE, sw, FAKE, G, R, K, N, FAKE, ws, n, None)
    assert mx(K=96) == 2 and mx(N=100) == 2 and mx(G=0) == 2 and mx(A=None) == 1 and mx(sa=None) == 1
    assert mx(sa=FAKE + 2) == 1 and mx(sw=FAKE + 2) == 1 and mx(A=BAD) == 1 and mx(R=0) == 0
    assert mx(ws=FAKE, n=16) == 3
    gu = lambda F=128, hg=FAKE: L.moe_grouped_gemm_fwd_mx_gate_up(FAKE, FAKE, FAKE, FAKE, FAKE, 4, 100, 128, F, hg,
                                                                  FAKE, None, None, 0, None)
    assert gu(F=64) == 2 and gu(hg=None) == 1
    sb = lambda hg=FAKE, hu=FAKE: L.moe_grouped_gemm_dx_swiglu_bwd_mx(FAKE, FAKE, FAKE, FAKE, FAKE, 4, 100, 128,
                                                                      128, hg, hu, FAKE, FAKE, None, 0, None)
    assert sb(hg=None) == 1 and sb(hu=BAD) == 1
    ld = 640
    tt = lambda G=4, C=128, ld=ld, x=FAKE, qt=FAKE: L.moe_quantize_mx_tokens_t(x, FAKE, G, 100, C, qt, FAKE, ld, None)
    assert tt(G=0) == 2 and tt(C=96) == 2 and tt(ld=700) == 1 and tt(ld=512) == 1 and tt(qt=None) == 1
    assert tt(x=BAD) == 1 and tt(qt=FAKE + 8) == 1
    tb = lambda col0=0, ldr=128, qt=FAKE, st=FAKE, q_r=FAKE, sr=FAKE: L.moe_quantize_mx_tokens(
        FAKE, FAKE, 4, 100, 128, qt, st, ld, q_r, sr, ldr, col0, None)
    assert tb(col0=32, ldr=256) == 1 and tb(col0=64, ldr=128) == 1 and tb(ldr=112) == 1
    assert tb(qt=None, st=None, q_r=None, sr=None) == 1 and tb(sr=None) == 1 and tb(q_r=FAKE + 4) == 1
    dw = lambda K=128, ld=ld, c2=None, s2=None, dB2=None, cnt=None, sa=FAKE: L.moe_grouped_gemm_dw_mx(
        FAKE, sa, FAKE, FAKE, c2, s2, FAKE, 4, 100, K, 128, ld, FAKE, dB2, 0, cnt, None)
    assert dw(ld=512) == 1 and dw(ld=700) == 1 and dw(K=100) == 2 and dw(c2=FAKE, dB2=FAKE) == 1
    assert dw(cnt=FAKE + 2) == 1 and dw(sa=FAKE + 2) == 1 and dw(K=1 << 22) == 2   # operand of 2 GiB or more


def test_fwd_combine_rejects():
    L = moe.lib()
    need = L.moe_grouped_gemm_fwd_combine_workspace_bytes(50, 512)
    assert need == 50 * 2 * 4 and L.moe_grouped_gemm_fwd_combine_workspace_bytes(0, 512) == 0
    fc = lambda R=100, T=50, k=2, N=512, cnt=FAKE, n=need, y=FAKE, add=None: L.moe_grouped_gemm_fwd_combine(
        FAKE, FAKE, FAKE, 4, R, 128, N, FAKE, FAKE, FAKE, T, k, add, FAKE, y, cnt, n, None, 0, None)
    assert fc(R=99) == 1 and fc(k=0) == 1 and fc(T=-1) == 1 and fc(cnt=None) == 1 and fc(y=None) == 1
    assert fc(y=BAD) == 1 and fc(add=BAD) == 1 and fc(cnt=FAKE + 2) == 1 and fc(n=need - 4) == 3
    assert fc(R=1 << 20, T=1 << 19, N=4096) == 2          # Y_perm of 2 GiB or more
    assert fc(R=0, T=0) == 0


def test_gather_rejects():
    L = moe.lib()
    fg = lambda T=50, src=FAKE, K=128, ws=None, n=0: L.moe_grouped_gemm_fwd_gather(
        FAKE, T, src, FAKE, None, FAKE, 4, 100, K, 128, FAKE, None, None, ws, n, None)
    assert fg(src=None) == 1 and fg(T=0) == 1 and fg(T=-1) == 1 and fg(K=100) == 2
    assert fg(T=1 << 20, K=1024) == 2                     # the source must be < 2 GiB
    assert fg(ws=FAKE, n=16) == 3                         # a split workspace that is too small
    gr = lambda T=10, d=128, k=2, x=FAKE: L.moe_gather_rows(x, T, d, k, FAKE, FAKE, None)
    assert gr(d=100) == 2 and gr(k=0) == 1 and gr(x=None) == 1 and gr(x=BAD) == 1 and gr(T=0) == 0


def test_dw_t_and_transpose_rejects():
    L = moe.lib()
    assert L.moe_transposed_cols_bound(100, 4) == 128 + 128
    ld = 256
    dwt = lambda G=4, R=100, K=128, N=128, ld=ld, dC2t=None, dB2=None: L.moe_grouped_gemm_dw_t(
        FAKE, FAKE, dC2t, FAKE, G, R, K, N, ld, FAKE, dB2, 0, None)
    assert dwt(ld=192) == 1 and dwt(ld=300) == 1          # below the bound / not a multiple of 64
    assert dwt(K=100) == 2 and dwt(G=0) == 2 and dwt(dC2t=FAKE) == 1
    assert dwt(K=1 << 20, ld=1 << 12) == 2                # operand of 2 GiB or more
    tr = lambda C=128, ld=ld, src=FAKE: L.moe_transpose_grouped(src, FAKE, 4, 100, C, FAKE, ld, None)
    assert tr(C=100) == 2 and tr(ld=128) == 1 and tr(src=BAD) == 1


def test_router_rejects():
    L = moe.lib()
    assert L.moe_router_logits(FAKE, FAKE, None, 10, 100, 8, FAKE, None) == 2     # d % 64
    assert L.moe_router_logits(FAKE, FAKE, None, 10, 128, 257, FAKE, None) == 1   # E > 256
    assert L.moe_router_logits(FAKE, FAKE, None, 10, 128, 8, None, None) == 1
    assert L.moe_router_logits(BAD, FAKE, None, 10, 128, 8, FAKE, None) == 1
    assert L.moe_router_logits(FAKE, FAKE, None, 0, 128, 8, FAKE, None) == 0       # empty: no-op
    assert L.moe_router_bwd_workspace_bytes(1000, 128, 8) == (4 + 1) * 128 * 8 * 4   # 4 token chunks + Wr^T
    bwd = lambda ws=FAKE, nbytes=1 << 20, k=2, offsets=None, alpha=0.0, dx=None: L.moe_router_bwd(
        FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, offsets, 1000, 128, 8, k, 1, alpha, ws, nbytes, FAKE, FAKE, dx, None)
    assert bwd(ws=None) == 3 and bwd(nbytes=100) == 3                            # workspace
    assert bwd(k=9) == 1 and bwd(alpha=0.01) == 1                                 # k > E; aux without offsets
    assert bwd(dx=BAD) == 1
    assert L.moe_router_aux_loss(FAKE, FAKE, 100, 8, 2, 0.01, None, 0, FAKE, None) == 3
    assert L.moe_router_aux_loss(FAKE, None, 100, 8, 2, 0.01, FAKE, 1 << 20, FAKE, None) == 1


def test_elementwise_rejects():
    L = moe.lib()
    assert L.moe_swiglu(FAKE, FAKE, FAKE, 10, 100, None) == 2
    assert L.moe_swiglu(FAKE, FAKE, None, 10, 128, None) == 1
    assert L.moe_swiglu(FAKE, FAKE, FAKE, 0, 128, None) == 0
    assert L.moe_swiglu_bwd(FAKE, FAKE, FAKE, FAKE, BAD, 10, 128, None) == 1
    assert L.moe_unpermute_combine(FAKE, FAKE, FAKE, None, 10, 128, 0, FAKE, None) == 1
    assert L.moe_unpermute_combine(FAKE, FAKE, FAKE, None, 10, 96, 2, FAKE, None) == 2
    assert L.moe_unpermute_combine(FAKE, FAKE, FAKE, None, 0, 128, 2, FAKE, None) == 0
    assert L.moe_unpermute_combine_bwd(FAKE, None, FAKE, None, 10, 128, 2, FAKE, None, None) == 1


def test_binding_refuses_cpu_tensors():
    import torch
    with pytest.raises(ValueError):
        moe._ptr(torch.zeros(4))
