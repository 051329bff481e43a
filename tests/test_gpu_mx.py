"""GPU parity of the MX variant (E4M3 elements with a power-of-two E8M0 scale per 32 contraction
elements): the row and weight quantizers (codes and scale bytes bit for bit against the oracle,
both weight orientations from one read), the grouped products on MX operands (exact on
small-integer codes with random block scales, where every sum is exact in fp32; within tolerance on
quantized Gaussian data; with and without the split tail; up to 256 groups), the gate/up and the
dX-down + SwiGLU-backward forms, and the whole layer with every expert data product on MX operands
against an end-to-end oracle run, all through the C ABI."""
import sys

import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2606_26453_amd import moe
from tests.gpu_util import check_float, f64, gpu_available, poison_

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]
DEV = "cuda:0"
GROUPS = [1, 63, 64, 65, 127, 0, 128, 129, 300, 513, 0, 31]


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _u8(t):
    return t.cpu().numpy().astype(np.uint8)


def _blocks(t, C):
    """The library's MX scale array [ceil(C/128), *rows, 4] as [*rows, C/32] (padding dropped)."""
    return _u8(moe.mx_scales_by_row(t, C))


def _spread(g, shape):
    """bf16 values whose 32-element blocks span 2^-40 .. 2^40 (per block), with zero blocks."""
    *lead, C = shape
    x = torch.randn(shape, generator=g, dtype=torch.float64)
    mag = 2.0 ** torch.randint(-40, 41, tuple(lead) + (C // 32, 1), generator=g).double()
    x = (x.reshape(tuple(lead) + (C // 32, 32)) * mag).reshape(shape)
    keep = torch.rand(tuple(lead) + (C // 32, 1), generator=g) > 0.05
    return (x.reshape(tuple(lead) + (C // 32, 32)) * keep).reshape(shape).to(torch.bfloat16)


@pytest.mark.parametrize("M,K,joined", [(1, 32, False), (7, 96, True), (300, 4096 + 32, False),
                                        (33, 14336, True), (5, 2880, False), (64, 4096, True)])
def test_quantize_mx_rows(M, K, joined):
    """Codes and scale bytes bit for bit against the oracle on blocks of very different magnitudes,
    all-zero blocks and bf16 subnormals; with x2, the joined rows [x | x2]."""
    _say("quantize mx rows", M, K, joined)
    g = torch.Generator().manual_seed(M * 31 + K + joined)
    x = _spread(g, (M, K))
    if M > 3:
        x[2] = 0
        x[3, :32] = (torch.randn(32, generator=g) * 2.0 ** -131).to(torch.bfloat16)   # subnormals
    x2 = _spread(g, (M, K)) if joined else None
    C = 2 * K if joined else K
    P = moe.mx_groups(C)
    assert moe.lib().moe_mx_scale_bytes(M, C) == P * M * 4
    q = poison_(torch.empty((M, C), dtype=torch.uint8, device=DEV))
    s = poison_(torch.empty((P, M, 4), dtype=torch.uint8, device=DEV))
    moe.moe_quantize_mx_rows(x.to(DEV), None if x2 is None else x2.to(DEV), q, s)
    torch.cuda.synchronize()
    src = f64(x) if x2 is None else np.concatenate([f64(x), f64(x2)], axis=1)
    rq, rs = O.quantize_rows_mx(src)
    np.testing.assert_array_equal(_u8(q), rq)
    np.testing.assert_array_equal(_blocks(s, C), rs)


def _every_bf16_in_range():
    """Every finite bf16 value with |x| <= 448 (both zeros, subnormals, every exact tie between two
    E4M3 values), 31 to a 32-element block whose last element is 448: each block's scale is then 2^0
    (and each row's amax is 448), so every value's code is E4M3's rounding of the value itself."""
    v = torch.arange(65536, dtype=torch.int32).to(torch.int16).view(torch.bfloat16)
    v = v[torch.isfinite(v) & (v.float().abs() <= 448.0)]
    n = (v.numel() + 31 * 64 - 1) // (31 * 64) * (31 * 64)
    v = torch.cat([v, torch.zeros(n - v.numel(), dtype=torch.bfloat16)]).reshape(-1, 31)
    x = torch.cat([v, torch.full((v.shape[0], 1), 448.0, dtype=torch.bfloat16)], dim=1)
    return x.reshape(-1, 32 * 64)


def test_quantize_every_bf16_value():
    """The quantizers' E4M3 rounding (the hardware conversion) over every bf16 input in range, code
    for code against the oracle: MX rows (block scale 2^0) and fp32-scale rows (scale 1)."""
    x = _every_bf16_in_range()
    M, K = x.shape
    _say("quantize every bf16 value", M, K)
    q = poison_(torch.empty((M, K), dtype=torch.uint8, device=DEV))
    s = poison_(torch.empty((moe.mx_groups(K), M, 4), dtype=torch.uint8, device=DEV))
    moe.moe_quantize_mx_rows(x.to(DEV), None, q, s)
    q8 = poison_(torch.empty((M, K), dtype=torch.uint8, device=DEV))
    s8 = poison_(torch.empty(M, dtype=torch.float32, device=DEV))
    moe.moe_quantize_fp8_rows(x.to(DEV), q8, s8)
    torch.cuda.synchronize()
    rq, rs = O.quantize_rows_mx(f64(x))
    assert (rs == 127).all()
    np.testing.assert_array_equal(_u8(q), rq)
    np.testing.assert_array_equal(_blocks(s, K), rs)
    rq8, rs8 = O.quantize_rows_fp8(f64(x))
    assert (rs8 == 1.0).all()
    np.testing.assert_array_equal(_u8(q8), rq8)
    np.testing.assert_array_equal(s8.cpu().numpy(), rs8)
    np.testing.assert_array_equal(rq8, rq)   # the two formats agree when both scales are 1


@pytest.mark.parametrize("G,K,N,dual", [(2, 64, 64, False), (3, 224, 128, True), (2, 4096, 256, True),
                                         (1, 2880, 2880, False), (2, 512, 1408, True), (1, 14336, 128, False)])
def test_quantize_mx_weight(G, K, N, dual):
    """Both orientations from one read, bit for bit against the oracle's row quantizer: qt/st on the
    transposed weight (interleaved by 128 channels with W2), qr/sr on the rows of W (joined with W2's
    rows); each orientation alone gives the same bytes; K = 224 leaves a partial 128-row block."""
    _say("quantize mx weight", G, K, N, dual)
    gen = torch.Generator().manual_seed(G * 7 + K + N + dual)
    # magnitudes that change from block to block along both K and N
    m1 = 2.0 ** torch.randint(-20, 21, (G, K // 32, 1, N), generator=gen).double()
    m2 = 2.0 ** torch.randint(-20, 21, (G, K, N // 32, 1), generator=gen).double()
    w = (torch.randn((G, K, N), generator=gen, dtype=torch.float64) * m1.repeat_interleave(32, dim=1).reshape(G, K, N)
         * m2.repeat_interleave(32, dim=3).reshape(G, K, N)).to(torch.bfloat16)
    w[:, :, 5] = 0
    w[:, 32:64, 64:96] = 0
    w2 = _spread(gen, (G, K, N)) if dual else None
    wd, w2d = w.to(DEV), None if w2 is None else w2.to(DEV)
    n2 = 2 * N if dual else N
    qt, st, qr, sr = moe.moe_quantize_mx_weight(
        wd, w2d, qt=poison_(torch.empty((G, n2, K), dtype=torch.uint8, device=DEV)),
        st=poison_(torch.empty((moe.mx_groups(K), G, n2, 4), dtype=torch.uint8, device=DEV)),
        qr=poison_(torch.empty((G, K, n2), dtype=torch.uint8, device=DEV)),
        sr=poison_(torch.empty((moe.mx_groups(n2), G, K, 4), dtype=torch.uint8, device=DEV)))
    torch.cuda.synchronize()
    wt = w.transpose(1, 2).contiguous()
    if dual:
        wt = moe.interleave_gate_up(wt, w2.transpose(1, 2).contiguous())
    rq, rs = O.quantize_rows_mx(f64(wt))
    np.testing.assert_array_equal(_u8(qt), rq)
    np.testing.assert_array_equal(_blocks(st, K), rs)
    rows = f64(w) if not dual else np.concatenate([f64(w), f64(w2)], axis=2)
    rq, rs = O.quantize_rows_mx(rows)
    np.testing.assert_array_equal(_u8(qr), rq)
    np.testing.assert_array_equal(_blocks(sr, n2), rs)
    qt1, st1, _, _ = moe.moe_quantize_mx_weight(wd, w2d, want_r=False)
    _, _, qr1, sr1 = moe.moe_quantize_mx_weight(wd, w2d, want_t=False)
    torch.cuda.synchronize()
    assert torch.equal(qt1, qt) and torch.equal(qr1, qr)
    assert np.array_equal(_blocks(st1, K), _blocks(st, K)) and np.array_equal(_blocks(sr1, n2), _blocks(sr, n2))


def _int_codes(g, shape, lim=4):
    vals = torch.randint(-lim, lim + 1, shape, generator=g).double().numpy()
    return torch.from_numpy(O.e4m3_encode(vals))


def _scale_rows(g, rows_shape, C, lo=125, hi=129):
    """Random E8M0 bytes in [lo, hi] for the C/32 blocks of each row: [*rows, C/32]."""
    return torch.randint(lo, hi + 1, tuple(rows_shape) + (C // 32,), generator=g).to(torch.uint8)


def _scale_bytes(g, rows_shape, C, lo=125, hi=129):
    """The same in the library's MX scale layout, its padding set to 255 (the NaN scale: a product
    that read it would turn NaN)."""
    return moe.mx_scales_from_rows(_scale_rows(g, rows_shape, C, lo, hi), C, pad=255)


@pytest.mark.parametrize("K,N", [(64, 64), (256, 320), (512, 576), (2880, 192)])
def test_grouped_gemm_mx_exact(K, N):
    """Integer codes |c| <= 4 with block scales 2^-2 .. 2^2 on both sides: every partial sum is a
    multiple of 2^-4 below 2^21, exact in fp32, so the product equals the oracle bit for bit after
    the bf16 rounding; ragged and empty groups, with and without the split tail.  K = 2880 gives
    scale rows with padding (90 blocks in 92 bytes)."""
    _say("gemm mx exact", K, N)
    g = torch.Generator().manual_seed(K * 3 + N)
    G, R = len(GROUPS), sum(GROUPS)
    off = torch.tensor(np.concatenate([[0], np.cumsum(GROUPS)]), dtype=torch.int32)
    a, w = _int_codes(g, (R, K)), _int_codes(g, (G, N, K))
    sa, sw = _scale_bytes(g, (R,), K), _scale_bytes(g, (G, N), K)
    ref = O.grouped_gemm_mx(_u8(a), _blocks(sa, K), _u8(w), _blocks(sw, K), off.numpy())
    ws = moe.split_workspace(DEV)
    for wsp in (None, ws):
        C = poison_(torch.empty((R, N), dtype=torch.bfloat16, device=DEV))
        moe.moe_grouped_gemm_fwd_mx(a.to(DEV), sa.to(DEV), w.to(DEV), sw.to(DEV), off.to(DEV), C=C, workspace=wsp)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(f64(C), ref)


def test_grouped_gemm_mx_block_scales_apply_per_block():
    """One block scale raised on one side scales exactly that block's share of the sum: the product
    with A's block b of row r at byte + 3 equals the oracle's (exact data), for blocks in both halves
    of a stage (b even and odd) and in later stages."""
    _say("gemm mx per-block scales")
    g = torch.Generator().manual_seed(77)
    counts = [40, 0, 90]
    G, R, K, N = len(counts), sum(counts), 256, 256
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    a, w = _int_codes(g, (R, K)), _int_codes(g, (G, N, K))
    sa = _scale_rows(g, (R,), K, 127, 127)
    sw = _scale_rows(g, (G, N), K, 127, 127)
    for b in range(K // 32):
        sa[(5 * b) % R, b] = 130
        sw[2, (37 * b) % N, b] = 124
    sa, sw = moe.mx_scales_from_rows(sa, K), moe.mx_scales_from_rows(sw, K)
    ref = O.grouped_gemm_mx(_u8(a), _blocks(sa, K), _u8(w), _blocks(sw, K), off.numpy())
    C = moe.moe_grouped_gemm_fwd_mx(a.to(DEV), sa.to(DEV), w.to(DEV), sw.to(DEV), off.to(DEV))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(f64(C), ref)


def test_grouped_gemm_mx_split_tail_exact():
    """A tile count a few tiles past a full round and a contraction long enough to split (K = 8192):
    bitwise equal to the unsplit product, and exact against the oracle on sampled rows."""
    _say("gemm mx split tail")
    counts = [4096] * 7 + [4700]
    G, R, K, N = len(counts), sum(counts), 8192, 512
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32, device=DEV)
    g = torch.Generator(device=DEV).manual_seed(4)
    vals = torch.tensor([0x00, 0x38, 0x40, 0x44, 0x48, 0xB8, 0xC0, 0xC4, 0xC8], dtype=torch.uint8, device=DEV)
    a = vals[torch.randint(0, 9, (R, K), generator=g, device=DEV)]      # 0, +-1, +-2, +-3, +-4
    w = vals[torch.randint(0, 9, (G, N, K), generator=g, device=DEV)]
    P = moe.mx_groups(K)
    sa = torch.randint(126, 129, (P, R, 4), generator=g, device=DEV).to(torch.uint8)
    sw = torch.randint(126, 129, (P, G, N, 4), generator=g, device=DEV).to(torch.uint8)
    ws = moe.split_workspace(DEV)
    c0 = moe.moe_grouped_gemm_fwd_mx(a, sa, w, sw, off)
    c1 = moe.moe_grouped_gemm_fwd_mx(a, sa, w, sw, off, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(c0.view(torch.int16), c1.view(torch.int16))
    rng = np.random.default_rng(5)
    rows = np.sort(rng.choice(R, 48, replace=False))
    grp = np.searchsorted(np.concatenate([[0], np.cumsum(counts)]), rows, side="right") - 1
    sub = np.concatenate([[0], np.cumsum(np.bincount(grp, minlength=G))])
    ridx = torch.tensor(rows, device=DEV)
    ref = O.grouped_gemm_mx(_u8(a[ridx]), _blocks(sa[:, ridx], K), _u8(w), _blocks(sw, K), sub)
    np.testing.assert_array_equal(f64(c1[ridx]), ref)


@pytest.mark.parametrize("K,N", [(1024, 512), (2880, 2880)])
def test_grouped_gemm_mx_quantized_gaussian(K, N):
    """bf16 activations and weights quantized on the GPU (codes checked bit for bit against the
    oracle's), the product against the oracle's product of its own codes (fp32 accumulation:
    Frobenius error <= 1e-3); the deviation from the unquantized bf16 product is reported."""
    _say("gemm mx gaussian", K, N)
    g = torch.Generator().manual_seed(K + N)
    counts = [300, 0, 1000, 77, 513]
    G, R = len(counts), sum(counts)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    x = torch.randn((R, K), generator=g).to(torch.bfloat16)
    wt = (torch.randn((G, N, K), generator=g) * 0.02).to(torch.bfloat16)
    aq, sa = moe.moe_quantize_mx_rows(x.to(DEV))
    wq, sw = moe.moe_quantize_mx_rows(wt.to(DEV))
    C = moe.moe_grouped_gemm_fwd_mx(aq, sa, wq, sw, off.to(DEV), workspace=moe.split_workspace(DEV))
    torch.cuda.synchronize()
    ra, rsa = O.quantize_rows_mx(f64(x))
    rw, rsw = O.quantize_rows_mx(f64(wt))
    np.testing.assert_array_equal(_u8(aq), ra)
    np.testing.assert_array_equal(_blocks(sw, K), rsw)
    ref = O.grouped_gemm_mx(ra, rsa, rw, rsw, off.numpy())
    check_float("C mx", f64(C), ref, 1e-3)
    exact = O.grouped_gemm(f64(x), np.transpose(f64(wt), (0, 2, 1)), off.numpy(), rnd=None)
    err = O.rel_fro(f64(C), exact)
    _say(f"mx vs unquantized bf16 product: relative Frobenius {err:.3e}")
    assert err < 0.1


@pytest.mark.parametrize("K,F", [(64, 128), (512, 384), (2048, 1408)])
def test_grouped_gemm_mx_gate_up(K, F):
    """The gate/up product over the weight moe_quantize_mx_weight interleaves by 128 channels equals
    the two separate MX products (on the gate and up codes of the same call) bit for bit, and its
    SwiGLU equals moe_swiglu on those outputs bit for bit; with and without the split tail."""
    _say("gemm mx gate/up", K, F)
    g = torch.Generator().manual_seed(K + F)
    G, R = len(GROUPS), sum(GROUPS)
    off = torch.tensor(np.concatenate([[0], np.cumsum(GROUPS)]), dtype=torch.int32, device=DEV)
    x = torch.randn((R, K), generator=g).to(torch.bfloat16).to(DEV)
    wg = (torch.randn((G, K, F), generator=g) * 0.05).to(torch.bfloat16).to(DEV)
    wu = (torch.randn((G, K, F), generator=g) * 0.05).to(torch.bfloat16).to(DEV)
    aq, sa = moe.moe_quantize_mx_rows(x)
    iq, is_, _, _ = moe.moe_quantize_mx_weight(wg, wu, want_r=False)
    P = is_.shape[0]
    gq = iq.reshape(G, F // 128, 2, 128, K)[:, :, 0].reshape(G, F, K).contiguous()
    uq = iq.reshape(G, F // 128, 2, 128, K)[:, :, 1].reshape(G, F, K).contiguous()
    gs = is_.reshape(P, G, F // 128, 2, 128, 4)[:, :, :, 0].reshape(P, G, F, 4).contiguous()
    us = is_.reshape(P, G, F // 128, 2, 128, 4)[:, :, :, 1].reshape(P, G, F, 4).contiguous()
    hg = moe.moe_grouped_gemm_fwd_mx(aq, sa, gq, gs, off)
    hu = moe.moe_grouped_gemm_fwd_mx(aq, sa, uq, us, off)
    act = moe.moe_swiglu(hg, hu)
    for ws in (None, moe.split_workspace(DEV)):
        h1, h2, a1 = moe.moe_grouped_gemm_fwd_mx_gate_up(aq, sa, iq, is_, off, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(h1.view(torch.int16), hg.view(torch.int16))
        assert torch.equal(h2.view(torch.int16), hu.view(torch.int16))
        assert torch.equal(a1.view(torch.int16), act.view(torch.int16))


@pytest.mark.parametrize("K,N", [(64, 128), (256, 320), (512, 576)])
def test_dx_swiglu_bwd_mx_exact(K, N):
    """The MX dX-down product with the SwiGLU backward in its epilogue, on small-integer codes with
    random block scales (every sum exact in fp32): bitwise equal to the bf16 product with the same
    epilogue (moe_grouped_gemm_dx_swiglu_bwd) on the decoded operands, with and without the split
    tail, over ragged and empty groups; and against the oracle's SwiGLU backward of the oracle's MX
    product."""
    _say("dx swiglu bwd mx exact", K, N)
    g = torch.Generator().manual_seed(K * 5 + N)
    G, R = len(GROUPS), sum(GROUPS)
    off = torch.tensor(np.concatenate([[0], np.cumsum(GROUPS)]), dtype=torch.int32)
    a, w = _int_codes(g, (R, K)), _int_codes(g, (G, N, K))
    sa, sw = _scale_bytes(g, (R,), K), _scale_bytes(g, (G, N), K)
    hg = torch.randn((R, N), generator=g).to(torch.bfloat16)
    hu = torch.randn((R, N), generator=g).to(torch.bfloat16)
    D = lambda t: t.contiguous().to(DEV)
    dec = lambda c, s_: torch.from_numpy(O.mx_decode(_u8(c), _blocks(s_, K))).to(torch.bfloat16)
    rg, ru = moe.moe_grouped_gemm_dx_swiglu_bwd(D(dec(a, sa)), D(dec(w, sw)), D(off), D(hg), D(hu))
    da = O.grouped_gemm_mx(_u8(a), _blocks(sa, K), _u8(w), _blocks(sw, K), off.numpy())
    og, ou = O.swiglu_bwd(f64(hg), f64(hu), da)
    for ws in (None, moe.split_workspace(DEV)):
        dg, du = moe.moe_grouped_gemm_dx_swiglu_bwd_mx(D(a), D(sa), D(w), D(sw), D(off), D(hg), D(hu), workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(dg.view(torch.int16), rg.view(torch.int16))
        assert torch.equal(du.view(torch.int16), ru.view(torch.int16))
        check_float("dh_gate", f64(dg), og, 2e-3)
        check_float("dh_up", f64(du), ou, 2e-3)


def test_grouped_gemm_mx_256_groups_exact():
    """The maximum group count (G = 256, empty groups included, more row tiles than CUs): the MX
    product and the MX gate/up product exact against the oracle on integer codes."""
    _say("gemm mx 256 groups")
    rng = np.random.default_rng(2561)
    counts = rng.integers(0, 400, 256)
    counts[rng.choice(256, 20, replace=False)] = 0
    G, R, K, N = 256, int(counts.sum()), 128, 256
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    g = torch.Generator().manual_seed(2561)
    a, w, w2 = _int_codes(g, (R, K)), _int_codes(g, (G, N, K)), _int_codes(g, (G, N, K))
    sa, sw, sw2 = _scale_bytes(g, (R,), K), _scale_rows(g, (G, N), K), _scale_rows(g, (G, N), K)
    isc = moe.mx_scales_from_rows(moe.interleave_gate_up(sw, sw2), K).to(DEV)
    sw, sw2 = moe.mx_scales_from_rows(sw, K), moe.mx_scales_from_rows(sw2, K)
    ws = moe.split_workspace(DEV)
    C = moe.moe_grouped_gemm_fwd_mx(a.to(DEV), sa.to(DEV), w.to(DEV), sw.to(DEV), off.to(DEV), workspace=ws)
    iq = moe.interleave_gate_up(w.to(DEV), w2.to(DEV))
    hg, hu, act = moe.moe_grouped_gemm_fwd_mx_gate_up(a.to(DEV), sa.to(DEV), iq, isc, off.to(DEV), workspace=ws)
    torch.cuda.synchronize()
    ref = O.grouped_gemm_mx(_u8(a), _blocks(sa, K), _u8(w), _blocks(sw, K), off.numpy())
    np.testing.assert_array_equal(f64(C), ref)
    np.testing.assert_array_equal(f64(hg), ref)
    np.testing.assert_array_equal(f64(hu), O.grouped_gemm_mx(_u8(a), _blocks(sa, K), _u8(w2), _blocks(sw2, K),
                                                             off.numpy()))
    check_float("act", f64(act), O.swiglu(f64(hg), f64(hu)), 1e-2)


# ------------------------------------------------------------------------------------------------
# The weight gradient on MX operands quantized along the tokens
# ------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("counts,C", [([5, 0, 130, 128, 1, 300], 64), ([129, 127, 0, 0, 256], 320),
                                      ([1], 128), ([700, 3, 41], 192), ([129, 1, 300, 0], 384)])
def test_quantize_mx_tokens_t(counts, C):
    """Token-major codes and scales bit for bit against the oracle's packing (each expert's rows as
    columns from a 128-aligned start, zeros in the padding) quantized row by row; empty groups,
    groups of 1, 127, 128, 129 rows; blocks of very different magnitudes."""
    _say("quantize mx tokens", counts, C)
    g = torch.Generator().manual_seed(sum(counts) + C)
    R = sum(counts)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    mag = 2.0 ** torch.randint(-20, 21, (R, 1), generator=g).double() * 2.0 ** torch.randint(-20, 21, (1, C),
                                                                                             generator=g).double()
    x = (torch.randn((R, C), generator=g, dtype=torch.float64) * mag).to(torch.bfloat16)
    x[::7] = 0                                         # zero rows, so some blocks are all zero
    G = len(counts)
    ld = moe.mx_tokens_cols(R, G)
    qt = poison_(torch.empty((C, ld), dtype=torch.uint8, device=DEV))
    st = poison_(torch.empty((ld // 128, C, 4), dtype=torch.uint8, device=DEV))
    moe.moe_quantize_mx_tokens_t(x.to(DEV), off.to(DEV), qt, st)
    torch.cuda.synchronize()
    packed, p = O.pack_groups_t(f64(x), off.numpy())
    L = int(p[-1])
    rq, rs = O.quantize_rows_mx(packed)
    np.testing.assert_array_equal(_u8(qt)[:, :L], rq)
    np.testing.assert_array_equal(_blocks(st, ld)[:, : L // 32], rs)


@pytest.mark.parametrize("counts,C", [([5, 0, 130, 128, 1, 300], 64), ([700, 3, 41], 192),
                                      ([129, 1, 300, 0], 256)])   # 128-column tiles (C, col0 % 128 == 0)
def test_quantize_mx_tokens_both(counts, C):
    """moe_quantize_mx_tokens: from one read, the token-major codes (equal to
    moe_quantize_mx_tokens_t's) and the row codes bit for bit against the oracle's row quantizer;
    two calls at col0 = 0 and C fill the joined rows [x | x2] as the oracle quantizes them."""
    _say("quantize mx tokens both", counts, C)
    g = torch.Generator().manual_seed(3 * sum(counts) + C)
    R, G = sum(counts), len(counts)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32, device=DEV)
    mk = lambda: (torch.randn((R, C), generator=g, dtype=torch.float64)
                  * 2.0 ** torch.randint(-20, 21, (R, C // 32), generator=g).double().repeat_interleave(32, dim=1)
                  ).to(torch.bfloat16)
    x, x2 = mk(), mk()
    qt0, st0 = moe.moe_quantize_mx_tokens_t(x.to(DEV), off)
    qt, st, qr, sr = moe.moe_quantize_mx_tokens(x.to(DEV), off)
    torch.cuda.synchronize()
    L = int(O.pack_groups_t(np.zeros((R, 1)), off.cpu().numpy())[1][-1])
    assert torch.equal(qt[:, :L], qt0[:, :L])
    assert np.array_equal(_blocks(st, qt.shape[1])[:, : L // 32], _blocks(st0, qt.shape[1])[:, : L // 32])
    rq, rs = O.quantize_rows_mx(f64(x))
    np.testing.assert_array_equal(_u8(qr), rq)
    np.testing.assert_array_equal(_blocks(sr, C), rs)
    jq = poison_(torch.empty((R, 2 * C), dtype=torch.uint8, device=DEV))
    js = poison_(torch.empty((moe.mx_groups(2 * C), R, 4), dtype=torch.uint8, device=DEV))
    moe.moe_quantize_mx_tokens(x.to(DEV), off, qr=jq, sr=js, col0=0, want_t=False)
    moe.moe_quantize_mx_tokens(x2.to(DEV), off, qr=jq, sr=js, col0=C, want_t=False)
    torch.cuda.synchronize()
    rq, rs = O.quantize_rows_mx(np.concatenate([f64(x), f64(x2)], axis=1))
    np.testing.assert_array_equal(_u8(jq), rq)
    np.testing.assert_array_equal(_blocks(js, 2 * C), rs)


def _tokens_operand(g, rows, counts, lo=125, hi=129):
    """Integer codes |c| <= 4 in the token-major layout (zeros in each group's padding) and random
    scale bytes: (codes [rows, ld], scales in the library's layout, scale bytes [rows, ld/32])."""
    G, R = len(counts), sum(counts)
    ld = moe.mx_tokens_cols(R, G)
    _, p = O.pack_groups_t(np.zeros((R, 1)), np.concatenate([[0], np.cumsum(counts)]))
    codes = torch.zeros((rows, ld), dtype=torch.uint8)
    for i in range(G):
        codes[:, p[i]:p[i] + counts[i]] = _int_codes(g, (rows, counts[i]))
    sb = _scale_rows(g, (rows,), ld, lo, hi)
    return codes, moe.mx_scales_from_rows(sb, ld), sb


@pytest.mark.parametrize("K,N,dual,out16", [(64, 64, False, False), (320, 192, True, False),
                                             (256, 512, False, True), (192, 320, True, True)])
def test_grouped_gemm_dw_mx_exact(K, N, dual, out16):
    """Integer codes with block scales 2^-2 .. 2^2 along the tokens: every partial sum is exact in
    fp32, so dW (fp32) equals the oracle's ragged MX weight gradient exactly (bf16 output: its
    rounding); empty groups give exact zeros; the dual form reads one At for two outputs."""
    _say("dw mx exact", K, N, dual, out16)
    g = torch.Generator().manual_seed(K * 7 + N + dual)
    counts = [5, 0, 130, 128, 1, 300, 0, 61]
    G, R = len(counts), sum(counts)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    a, sa, sab = _tokens_operand(g, K, counts)
    c, sc, scb = _tokens_operand(g, N, counts)
    c2, sc2, sc2b = _tokens_operand(g, N, counts) if dual else (None, None, None)
    rnd = O.bf16_round if out16 else (lambda v: v)
    ref = rnd(O.grouped_gemm_dw_mx(_u8(a), _u8(sab), _u8(c), _u8(scb), off.numpy()))
    D = lambda t: None if t is None else t.to(DEV)
    ref2 = rnd(O.grouped_gemm_dw_mx(_u8(a), _u8(sab), _u8(c2), _u8(sc2b), off.numpy())) if dual else None
    for cnt in (None, moe.dw_counters(DEV)):   # one workgroup per tile; persistent with tile claims
        out = moe.moe_grouped_gemm_dw_mx(D(a), D(sa), D(c), D(sc), D(off), R, D(c2), D(sc2), out_bf16=out16,
                                         counters=cnt)
        torch.cuda.synchronize()
        dB = out[0] if dual else out
        np.testing.assert_array_equal(f64(dB), ref)
        if dual:
            np.testing.assert_array_equal(f64(out[1]), ref2)


# ------------------------------------------------------------------------------------------------
# The layer with its expert data products on MX operands, against an end-to-end oracle run
# ------------------------------------------------------------------------------------------------
def _oracle_layer_mx(inp, cfg, mx_dw=False, mx_fwd=True, mx_bwd=True):
    """The layer's forward and backward with the expert data products on MX operands (mx_fwd: the
    forward's, X_perm and the SwiGLU output quantized per 32-element block of their rows; mx_bwd:
    the data gradient's, dY_perm and [dH_gate | dH_up]; the weights per block of the matching
    contraction), with mx_dw the weight gradients on operands quantized along the tokens, and
    everything else as the bf16 oracle."""
    x = f64(inp["x"])
    wg, wu, wd = (f64(inp[n]) for n in ("w_gate", "w_up", "w_down"))
    shared = None
    if cfg.f_shared:
        shared = tuple(f64(inp[n]) for n in ("w_gate_sh", "w_up_sh", "w_down_sh"))
    k = cfg.k
    idx, tw = O.route_topk(inp["logits"].numpy(), k)
    off, ros, tor = O.permute(idx, cfg.E)
    xp = O.gather(x, tor)
    q = O.quantize_rows_mx
    xq, xs = q(xp)
    gq, gs = q(np.transpose(wg, (0, 2, 1)))
    uq, us = q(np.transpose(wu, (0, 2, 1)))
    dq, ds = q(np.transpose(wd, (0, 2, 1)))
    if mx_fwd:
        hg = O.grouped_gemm_mx(xq, xs, gq, gs, off)
        hu = O.grouped_gemm_mx(xq, xs, uq, us, off)
    else:
        hg, hu = O.grouped_gemm(xp, wg, off), O.grouped_gemm(xp, wu, off)
    act = O.swiglu(hg, hu)
    aq, as_ = q(act)
    y_perm = O.grouped_gemm_mx(aq, as_, dq, ds, off) if mx_fwd else O.grouped_gemm(act, wd, off)
    fwd = {"offsets": off, "row_of_slot": ros, "topk_w": tw, "y_perm": y_perm}
    y_sh = None
    if shared is not None:
        fwd["shared"] = O.dense_ffn_forward(x, *shared)
        y_sh = fwd["shared"]["y"]
    y = O.combine(y_perm, tw, ros, k, add=y_sh)
    dy = f64(inp["dy"])
    dy_perm, _ = O.combine_bwd(dy, tw, ros, y_perm, k)
    yq, ys = q(dy_perm)
    wdq, wds = q(wd)                                           # rows of W_down [E, f, d]
    da = O.grouped_gemm_mx(yq, ys, wdq, wds, off) if mx_bwd else O.grouped_gemm_dx(dy_perm, wd, off)
    dhg, dhu = O.swiglu_bwd(hg, hu, da)
    hq, hs = q(np.concatenate([dhg, dhu], axis=1))
    wjq, wjs = q(np.concatenate([wg, wu], axis=2))             # rows [W_gate | W_up] [E, d, 2f]
    dx_perm = (O.grouped_gemm_mx(hq, hs, wjq, wjs, off) if mx_bwd
               else O.grouped_gemm_dx(dhg, wg, off, dhu, wu))
    dx_sh = None
    if shared is not None:
        dx_sh = O.dense_ffn_backward(fwd["shared"], x, dy, *shared)["dx"]
    dx = O.combine(dx_perm, None, ros, k, add=dx_sh)
    if mx_dw:   # operands quantized along the tokens (the packed, 128-aligned token-major form)
        qt = lambda v: q(O.pack_groups_t(v, off)[0])
        dws = {"dw_down": O.grouped_gemm_dw_mx(*qt(act), *qt(dy_perm), off),
               "dw_gate": O.grouped_gemm_dw_mx(*qt(xp), *qt(dhg), off),
               "dw_up": O.grouped_gemm_dw_mx(*qt(xp), *qt(dhu), off)}
    else:
        dws = {"dw_down": O.grouped_gemm_dw(act, dy_perm, off), "dw_gate": O.grouped_gemm_dw(xp, dhg, off),
               "dw_up": O.grouped_gemm_dw(xp, dhu, off)}
    return {"y": y, "y_perm": y_perm, "h_gate": hg, "h_up": hu, "act": act, "dy_perm": dy_perm,
            "dh_gate": dhg, "dh_up": dhu, "dx_perm": dx_perm, "dx": dx, **dws,
            "w": {"gate_up_t": (gq, gs, uq, us), "down_t": (dq, ds), "down_r": (wdq, wds),
                  "gate_up_r": (wjq, wjs)}}


@pytest.mark.parametrize("cfg_id,mx_dw,fwd,bwd", [(0, False, True, True), (2, False, True, True),
                                                  (0, True, True, True), (2, True, True, True),
                                                  (0, True, False, True), (0, True, True, False)])
def test_layer_mx(cfg_id, mx_dw, fwd, bwd):
    """The layer with MX forward and data-gradient products (fp8_forward, fp8_backward, mx), two
    steps (the second re-quantizes the weights, both orientations from one read per weight): the
    weight codes and scale bytes bit for bit, and every output and gradient against the end-to-end
    oracle run, which quantizes its own bf16 intermediates (a code may differ where the two sides'
    bf16 intermediates differ in the last bit; the tolerances cover that).  With mx_dw the weight
    gradients run on operands quantized along the tokens as well; with only one of the forward and
    data-gradient products in MX, the other stays bf16 and the token-major codes of the tensors it
    does not quantize come from the token-only quantization.  Config 2 at 1024 tokens."""
    import dataclasses
    from paper_2606_26453_amd import layer as L, workloads as W
    cfg = W.CONFIGS[cfg_id]
    if cfg_id:
        cfg = dataclasses.replace(cfg, T=1024)
    _say("layer mx", cfg, mx_dw, fwd, bwd)
    inp = W.make_inputs(cfg, 0, "cpu")
    lay = L.MoELayer(cfg, {k_: v.to(DEV) for k_, v in inp.items()}, fp8_forward=fwd, fp8_backward=bwd, mx=True,
                     fp8_dw=mx_dw)
    lay.step()
    lay.step()
    torch.cuda.synchronize()
    b = lay.buf
    ref = _oracle_layer_mx(inp, cfg, mx_dw, fwd, bwd)
    d, f, E = cfg.d, cfg.f, cfg.E
    assert set(lay.wmx) == ({"gate_up_t", "down_t"} if fwd else set()) | ({"gate_up_r", "down_r"} if bwd else set())
    if fwd:
        gq, gs, uq, us = ref["w"]["gate_up_t"]
        lq = _u8(lay.wmx["gate_up_t"][0]).reshape(E, f // 128, 2, 128, d)
        ls = _blocks(lay.wmx["gate_up_t"][1], d).reshape(E, f // 128, 2, 128, d // 32)
        np.testing.assert_array_equal(lq[:, :, 0].reshape(E, f, d), gq)
        np.testing.assert_array_equal(lq[:, :, 1].reshape(E, f, d), uq)
        np.testing.assert_array_equal(ls[:, :, 0].reshape(E, f, d // 32), gs)
        np.testing.assert_array_equal(ls[:, :, 1].reshape(E, f, d // 32), us)
        np.testing.assert_array_equal(_u8(lay.wmx["down_t"][0]), ref["w"]["down_t"][0])
        np.testing.assert_array_equal(_blocks(lay.wmx["down_t"][1], f), ref["w"]["down_t"][1])
    if bwd:
        np.testing.assert_array_equal(_u8(lay.wmx["down_r"][0]), ref["w"]["down_r"][0])
        np.testing.assert_array_equal(_blocks(lay.wmx["down_r"][1], d), ref["w"]["down_r"][1])
        np.testing.assert_array_equal(_u8(lay.wmx["gate_up_r"][0]), ref["w"]["gate_up_r"][0])
        np.testing.assert_array_equal(_blocks(lay.wmx["gate_up_r"][1], 2 * f), ref["w"]["gate_up_r"][1])
    for key in ("h_gate", "h_up", "act", "y_perm", "y", "dy_perm", "dh_gate", "dh_up", "dx_perm", "dx"):
        check_float(key, f64(b[key]), ref[key], 1e-2)
    for key in ("dw_down", "dw_gate", "dw_up"):
        check_float(key, f64(b[key]), ref[key], 1e-2)
    x = f64(inp["x"])
    wg, wu, wd = (f64(inp[n]) for n in ("w_gate", "w_up", "w_down"))
    shared = None
    if cfg.f_shared:
        shared = tuple(f64(inp[n]) for n in ("w_gate_sh", "w_up_sh", "w_down_sh"))
    bf = O.layer_forward(x, inp["logits"].numpy(), wg, wu, wd, cfg.k, shared=shared)
    bb = O.layer_backward(bf, x, f64(inp["dy"]), wg, wu, wd, shared=shared)
    _say(f"mx layer vs the all-bf16 oracle: Y {O.rel_fro(f64(b['y']), bf['y']):.3e}, "
         f"dX {O.rel_fro(f64(b['dx']), bb['dx']):.3e}")


def test_mx_fullsize_sampled():
    """The three MX expert products at the Mixtral-shaped layer's full size (R = 16384 routed rows
    over 8 experts, d = 4096, f = 14336), in the launch configuration the benchmark times (split
    tail on, weights quantized by moe_quantize_mx_weight), each on seeded Gaussian inputs of its
    own: gate/up + SwiGLU, the down product, and the dX-down product with its SwiGLU backward.
    16 sampled rows x 64 sampled columns of the first and of the last expert against the oracle's
    product of its own codes of those rows and of the matching weight channels."""
    from paper_2606_26453_amd import workloads as W
    cfg = W.CONFIGS[1]
    R, d, f, E = cfg.T * cfg.k, cfg.d, cfg.f, cfg.E
    _say("mx full size", R, d, f, E)
    g = torch.Generator(device=DEV).manual_seed(13)
    counts = [R // E] * E
    off_np = np.concatenate([[0], np.cumsum(counts)])
    off = torch.tensor(off_np, dtype=torch.int32, device=DEV)
    rnd = lambda shape, s=1.0: (torch.randn(shape, generator=g, device=DEV) * s).to(torch.bfloat16)
    x, act0, dy = rnd((R, d)), rnd((R, f)), rnd((R, d), 1e-3)
    hg0, hu0 = rnd((R, f)), rnd((R, f))
    ws = moe.split_workspace(DEV)
    wg, wu, wd = rnd((E, d, f), 0.02), rnd((E, d, f), 0.02), rnd((E, f, d), 0.02)
    iq, is_, _, _ = moe.moe_quantize_mx_weight(wg, wu, want_r=False)
    dq, ds, rq, rs = moe.moe_quantize_mx_weight(wd)
    xq, xs = moe.moe_quantize_mx_rows(x)
    hg, hu, act = moe.moe_grouped_gemm_fwd_mx_gate_up(xq, xs, iq, is_, off, workspace=ws)
    aq, as_ = moe.moe_quantize_mx_rows(act0)
    y = moe.moe_grouped_gemm_fwd_mx(aq, as_, dq, ds, off, workspace=ws)
    yq, ys = moe.moe_quantize_mx_rows(dy)
    dhg, dhu = moe.moe_grouped_gemm_dx_swiglu_bwd_mx(yq, ys, rq, rs, off, hg0, hu0, workspace=ws)
    torch.cuda.synchronize()
    rng = np.random.default_rng(14)
    q = O.quantize_rows_mx
    for e in (0, E - 1):
        rows = np.sort(rng.choice(np.arange(off_np[e], off_np[e + 1]), 16, replace=False))
        cf = np.sort(rng.choice(f, 64, replace=False))
        cd = np.sort(rng.choice(d, 64, replace=False))
        ridx, cfi, cdi = (torch.tensor(v, device=DEV) for v in (rows, cf, cd))
        sub = np.array([0, 16])
        pick = lambda t, cols: f64(t[ridx][:, cols])
        # gate/up + SwiGLU: channels cf of W_gate and W_up (columns of the stored [d, f] weights)
        xr, xrs = q(f64(x[ridx]))
        gqe, gse = q(f64(wg[e][:, cfi]).T[None])
        uqe, use = q(f64(wu[e][:, cfi]).T[None])
        rg = O.grouped_gemm_mx(xr, xrs, gqe, gse, sub)
        ru = O.grouped_gemm_mx(xr, xrs, uqe, use, sub)
        check_float(f"h_gate e{e}", pick(hg, cfi), rg, 2e-3)
        check_float(f"h_up e{e}", pick(hu, cfi), ru, 2e-3)
        check_float(f"act e{e}", pick(act, cfi), O.swiglu(rg, ru), 4e-3)
        # down: channels cd of W_down (columns of the stored [f, d] weight)
        ar, ars = q(f64(act0[ridx]))
        dqe, dse = q(f64(wd[e][:, cdi]).T[None])
        check_float(f"y e{e}", pick(y, cdi), O.grouped_gemm_mx(ar, ars, dqe, dse, sub), 2e-3)
        # dX down + SwiGLU backward: channels cf of dA (rows of the stored [f, d] weight)
        yr, yrs = q(f64(dy[ridx]))
        rqe, rse = q(f64(wd[e][cfi])[None])
        og, ou = O.swiglu_bwd(pick(hg0, cfi), pick(hu0, cfi), O.grouped_gemm_mx(yr, yrs, rqe, rse, sub))
        check_float(f"dh_gate e{e}", pick(dhg, cfi), og, 4e-3)
        check_float(f"dh_up e{e}", pick(dhu, cfi), ou, 4e-3)


def test_mx_dw_fullsize_sampled():
    """The MX weight gradients at the Mixtral-shaped layer's full size (R = 16384 routed rows over 8
    experts, d = 4096, f = 14336) on seeded Gaussian operands: the four token-major quantizations and
    the dual gate/up and single down products as the layer runs them; 16 sampled rows x 64 sampled
    columns of each output for the first and the last expert against the oracle's MX weight
    gradient of its own token-major codes of the sampled columns."""
    from paper_2606_26453_amd import workloads as W
    cfg = W.CONFIGS[1]
    R, d, f, E = cfg.T * cfg.k, cfg.d, cfg.f, cfg.E
    _say("mx dW full size", R, d, f, E)
    g = torch.Generator(device=DEV).manual_seed(15)
    counts = [R // E - 37, R // E + 37] * (E // 2)
    off_np = np.concatenate([[0], np.cumsum(counts)])
    off = torch.tensor(off_np, dtype=torch.int32, device=DEV)
    rnd = lambda shape, s_=1.0: (torch.randn(shape, generator=g, device=DEV) * s_).to(torch.bfloat16)
    x, act, dy, dhg, dhu = rnd((R, d)), rnd((R, f)), rnd((R, d), 1e-3), rnd((R, f), 1e-3), rnd((R, f), 1e-3)
    xq, xs = moe.moe_quantize_mx_tokens_t(x, off)
    aq, as_ = moe.moe_quantize_mx_tokens_t(act, off)
    yq, ys = moe.moe_quantize_mx_tokens_t(dy, off)
    gq, gs = moe.moe_quantize_mx_tokens_t(dhg, off)
    uq, us = moe.moe_quantize_mx_tokens_t(dhu, off)
    dw_g, dw_u = moe.moe_grouped_gemm_dw_mx(xq, xs, gq, gs, off, R, uq, us)
    del xq, gq, uq
    dw_d = moe.moe_grouped_gemm_dw_mx(aq, as_, yq, ys, off, R)
    torch.cuda.synchronize()
    rng = np.random.default_rng(16)
    q = O.quantize_rows_mx
    qt = lambda t, cols: q(O.pack_groups_t(f64(t[:, torch.tensor(cols, device=DEV)]), off_np)[0])
    for e in (0, E - 1):
        rd = np.sort(rng.choice(d, 16, replace=False))
        cf = np.sort(rng.choice(f, 64, replace=False))
        rf = np.sort(rng.choice(f, 16, replace=False))
        cd = np.sort(rng.choice(d, 64, replace=False))
        pick = lambda t, r, c: f64(t[e][torch.tensor(r, device=DEV)][:, torch.tensor(c, device=DEV)])
        xr = qt(x, rd)
        check_float(f"dw_gate e{e}", pick(dw_g, rd, cf), O.grouped_gemm_dw_mx(*xr, *qt(dhg, cf), off_np)[e], 2e-3)
        check_float(f"dw_up e{e}", pick(dw_u, rd, cf), O.grouped_gemm_dw_mx(*xr, *qt(dhu, cf), off_np)[e], 2e-3)
        check_float(f"dw_down e{e}", pick(dw_d, rf, cd), O.grouped_gemm_dw_mx(*qt(act, rf), *qt(dy, cd), off_np)[e],
                    2e-3)
