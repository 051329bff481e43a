"""GPU parity of the FP8 variant of the forward product: the per-row E4M3 quantizer (codes and
scales bit for bit against the oracle) and the grouped product on E4M3 operands (exact on
small-integer codes with power-of-two scales, where every sum is exact in fp32; within tolerance on
quantized Gaussian data; with and without the split tail), all through the C ABI."""
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


@pytest.mark.parametrize("M,K", [(1, 16), (7, 64), (300, 4096 + 16), (64, 14336), (5, 2880)])
def test_quantize_fp8_rows(M, K):
    _say("quantize fp8", M, K)
    g = torch.Generator().manual_seed(M + K)
    x = (torch.randn((M, K), generator=g) * torch.exp(torch.randn((M, 1), generator=g) * 3)).to(torch.bfloat16)
    if M > 3:
        x[2] = 0
        x[3, : K // 2] = 0
    q = poison_(torch.empty((M, K), dtype=torch.uint8, device=DEV))
    s = poison_(torch.empty(M, dtype=torch.float32, device=DEV))
    moe.moe_quantize_fp8_rows(x.to(DEV), q, s)
    torch.cuda.synchronize()
    rq, rs = O.quantize_rows_fp8(f64(x))
    np.testing.assert_array_equal(_u8(q), rq)
    np.testing.assert_array_equal(s.cpu().numpy(), rs)


@pytest.mark.parametrize("G,K,N,dual", [(2, 64, 64, False), (3, 208, 128, True), (2, 4096, 256, True),
                                         (1, 2880, 2880, False), (2, 512, 1408, True), (1, 14336, 128, False),
                                         (2, 4112, 256, True)])
def test_quantize_fp8_weight(G, K, N, dual):
    """The one-pass weight quantizer (transpose, optional 128-channel gate/up interleave, per-channel
    E4M3): codes and scales bit for bit against the oracle's row quantizer on the transposed
    (interleaved) weight and against moe_quantize_fp8_rows on the GPU; zero and half-zero columns
    included; K = 208 leaves a partial block of rows, K = 14336 and 4112 span several 4096-row chunks
    (the last one partial)."""
    _say("quantize fp8 weight", G, K, N, dual)
    gen = torch.Generator().manual_seed(G * 7 + K + N)
    mk = lambda: (torch.randn((G, K, N), generator=gen) * torch.exp(torch.randn((G, 1, N), generator=gen) * 3)
                  ).to(torch.bfloat16)
    w = mk()
    w[:, :, 5] = 0
    w[0, : K // 2, 7] = 0
    w2 = mk() if dual else None
    q, sc = moe.moe_quantize_fp8_weight(w.to(DEV), None if w2 is None else w2.to(DEV),
                                        q=poison_(torch.empty((G, 2 * N if dual else N, K), dtype=torch.uint8, device=DEV)),
                                        scale=poison_(torch.empty((G, 2 * N if dual else N), dtype=torch.float32, device=DEV)))
    torch.cuda.synchronize()
    wt = w.transpose(1, 2).contiguous()
    if dual:
        wt = moe.interleave_gate_up(wt, w2.transpose(1, 2).contiguous())
    rq, rs = O.quantize_rows_fp8(f64(wt.reshape(-1, K)))
    np.testing.assert_array_equal(_u8(q).reshape(-1, K), rq)
    np.testing.assert_array_equal(sc.cpu().numpy().reshape(-1), rs)
    q2, s2 = moe.moe_quantize_fp8_rows(wt.to(DEV))
    torch.cuda.synchronize()
    assert torch.equal(q2, q) and torch.equal(s2, sc)


def _int_codes(g, shape, lim=4):
    vals = torch.randint(-lim, lim + 1, shape, generator=g).double().numpy()
    return torch.from_numpy(O.e4m3_encode(vals))


def _pow2(g, shape):
    return (2.0 ** torch.randint(-3, 3, shape, generator=g)).float()


@pytest.mark.parametrize("K,N", [(64, 64), (256, 320), (512, 576)])
def test_grouped_gemm_fp8_exact(K, N):
    _say("gemm fp8 exact", K, N)
    g = torch.Generator().manual_seed(K * 3 + N)
    G, R = len(GROUPS), sum(GROUPS)
    off = torch.tensor(np.concatenate([[0], np.cumsum(GROUPS)]), dtype=torch.int32)
    a, w = _int_codes(g, (R, K)), _int_codes(g, (G, N, K))
    sa, sw = _pow2(g, (R,)), _pow2(g, (G, N))
    ref = O.grouped_gemm_fp8(_u8(a), sa.numpy(), _u8(w), sw.numpy(), off.numpy())
    ws = moe.split_workspace(DEV)
    for wsp in (None, ws):
        C = poison_(torch.empty((R, N), dtype=torch.bfloat16, device=DEV))
        moe.moe_grouped_gemm_fwd_fp8(a.to(DEV), sa.to(DEV), w.to(DEV), sw.to(DEV), off.to(DEV), C=C, workspace=wsp)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(f64(C), ref)


def test_grouped_gemm_fp8_split_tail_exact():
    """A tile count a few tiles past a full round (131 row tiles x 2 column tiles) and a
    contraction long enough to split (K = 8192: 128 steps of 64): bitwise equal to the unsplit
    product and exact against the oracle on sampled rows (sums up to 16 * 8192 stay exact)."""
    _say("gemm fp8 split tail")
    counts = [4096] * 7 + [4700]
    G, R, K, N = len(counts), sum(counts), 8192, 512
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32, device=DEV)
    g = torch.Generator(device=DEV).manual_seed(4)
    vals = torch.tensor([0x00, 0x38, 0x40, 0x44, 0x48, 0xB8, 0xC0, 0xC4, 0xC8], dtype=torch.uint8, device=DEV)
    a = vals[torch.randint(0, 9, (R, K), generator=g, device=DEV)]      # 0, +-1, +-2, +-3, +-4
    w = vals[torch.randint(0, 9, (G, N, K), generator=g, device=DEV)]
    sa = torch.ones(R, device=DEV)
    sw = torch.ones((G, N), device=DEV)
    ws = moe.split_workspace(DEV)
    c0 = moe.moe_grouped_gemm_fwd_fp8(a, sa, w, sw, off)
    c1 = moe.moe_grouped_gemm_fwd_fp8(a, sa, w, sw, off, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(c0.view(torch.int16), c1.view(torch.int16))
    rng = np.random.default_rng(5)
    rows = np.sort(rng.choice(R, 64, replace=False))
    grp = np.searchsorted(np.concatenate([[0], np.cumsum(counts)]), rows, side="right") - 1
    sub = np.concatenate([[0], np.cumsum(np.bincount(grp, minlength=G))])
    ridx = torch.tensor(rows, device=DEV)
    ref = O.grouped_gemm_fp8(_u8(a[ridx]), np.ones(64, np.float32), _u8(w), np.ones((G, N), np.float32), sub)
    np.testing.assert_array_equal(f64(c1[ridx]), ref)


@pytest.mark.parametrize("K,N", [(1024, 512), (2880, 2880)])
def test_grouped_gemm_fp8_quantized_gaussian(K, N):
    """Quantized bf16 activations and weights (the quantizer on the GPU): the product against the
    oracle on the same codes and scales (fp32 accumulation: Frobenius error <= 1e-3), and the
    deviation from the unquantized bf16 product, which E4M3 rounding bounds, reported."""
    _say("gemm fp8 gaussian", K, N)
    g = torch.Generator().manual_seed(K + N)
    counts = [300, 0, 1000, 77, 513]
    G, R = len(counts), sum(counts)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    x = torch.randn((R, K), generator=g).to(torch.bfloat16)
    wt = (torch.randn((G, N, K), generator=g) * 0.02).to(torch.bfloat16)
    aq, sa = moe.moe_quantize_fp8_rows(x.to(DEV))
    wq, sw = moe.moe_quantize_fp8_rows(wt.to(DEV))
    C = moe.moe_grouped_gemm_fwd_fp8(aq, sa, wq, sw, off.to(DEV), workspace=moe.split_workspace(DEV))
    torch.cuda.synchronize()
    ref = O.grouped_gemm_fp8(_u8(aq), sa.cpu().numpy(), _u8(wq), sw.cpu().numpy(), off.numpy())
    check_float("C fp8", f64(C), ref, 1e-3)
    exact = O.grouped_gemm(f64(x), np.transpose(f64(wt), (0, 2, 1)), off.numpy(), rnd=None)
    err = O.rel_fro(f64(C), exact)
    _say(f"fp8 vs unquantized bf16 product: relative Frobenius {err:.3e}")
    assert err < 0.1


@pytest.mark.parametrize("K,F", [(64, 128), (512, 384), (2048, 1408)])
def test_grouped_gemm_fp8_gate_up(K, F):
    """The gate/up product over the 128-channel-interleaved weight equals the two separate FP8
    products bit for bit (same codes, scales and accumulation order per output), and its SwiGLU
    equals moe_swiglu on those outputs bit for bit; with and without the split tail."""
    _say("gemm fp8 gate/up", K, F)
    g = torch.Generator().manual_seed(K + F)
    G, R = len(GROUPS), sum(GROUPS)
    off = torch.tensor(np.concatenate([[0], np.cumsum(GROUPS)]), dtype=torch.int32, device=DEV)
    x = torch.randn((R, K), generator=g).to(torch.bfloat16).to(DEV)
    wg = (torch.randn((G, F, K), generator=g) * 0.05).to(torch.bfloat16).to(DEV)
    wu = (torch.randn((G, F, K), generator=g) * 0.05).to(torch.bfloat16).to(DEV)
    aq, sa = moe.moe_quantize_fp8_rows(x)
    gq, gs = moe.moe_quantize_fp8_rows(wg)
    uq, us = moe.moe_quantize_fp8_rows(wu)
    iq, is_ = moe.moe_quantize_fp8_rows(moe.interleave_gate_up(wg, wu))
    hg = moe.moe_grouped_gemm_fwd_fp8(aq, sa, gq, gs, off)
    hu = moe.moe_grouped_gemm_fwd_fp8(aq, sa, uq, us, off)
    act = moe.moe_swiglu(hg, hu)
    for ws in (None, moe.split_workspace(DEV)):
        h1, h2, a1 = moe.moe_grouped_gemm_fwd_fp8_gate_up(aq, sa, iq, is_, off, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(h1.view(torch.int16), hg.view(torch.int16))
        assert torch.equal(h2.view(torch.int16), hu.view(torch.int16))
        assert torch.equal(a1.view(torch.int16), act.view(torch.int16))


@pytest.mark.parametrize("cfg_id", [0, 2])
def test_layer_fp8_forward(cfg_id):
    """The layer with its expert forward products in FP8, checked stage by stage on the GPU's own
    intermediate tensors: the per-channel weight codes and the per-row activation codes bit for
    bit, each FP8 product and the SwiGLU against the oracle on the same codes, Y against the
    combine, and the (bf16) backward against the oracle's backward of those forward tensors; the
    deviation of Y from the all-bf16 oracle forward is reported.  Config 2 at 1024 tokens."""
    import dataclasses
    from paper_2606_26453_amd import layer as L, workloads as W
    cfg = W.CONFIGS[cfg_id]
    if cfg_id:
        cfg = dataclasses.replace(cfg, T=1024)
    _say("layer fp8 forward", cfg)
    inp = W.make_inputs(cfg, 0, "cpu")
    lay = L.MoELayer(cfg, {k_: v.to(DEV) for k_, v in inp.items()}, fp8_forward=True)
    lay.step()
    torch.cuda.synchronize()
    b = lay.buf
    wg, wu, wd = (f64(inp[n]) for n in ("w_gate", "w_up", "w_down"))
    gq, gs = O.quantize_rows_fp8(np.transpose(wg, (0, 2, 1)))
    uq, us = O.quantize_rows_fp8(np.transpose(wu, (0, 2, 1)))
    dq, ds = O.quantize_rows_fp8(np.transpose(wd, (0, 2, 1)))
    # the gate/up weight interleaved by 128 channels: per-channel codes are those of each weight
    E, F = gq.shape[0], gq.shape[1]
    lq, ls = _u8(lay.w8["gate_up"][0]).reshape(E, F // 128, 2, 128, -1), lay.w8["gate_up"][1].cpu().numpy()
    np.testing.assert_array_equal(lq[:, :, 0].reshape(E, F, -1), gq)
    np.testing.assert_array_equal(lq[:, :, 1].reshape(E, F, -1), uq)
    np.testing.assert_array_equal(ls.reshape(E, F // 128, 2, 128)[:, :, 0].reshape(E, F), gs)
    np.testing.assert_array_equal(ls.reshape(E, F // 128, 2, 128)[:, :, 1].reshape(E, F), us)
    np.testing.assert_array_equal(_u8(lay.w8["down"][0]), dq)
    np.testing.assert_array_equal(lay.w8["down"][1].cpu().numpy(), ds)
    off = b["offsets"].cpu().numpy()
    xq, xs = O.quantize_rows_fp8(f64(b["x_perm"]))
    np.testing.assert_array_equal(_u8(b["x_q"]), xq)
    np.testing.assert_array_equal(b["x_s"].cpu().numpy(), xs)
    check_float("h_gate", f64(b["h_gate"]), O.grouped_gemm_fp8(xq, xs, gq, gs, off), 2e-3)
    check_float("h_up", f64(b["h_up"]), O.grouped_gemm_fp8(xq, xs, uq, us, off), 2e-3)
    check_float("act", f64(b["act"]), O.swiglu(f64(b["h_gate"]), f64(b["h_up"])), 2e-3)
    aq, as_ = O.quantize_rows_fp8(f64(b["act"]))
    np.testing.assert_array_equal(_u8(b["act_q"]), aq)
    np.testing.assert_array_equal(b["act_s"].cpu().numpy(), as_)
    check_float("y_perm", f64(b["y_perm"]), O.grouped_gemm_fp8(aq, as_, dq, ds, off), 2e-3)
    x = f64(inp["x"])
    shared = None
    if cfg.f_shared:
        shared = tuple(f64(inp[n]) for n in ("w_gate_sh", "w_up_sh", "w_down_sh"))
    ref = O.layer_forward(x, inp["logits"].numpy(), wg, wu, wd, cfg.k, shared=shared)
    fwd = dict(ref)
    for key in ("h_gate", "h_up", "act", "y_perm"):
        fwd[key] = f64(b[key])
    y_sh = ref["shared"]["y"] if shared else None
    check_float("y", f64(b["y"]), O.combine(fwd["y_perm"], ref["topk_w"], ref["row_of_slot"], cfg.k, add=y_sh))
    bwd = O.layer_backward(fwd, x, f64(inp["dy"]), wg, wu, wd, shared=shared)
    for key in ("dh_gate", "dh_up", "dx_perm", "dw_gate", "dw_up", "dw_down", "dx"):
        check_float(key, f64(b[key]), bwd[key])
    _say(f"fp8 forward Y vs the all-bf16 oracle: relative Frobenius {O.rel_fro(f64(b['y']), ref['y']):.3e}")


def test_fp8_forward_fullsize_sampled():
    """The FP8 forward products at the Mixtral-shaped layer's full size (R = 16384 routed rows over
    8 experts, d = 4096, f = 14336), in the launch configuration the benchmark times (split tail
    on): gate/up + SwiGLU over the interleaved weight and the down product, on quantized Gaussian
    operands; 16 sampled rows of the first and of the last expert against the oracle on the same
    codes and scales (the product for those rows alone, the expert's weight decoded once)."""
    from paper_2606_26453_amd import workloads as W
    cfg = W.CONFIGS[1]
    R, d, f, E = cfg.T * cfg.k, cfg.d, cfg.f, cfg.E
    _say("fp8 full size", R, d, f, E)
    g = torch.Generator(device=DEV).manual_seed(11)
    counts = [R // E] * E
    off_np = np.concatenate([[0], np.cumsum(counts)])
    off = torch.tensor(off_np, dtype=torch.int32, device=DEV)
    x = torch.randn((R, d), generator=g, device=DEV).to(torch.bfloat16)
    ws = moe.split_workspace(DEV)
    wg = (torch.randn((E, f, d), generator=g, device=DEV) * 0.02).to(torch.bfloat16)
    wu = (torch.randn((E, f, d), generator=g, device=DEV) * 0.02).to(torch.bfloat16)
    iq, is_ = moe.moe_quantize_fp8_rows(moe.interleave_gate_up(wg, wu))
    del wg, wu
    wd = (torch.randn((E, d, f), generator=g, device=DEV) * 0.02).to(torch.bfloat16)
    dq, ds = moe.moe_quantize_fp8_rows(wd)
    del wd
    xq, xs = moe.moe_quantize_fp8_rows(x)
    hg, hu, act = moe.moe_grouped_gemm_fwd_fp8_gate_up(xq, xs, iq, is_, off, workspace=ws)
    aq, as_ = moe.moe_quantize_fp8_rows(act)
    y = moe.moe_grouped_gemm_fwd_fp8(aq, as_, dq, ds, off, workspace=ws)
    torch.cuda.synchronize()
    rng = np.random.default_rng(12)
    for e in (0, E - 1):
        rows = np.sort(rng.choice(np.arange(off_np[e], off_np[e + 1]), 16, replace=False))
        ridx = torch.tensor(rows, device=DEV)
        sub = np.array([0, 16])
        il = _u8(iq[e]).reshape(f // 128, 2, 128, d)
        ils = is_[e].cpu().numpy().reshape(f // 128, 2, 128)
        gq, uq = il[:, 0].reshape(1, f, d), il[:, 1].reshape(1, f, d)
        gs, us = ils[:, 0].reshape(1, f), ils[:, 1].reshape(1, f)
        a_c, a_s = _u8(xq[ridx]), xs[ridx].cpu().numpy()
        check_float(f"h_gate e{e}", f64(hg[ridx]), O.grouped_gemm_fp8(a_c, a_s, gq, gs, sub), 2e-3)
        check_float(f"h_up e{e}", f64(hu[ridx]), O.grouped_gemm_fp8(a_c, a_s, uq, us, sub), 2e-3)
        check_float(f"act e{e}", f64(act[ridx]), O.swiglu(f64(hg[ridx]), f64(hu[ridx])), 2e-3)
        rq, rs = O.quantize_rows_fp8(f64(act[ridx]))
        np.testing.assert_array_equal(_u8(aq[ridx]), rq)
        np.testing.assert_array_equal(as_[ridx].cpu().numpy(), rs)
        check_float(f"y e{e}", f64(y[ridx]), O.grouped_gemm_fp8(rq, rs, _u8(dq[e])[None], ds[e].cpu().numpy()[None], sub),
                    2e-3)


def test_grouped_gemm_fp8_256_groups_exact():
    """The maximum group count (G = 256, empty groups included, more row tiles than CUs): the FP8
    product and the FP8 gate/up product exact against the oracle on integer codes."""
    _say("gemm fp8 256 groups")
    rng = np.random.default_rng(2560)
    counts = rng.integers(0, 400, 256)
    counts[rng.choice(256, 20, replace=False)] = 0
    G, R, K, N = 256, int(counts.sum()), 128, 256
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    g = torch.Generator().manual_seed(2560)
    a, w, w2 = _int_codes(g, (R, K)), _int_codes(g, (G, N, K)), _int_codes(g, (G, N, K))
    sa, sw, sw2 = _pow2(g, (R,)), _pow2(g, (G, N)), _pow2(g, (G, N))
    ws = moe.split_workspace(DEV)
    C = moe.moe_grouped_gemm_fwd_fp8(a.to(DEV), sa.to(DEV), w.to(DEV), sw.to(DEV), off.to(DEV), workspace=ws)
    iq = moe.interleave_gate_up(w.to(DEV), w2.to(DEV))
    iscale = moe.interleave_gate_up(sw.to(DEV)[..., None], sw2.to(DEV)[..., None])[..., 0]
    hg, hu, act = moe.moe_grouped_gemm_fwd_fp8_gate_up(a.to(DEV), sa.to(DEV), iq, iscale.contiguous(), off.to(DEV),
                                                        workspace=ws)
    torch.cuda.synchronize()
    ref = O.grouped_gemm_fp8(_u8(a), sa.numpy(), _u8(w), sw.numpy(), off.numpy())
    np.testing.assert_array_equal(f64(C), ref)
    np.testing.assert_array_equal(f64(hg), ref)
    np.testing.assert_array_equal(f64(hu), O.grouped_gemm_fp8(_u8(a), sa.numpy(), _u8(w2), sw2.numpy(), off.numpy()))
    check_float("act", f64(act), O.swiglu(f64(hg), f64(hu)), 1e-2)


# ------------------------------------------------------------------------------------------------
# The backward's data-gradient products on E4M3 operands
# ------------------------------------------------------------------------------------------------
def _dequant(codes, scale):
    """bf16 tensor of decode(codes) * scale (exact for small-integer codes and power-of-two scales)."""
    return torch.from_numpy(O.e4m3_decode(_u8(codes)) * scale.double().numpy()[..., None]).to(torch.bfloat16)


@pytest.mark.parametrize("M,K", [(1, 16), (7, 64), (300, 4112), (33, 14336)])
def test_quantize_fp8_rows2(M, K):
    """Joint per-row quantization of [x | x2]: codes and scales bit for bit against the oracle's row
    quantizer on the concatenated rows and against moe_quantize_fp8_rows on the concatenation;
    rows whose maximum sits in either half, an all-zero row and rows with one all-zero half."""
    _say("quantize fp8 rows2", M, K)
    g = torch.Generator().manual_seed(3 * M + K)
    mk = lambda: (torch.randn((M, K), generator=g) * torch.exp(torch.randn((M, 1), generator=g) * 3)).to(torch.bfloat16)
    x, x2 = mk(), mk()
    if M > 3:
        x[1] = 0
        x2[1] = 0
        x[2] = 0
        x2[3] = 0
    q = poison_(torch.empty((M, 2 * K), dtype=torch.uint8, device=DEV))
    s = poison_(torch.empty(M, dtype=torch.float32, device=DEV))
    moe.moe_quantize_fp8_rows2(x.to(DEV), x2.to(DEV), q, s)
    torch.cuda.synchronize()
    cat = torch.cat([x, x2], dim=1)
    rq, rs = O.quantize_rows_fp8(f64(cat))
    np.testing.assert_array_equal(_u8(q), rq)
    np.testing.assert_array_equal(s.cpu().numpy(), rs)
    q1, s1 = moe.moe_quantize_fp8_rows(cat.contiguous().to(DEV))
    torch.cuda.synchronize()
    assert torch.equal(q1, q) and torch.equal(s1, s)


@pytest.mark.parametrize("K,N", [(64, 128), (256, 320), (512, 576)])
def test_dx_swiglu_bwd_fp8_exact(K, N):
    """The FP8 dX-down product with the SwiGLU backward in its epilogue, on small-integer codes with
    power-of-two scales (every sum exact in fp32): bitwise equal to the bf16 product with the same
    epilogue (moe_grouped_gemm_dx_swiglu_bwd) on the decoded operands, with and without the split
    tail, over ragged and empty groups; and against the oracle's SwiGLU backward of the oracle's
    FP8 product."""
    _say("dx swiglu bwd fp8 exact", K, N)
    g = torch.Generator().manual_seed(K + 7 * N)
    G, R = len(GROUPS), sum(GROUPS)
    off = torch.tensor(np.concatenate([[0], np.cumsum(GROUPS)]), dtype=torch.int32)
    a, w = _int_codes(g, (R, K)), _int_codes(g, (G, N, K))
    sa, sw = _pow2(g, (R,)), _pow2(g, (G, N))
    hg = torch.randn((R, N), generator=g).to(torch.bfloat16)
    hu = torch.randn((R, N), generator=g).to(torch.bfloat16)
    D = lambda t: t.to(DEV)
    rg, ru = moe.moe_grouped_gemm_dx_swiglu_bwd(D(_dequant(a, sa)), D(_dequant(w, sw)), D(off), D(hg), D(hu))
    ws = moe.split_workspace(DEV)
    da = O.grouped_gemm_fp8(_u8(a), sa.numpy(), _u8(w), sw.numpy(), off.numpy())
    og, ou = O.swiglu_bwd(f64(hg), f64(hu), da)
    for wsp in (None, ws):
        dg = poison_(torch.empty((R, N), dtype=torch.bfloat16, device=DEV))
        du = poison_(torch.empty((R, N), dtype=torch.bfloat16, device=DEV))
        moe.moe_grouped_gemm_dx_swiglu_bwd_fp8(D(a), D(sa), D(w), D(sw), D(off), D(hg), D(hu), dg, du, workspace=wsp)
        torch.cuda.synchronize()
        assert torch.equal(dg.view(torch.int16), rg.view(torch.int16))
        assert torch.equal(du.view(torch.int16), ru.view(torch.int16))
        check_float("dh_gate", f64(dg), og, 2e-3)
        check_float("dh_up", f64(du), ou, 2e-3)


@pytest.mark.parametrize("F,N", [(64, 64), (192, 320), (704, 256)])
def test_dx_gate_up_fp8_joint_exact(F, N):
    """The gate/up data gradient as one FP8 product over the joined contraction [dH_g | dH_u] x
    [W_g | W_u] (moe_grouped_gemm_fwd_fp8 with K = 2F): on small-integer codes with one power-of-two
    scale per joined row and per output channel, bitwise equal to the bf16 dual product
    moe_grouped_gemm_dx on the decoded halves (with and without the split tail) and exact against
    the oracle's FP8 product."""
    _say("dx gate/up fp8 joint", F, N)
    g = torch.Generator().manual_seed(F + 3 * N)
    G, R = len(GROUPS), sum(GROUPS)
    off = torch.tensor(np.concatenate([[0], np.cumsum(GROUPS)]), dtype=torch.int32)
    a, w = _int_codes(g, (R, 2 * F)), _int_codes(g, (G, N, 2 * F))
    sa, sw = _pow2(g, (R,)), _pow2(g, (G, N))
    ad, wd = _dequant(a, sa), _dequant(w, sw)
    D = lambda t: t.contiguous().to(DEV)
    ref = moe.moe_grouped_gemm_dx(D(ad[:, :F]), D(wd[:, :, :F]), D(off), D(ad[:, F:]), D(wd[:, :, F:]))
    ws = moe.split_workspace(DEV)
    oref = O.grouped_gemm_fp8(_u8(a), sa.numpy(), _u8(w), sw.numpy(), off.numpy())
    for wsp in (None, ws):
        C = poison_(torch.empty((R, N), dtype=torch.bfloat16, device=DEV))
        moe.moe_grouped_gemm_fwd_fp8(D(a), D(sa), D(w), D(sw), D(off), C=C, workspace=wsp)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int16), ref.view(torch.int16))
        np.testing.assert_array_equal(f64(C), oref)


@pytest.mark.parametrize("cfg_id", [0, 2])
def test_layer_fp8_backward(cfg_id):
    """The layer with its expert data-gradient products in FP8 (forward in bf16), stage by stage on
    the GPU's own intermediate tensors: the weight codes (down per stored row, [W_gate | W_up] per
    joined row) and the dY_perm and [dH_gate | dH_up] codes bit for bit, dH against the oracle's
    SwiGLU backward of its FP8 product on the same codes, dX_perm against the oracle's FP8 product,
    dX against the unpermute-sum and the bf16 weight gradients against the oracle on the GPU's dY_perm
    and dH.  Two steps, so the second re-quantizes the weights.  Config 2 at 1024 tokens."""
    import dataclasses
    from paper_2606_26453_amd import layer as L, workloads as W
    cfg = W.CONFIGS[cfg_id]
    if cfg_id:
        cfg = dataclasses.replace(cfg, T=1024)
    _say("layer fp8 backward", cfg)
    inp = W.make_inputs(cfg, 0, "cpu")
    lay = L.MoELayer(cfg, {k_: v.to(DEV) for k_, v in inp.items()}, fp8_backward=True)
    lay.step()
    lay.step()
    torch.cuda.synchronize()
    b = lay.buf
    wg, wu, wd = (f64(inp[n]) for n in ("w_gate", "w_up", "w_down"))
    dq, ds = O.quantize_rows_fp8(wd)
    np.testing.assert_array_equal(_u8(lay.w8b["down"][0]), dq)
    np.testing.assert_array_equal(lay.w8b["down"][1].cpu().numpy(), ds)
    gq, gs = O.quantize_rows_fp8(np.concatenate([wg, wu], axis=2))
    np.testing.assert_array_equal(_u8(lay.w8b["gate_up"][0]), gq)
    np.testing.assert_array_equal(lay.w8b["gate_up"][1].cpu().numpy(), gs)
    off = b["offsets"].cpu().numpy()
    yq, ys = O.quantize_rows_fp8(f64(b["dy_perm"]))
    np.testing.assert_array_equal(_u8(b["dy_q"]), yq)
    np.testing.assert_array_equal(b["dy_s"].cpu().numpy(), ys)
    og, ou = O.swiglu_bwd(f64(b["h_gate"]), f64(b["h_up"]), O.grouped_gemm_fp8(yq, ys, dq, ds, off))
    check_float("dh_gate", f64(b["dh_gate"]), og, 4e-3)
    check_float("dh_up", f64(b["dh_up"]), ou, 4e-3)
    hq, hs = O.quantize_rows_fp8(np.concatenate([f64(b["dh_gate"]), f64(b["dh_up"])], axis=1))
    np.testing.assert_array_equal(_u8(b["dh_q"]), hq)
    np.testing.assert_array_equal(b["dh_s"].cpu().numpy(), hs)
    check_float("dx_perm", f64(b["dx_perm"]), O.grouped_gemm_fp8(hq, hs, gq, gs, off), 2e-3)
    ros = b["row_of_slot"].cpu().numpy()
    add = None
    if cfg.f_shared:
        add = f64(b["dx_sh"])
    check_float("dx", f64(b["dx"]), O.combine(f64(b["dx_perm"]), None, ros, cfg.k, add=add), 2e-3)
    check_float("dw_down", f64(b["dw_down"]), O.grouped_gemm_dw(f64(b["act"]), f64(b["dy_perm"]), off), 1e-4)
    check_float("dw_gate", f64(b["dw_gate"]), O.grouped_gemm_dw(f64(b["x_perm"]), f64(b["dh_gate"]), off), 1e-4)
    check_float("dw_up", f64(b["dw_up"]), O.grouped_gemm_dw(f64(b["x_perm"]), f64(b["dh_up"]), off), 1e-4)
    # how far the FP8 data gradient moves dX from the all-bf16 layer's
    x = f64(inp["x"])
    shared = None
    if cfg.f_shared:
        shared = tuple(f64(inp[n]) for n in ("w_gate_sh", "w_up_sh", "w_down_sh"))
    fwd = O.layer_forward(x, inp["logits"].numpy(), wg, wu, wd, cfg.k, shared=shared)
    bwd = O.layer_backward(fwd, x, f64(inp["dy"]), wg, wu, wd, shared=shared)
    _say(f"fp8 data gradient dX vs the all-bf16 oracle: relative Frobenius {O.rel_fro(f64(b['dx']), bwd['dx']):.3e}")


def _oracle_layer_fp8(inp, cfg):
    """The layer's forward and backward with the four expert data products on E4M3 operands with
    fp32 scales (X_perm, the SwiGLU output, dY_perm and [dH_gate | dH_up] per row; the forward
    weights per output channel, the data-gradient weights per row of their stored layouts), every
    quantization applied by the oracle to its own bf16 intermediates; the rest as the bf16 oracle."""
    x = f64(inp["x"])
    wg, wu, wd = (f64(inp[n]) for n in ("w_gate", "w_up", "w_down"))
    shared = None
    if cfg.f_shared:
        shared = tuple(f64(inp[n]) for n in ("w_gate_sh", "w_up_sh", "w_down_sh"))
    k = cfg.k
    q = O.quantize_rows_fp8
    idx, tw = O.route_topk(inp["logits"].numpy(), k)
    off, ros, tor = O.permute(idx, cfg.E)
    xp = O.gather(x, tor)
    xq, xs = q(xp)
    gq, gs = q(np.transpose(wg, (0, 2, 1)))
    uq, us = q(np.transpose(wu, (0, 2, 1)))
    dq, ds = q(np.transpose(wd, (0, 2, 1)))
    hg = O.grouped_gemm_fp8(xq, xs, gq, gs, off)
    hu = O.grouped_gemm_fp8(xq, xs, uq, us, off)
    act = O.swiglu(hg, hu)
    aq, as_ = q(act)
    y_perm = O.grouped_gemm_fp8(aq, as_, dq, ds, off)
    y_sh = dx_sh = None
    dy = f64(inp["dy"])
    if shared is not None:
        sf = O.dense_ffn_forward(x, *shared)
        y_sh = sf["y"]
        dx_sh = O.dense_ffn_backward(sf, x, dy, *shared)["dx"]
    y = O.combine(y_perm, tw, ros, k, add=y_sh)
    dy_perm, _ = O.combine_bwd(dy, tw, ros, y_perm, k)
    yq, ys = q(dy_perm)
    rq, rs = q(wd)
    dhg, dhu = O.swiglu_bwd(hg, hu, O.grouped_gemm_fp8(yq, ys, rq, rs, off))
    hq, hs = q(np.concatenate([dhg, dhu], axis=1))
    jq, js = q(np.concatenate([wg, wu], axis=2))
    dx_perm = O.grouped_gemm_fp8(hq, hs, jq, js, off)
    dx = O.combine(dx_perm, None, ros, k, add=dx_sh)
    return {"y": y, "y_perm": y_perm, "h_gate": hg, "h_up": hu, "act": act, "dy_perm": dy_perm,
            "dh_gate": dhg, "dh_up": dhu, "dx_perm": dx_perm, "dx": dx,
            "dw_down": O.grouped_gemm_dw(act, dy_perm, off), "dw_gate": O.grouped_gemm_dw(xp, dhg, off),
            "dw_up": O.grouped_gemm_dw(xp, dhu, off)}


@pytest.mark.parametrize("cfg_id", [0, 2])
def test_layer_fp8_end_to_end(cfg_id):
    """The layer with FP8 (fp32-scale) forward and data-gradient products, two steps, against an
    end-to-end oracle run that quantizes its own bf16 intermediates (no GPU tensor enters the
    oracle): every output and gradient within 1e-2 (a code may differ where the two sides' bf16
    intermediates differ in the last bit).  Config 2 at 1024 tokens."""
    import dataclasses
    from paper_2606_26453_amd import layer as L, workloads as W
    cfg = W.CONFIGS[cfg_id]
    if cfg_id:
        cfg = dataclasses.replace(cfg, T=1024)
    _say("layer fp8 end to end", cfg)
    inp = W.make_inputs(cfg, 0, "cpu")
    lay = L.MoELayer(cfg, {k_: v.to(DEV) for k_, v in inp.items()}, fp8_forward=True, fp8_backward=True)
    lay.step()
    lay.step()
    torch.cuda.synchronize()
    ref = _oracle_layer_fp8(inp, cfg)
    for key in ("h_gate", "h_up", "act", "y_perm", "y", "dy_perm", "dh_gate", "dh_up", "dx_perm", "dx",
                "dw_down", "dw_gate", "dw_up"):
        check_float(key, f64(lay.buf[key]), ref[key], 1e-2)
