"""GPU parity of the router: logits, the routing decision at near ties, the backward through the
routing weights with the load-balancing loss, dWr and the router's share of dX, all through the
C ABI and against the CPU oracle."""
import sys

import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2606_26453_amd import moe
from tests.gpu_util import check_float, f64, gpu_available, i64, poison_

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]
DEV = "cuda:0"


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _inputs(T, d, E, seed, bias=True):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((T, d), generator=g).to(torch.bfloat16)
    wr = torch.randn((d, E), generator=g) * 0.02
    b = torch.randn(E, generator=g) if bias else None
    return x, wr, b


# logits: fp32 sums of d products against the exact sum; bound |err| <= 2^-22 * d * sum|x_i wr_i|
@pytest.mark.parametrize("T,d,E", [(1, 64, 1), (130, 256, 4), (1000, 512, 8), (333, 128, 16), (257, 192, 40),
                                   (200, 1024, 64), (64, 64, 256), (2000, 4096, 8), (37, 2880, 9),
                                   (100, 4160, 8)])
def test_router_logits(T, d, E):
    _say("router logits", T, d, E)
    x, wr, b = _inputs(T, d, E, T + d + E)
    out = poison_(torch.empty((T, E), dtype=torch.float32, device=DEV))
    moe.moe_router_logits(x.to(DEV), wr.to(DEV), b.to(DEV), logits=out)
    torch.cuda.synchronize()
    ref = O.router_logits(f64(x), f64(wr), f64(b))
    bound = 2.0 ** -22 * d * (np.abs(f64(x)) @ np.abs(f64(wr))) + 1e-7 * np.abs(f64(b))
    err = np.abs(f64(out) - ref)
    assert np.isfinite(f64(out)).all() and (err <= bound).all(), float((err / bound).max())
    out2 = moe.moe_router_logits(x.to(DEV), wr.to(DEV), b.to(DEV))
    torch.cuda.synchronize()
    assert torch.equal(out, out2)                      # deterministic
    out3 = moe.moe_router_logits(x.to(DEV), wr.to(DEV))  # no bias
    torch.cuda.synchronize()
    assert (np.abs(f64(out3) - O.router_logits(f64(x), f64(wr))) <= bound).all()


def test_routing_decision_near_ties():
    """The decision on the GPU's logits equals the oracle's decision on those same logits bit for
    bit; against the oracle's exact logits it may differ only for tokens whose exact k-th and
    (k+1)-th logits are within twice the logit error bound (the near-tie policy)."""
    T, d, E, k = 4096, 512, 16, 2
    x, wr, b = _inputs(T, d, E, 11, bias=False)
    logits = moe.moe_router_logits(x.to(DEV), wr.to(DEV))
    r = moe.moe_route_permute(logits, None, k)
    torch.cuda.synchronize()
    idx_gpu = i64(r["topk_idx"])
    idx_same, _ = O.route_topk(f64(logits), k)
    np.testing.assert_array_equal(idx_gpu, idx_same)
    exact = O.router_logits(f64(x), f64(wr))
    idx_exact, _ = O.route_topk(exact, k)
    srt = -np.sort(-exact, axis=1)
    gap = srt[:, k - 1] - srt[:, k]
    bound = (2.0 ** -22 * d * (np.abs(f64(x)) @ np.abs(f64(wr)))).max(axis=1)
    differ = (idx_gpu != idx_exact).any(axis=1)
    assert (gap[differ] <= 2 * bound[differ]).all()
    _say("tokens whose decision differs from the exact logits':", int(differ.sum()), "of", T)


@pytest.mark.parametrize("normalize,alpha", [(True, 0.0), (True, 0.01), (False, 0.0), (False, 0.02)])
@pytest.mark.parametrize("T,d,E,k", [(300, 256, 8, 2), (257, 128, 64, 6), (64, 192, 40, 3), (513, 320, 16, 4),
                                     (700, 4160, 8, 2)])
def test_router_bwd(T, d, E, k, normalize, alpha):
    _say("router bwd", T, d, E, k, normalize, alpha)
    x, wr, b = _inputs(T, d, E, 7 * T + E)
    xd, wrd = x.to(DEV), wr.to(DEV)
    logits = moe.moe_router_logits(xd, wrd, b.to(DEV))
    r = moe.moe_route_permute(logits, None, k, normalize_topk=normalize)
    g = torch.Generator().manual_seed(3)
    d_w = torch.randn((T, k), generator=g).to(DEV)
    dx0 = torch.randn((T, d), generator=g).to(torch.bfloat16)
    dx = dx0.to(DEV).clone()
    dl = poison_(torch.empty((T, E), dtype=torch.float32, device=DEV))
    dwr = poison_(torch.empty((d, E), dtype=torch.float32, device=DEV))
    moe.moe_router_bwd(xd, wrd, logits, r["topk_idx"], r["topk_w"], d_w, r["offsets"], normalize, alpha,
                       dx=dx, dlogits=dl, dwr=dwr)
    torch.cuda.synchronize()
    L = f64(logits)
    idx = i64(r["topk_idx"])
    ref_dl = O.route_topk_bwd(L, idx, f64(d_w), normalize)
    if alpha:
        counts = np.diff(i64(r["offsets"]))
        ref_dl = ref_dl + O.aux_loss(L, counts, k, alpha)[1]
    check_float("dlogits", f64(dl), ref_dl, 1e-5)
    ref_dwr, ref_dx = O.router_bwd(f64(x), f64(wr), f64(dl), dx=f64(dx0))
    check_float("dwr", f64(dwr), ref_dwr, 1e-5)
    check_float("dx", f64(dx), ref_dx, 1e-3)
    # the router's share of dX at bf16 resolution: at most one bf16 step apart from the oracle
    ulp = np.maximum(np.abs(ref_dx), 2.0 ** -126) * 2.0 ** -7
    assert (np.abs(f64(dx) - ref_dx) <= ulp * 1.01).all()


@pytest.mark.parametrize("T,E,k", [(1000, 32, 4), (1000, 8, 2), (4099, 13, 3), (1, 4, 1)])
def test_router_aux_loss(T, E, k):
    alpha = 0.01
    g = torch.Generator().manual_seed(5)
    logits = (torch.randn((T, E), generator=g) * 2).to(DEV)
    r = moe.moe_route_permute(logits, None, k)
    loss = moe.moe_router_aux_loss(logits, r["offsets"], k, alpha)
    torch.cuda.synchronize()
    ref, _ = O.aux_loss(f64(logits), np.diff(i64(r["offsets"])), k, alpha)
    assert abs(loss.item() - ref) <= 1e-5 * abs(ref)
    # uniform logits: loss = alpha exactly in the closed form, to fp32 rounding here
    z = torch.zeros((T, E), device=DEV)
    lz = moe.moe_router_aux_loss(z, r["offsets"], k, alpha)
    torch.cuda.synchronize()
    assert abs(lz.item() - alpha) <= 1e-6


@pytest.mark.parametrize("T,d,E,k,with_add", [(1, 64, 1, 1, False), (37, 192, 5, 2, True), (300, 256, 8, 2, False),
                                               (129, 2048, 13, 3, True), (64, 4096, 16, 4, False),
                                               (50, 512, 8, 6, True), (40, 128, 16, 8, False),
                                               (1000, 4096, 8, 2, True)])
def test_unpermute_router_dx(T, d, E, k, with_add):
    """The unpermute-sum of dX fused with the router's share: bitwise equal to moe_unpermute_combine
    followed by moe_router_bwd's in-place update of dx (same dlogits), and within one bf16 step of
    the oracle's composition of the two (each rounded to bf16)."""
    _say("unpermute + router dx", T, d, E, k, with_add)
    x, wr, _ = _inputs(T, d, E, 3 * T + d + E, bias=False)
    xd, wrd = x.to(DEV), wr.to(DEV)
    logits = moe.moe_router_logits(xd, wrd)
    r = moe.moe_route_permute(logits, None, k)
    g = torch.Generator().manual_seed(T + k)
    d_w = torch.randn((T, k), generator=g).to(DEV)
    dx_perm = torch.randn((T * k, d), generator=g).to(torch.bfloat16)
    add = torch.randn((T, d), generator=g).to(torch.bfloat16) if with_add else None
    addd = add.to(DEV) if with_add else None
    two = moe.moe_unpermute_combine(dx_perm.to(DEV), None, r["row_of_slot"], k, add=addd)
    dl, _ = moe.moe_router_bwd(xd, wrd, logits, r["topk_idx"], r["topk_w"], d_w, r["offsets"], dx=two)
    fused = poison_(torch.empty((T, d), dtype=torch.bfloat16, device=DEV))
    moe.moe_unpermute_router_dx(dx_perm.to(DEV), r["row_of_slot"], k, dl, wrd, add=addd, dx=fused)
    torch.cuda.synchronize()
    assert torch.equal(fused.view(torch.int16), two.view(torch.int16))
    base = O.combine(f64(dx_perm), None, i64(r["row_of_slot"]), k, add=None if add is None else f64(add))
    _, ref = O.router_bwd(f64(x), f64(wr), f64(dl), dx=base)
    ulp = np.maximum(np.abs(ref), 2.0 ** -126) * 2.0 ** -7
    assert (np.abs(f64(fused) - ref) <= ulp * 1.01).all()


def test_unpermute_router_dx_refuses_unsupported_sizes():
    z = torch.zeros((4, 64), dtype=torch.bfloat16, device=DEV)
    ros = torch.arange(4, dtype=torch.int32, device=DEV)
    with pytest.raises(RuntimeError, match="E <= 16"):
        moe.moe_unpermute_router_dx(z, ros, 1, torch.zeros((4, 17), device=DEV), torch.zeros((64, 17), device=DEV))


@pytest.mark.parametrize("cfg_id", [0, 2])
def test_layer_with_router(cfg_id):
    """The whole layer with the router on the GPU (logits, load-balancing loss, router backward):
    the oracle routes the GPU's logits (the decision is compared bit for bit on the same logits;
    the logits themselves against the exact ones), then every output of the layer, the loss, dWr
    and the token gradient including the router's share are compared with the oracle's.  Config 2
    is run at a reduced token count (its shapes otherwise) to keep the oracle quick."""
    import dataclasses
    from paper_2606_26453_amd import layer as L, workloads as W
    cfg = W.CONFIGS[cfg_id]
    if cfg_id == 2:
        cfg = dataclasses.replace(cfg, T=128)
    alpha = 0.01
    inp = W.make_inputs(cfg, 0, "cpu")
    dinp = {k_: v.to(DEV) for k_, v in inp.items()}
    lay = L.MoELayer(cfg, dinp, router=True, aux_alpha=alpha)
    lay.step()
    torch.cuda.synchronize()
    b = lay.buf
    x, wr = f64(inp["x"]), f64(inp["wr"])
    bias = f64(inp["router_bias"]) if "router_bias" in inp else None
    exact = O.router_logits(x, wr, bias)
    bound = 2.0 ** -22 * cfg.d * (np.abs(x) @ np.abs(wr)) + (1e-7 * np.abs(bias) if bias is not None else 0)
    assert (np.abs(f64(b["logits"]) - exact) <= bound).all()
    logits = f64(b["logits"])
    shared = None
    if cfg.f_shared:
        shared = tuple(f64(inp[n]) for n in ("w_gate_sh", "w_up_sh", "w_down_sh"))
    fwd = O.layer_forward(x, logits, f64(inp["w_gate"]), f64(inp["w_up"]), f64(inp["w_down"]), cfg.k, shared=shared)
    np.testing.assert_array_equal(i64(b["topk_idx"]), fwd["topk_idx"])
    np.testing.assert_array_equal(i64(b["offsets"]), fwd["offsets"])
    check_float("y", f64(b["y"]), fwd["y"])
    bwd = O.layer_backward(fwd, x, f64(inp["dy"]), f64(inp["w_gate"]), f64(inp["w_up"]), f64(inp["w_down"]),
                           shared=shared)
    counts = np.diff(fwd["offsets"])
    loss, g_aux = O.aux_loss(logits, counts, cfg.k, alpha)
    assert abs(b["aux_loss"].item() - loss) <= 1e-5 * abs(loss)
    dl = O.route_topk_bwd(logits, fwd["topk_idx"], bwd["d_topk_w"]) + g_aux
    check_float("dlogits", f64(b["dlogits"]), dl)
    dwr, dx = O.router_bwd(x, wr, dl, dx=bwd["dx"])
    check_float("dwr", f64(b["dwr"]), dwr)
    check_float("dx (experts + router)", f64(b["dx"]), dx)
    for key in ("dw_gate", "dw_up", "dw_down"):
        check_float(key, f64(b[key]), bwd[key])
