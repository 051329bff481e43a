"""Pins of the CPU oracle against things other than itself: hand-evaluated examples of the
paper's definition, library routines (torch/scipy), brute force, closed forms, invariants,
automatic differentiation and finite differences.  CPU only."""
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import moe_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return json.load(fh)


# ---------------------------------------------------------------------------------------------
# bf16 rounding
# ---------------------------------------------------------------------------------------------
def _torch_bf16(x32):
    return torch.from_numpy(x32).to(torch.bfloat16).to(torch.float32).numpy().astype(np.float64)


def test_bf16_round_matches_torch_random():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(200_000) * np.exp2(rng.integers(-140, 120, 200_000))).astype(np.float32)
    np.testing.assert_array_equal(O.bf16_round(x.astype(np.float64)), _torch_bf16(x))


def test_bf16_round_ties_and_edges():
    # exact midpoints between neighbouring bf16 values, both parities, both signs, subnormals
    base = np.array([1.0, 1.0 + 2**-7, 3.0, 1.5, 2.0**-126, 2.0**-130, 2.0**100], dtype=np.float64)
    ulp = np.array([2**-7, 2**-7, 2**-6, 2**-7, 2**-133, 2**-133, 2.0**93])
    mids = np.concatenate([base + ulp / 2, -(base + ulp / 2), base + ulp / 2 + ulp / 64])
    x32 = mids.astype(np.float32)
    assert np.array_equal(x32.astype(np.float64), mids)       # exact in fp32, so torch sees them
    np.testing.assert_array_equal(O.bf16_round(mids), _torch_bf16(x32))
    # closed forms: 1 + 2^-8 is a tie -> even neighbour 1.0; 1 + 3*2^-8 -> 1 + 2^-6
    assert O.bf16_round(1 + 2**-8) == 1.0
    assert O.bf16_round(1 + 3 * 2**-8) == 1 + 2**-6
    assert O.bf16_round(1 + 2**-8 + 2**-30) == 1 + 2**-7
    assert math.copysign(1.0, O.bf16_round(-0.0)) == -1.0
    assert O.bf16_round(3.5e38) == np.inf and O.bf16_round(-3.5e38) == -np.inf
    assert O.bf16_round(O.BF16_MAX) == O.BF16_MAX


def test_bf16_bits_roundtrip():
    rng = np.random.default_rng(2)
    bits = rng.integers(0, 2**16, 5000, dtype=np.uint16)
    bits = bits[(bits & 0x7F80) != 0x7F80]      # drop inf/nan patterns
    vals = O.bf16_bits_to_f64(bits)
    np.testing.assert_array_equal(O.f64_to_bf16_bits(vals), bits)
    t = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).float().numpy()
    np.testing.assert_array_equal(vals, t.astype(np.float64))


# ---------------------------------------------------------------------------------------------
# routing
# ---------------------------------------------------------------------------------------------
def test_route_permute_worked_example():
    g = _load("route_permute_worked_example.json")
    idx, w = O.route_topk(np.array(g["logits"], dtype=np.float32), g["k"])
    np.testing.assert_array_equal(idx, g["topk_idx"])
    np.testing.assert_allclose(w, g["topk_w"], rtol=1e-15, atol=0)
    off, ros, tor = O.permute(idx, 4)
    np.testing.assert_array_equal(off, g["offsets"])
    np.testing.assert_array_equal(ros, g["row_of_slot"])
    np.testing.assert_array_equal(tor, g["token_of_row"])


@pytest.mark.parametrize("E,k", [(4, 1), (4, 2), (8, 3), (16, 16), (33, 5)])
def test_route_brute_force_with_ties(E, k):
    rng = np.random.default_rng(E * 100 + k)
    T = 60
    L = rng.integers(-3, 4, (T, E)).astype(np.float32)     # many exact ties
    L[::7] = 0.0
    L[1::11, 0] = -0.0                                      # -0 ties +0
    idx, w = O.route_topk(L, k)
    for t in range(T):
        brute = sorted(range(E), key=lambda e: (-float(L[t, e]), e))[:k]
        assert list(idx[t]) == brute
    # softmax over the selected logits: weights sum to one, ratios follow exp of logit gaps,
    # and equal logits share equal weight
    np.testing.assert_allclose(w.sum(1), 1.0, rtol=1e-14)
    sel = np.take_along_axis(L.astype(np.float64), idx, 1)
    np.testing.assert_allclose(w[:, 1:] / w[:, :1], np.exp(sel[:, 1:] - sel[:, :1]), rtol=1e-13)


def test_route_weights_library_softmax():
    from scipy.special import softmax
    rng = np.random.default_rng(3)
    L = rng.standard_normal((50, 12)).astype(np.float32)
    # k = E: the selected-k softmax is the full softmax, in descending-logit order
    idx, w = O.route_topk(L, 12)
    full = softmax(L.astype(np.float64), axis=1)
    np.testing.assert_allclose(w, np.take_along_axis(full, idx, 1), rtol=1e-13)
    # normalize=False: the full-softmax probability of each selected expert
    idx3, w3 = O.route_topk(L, 3, normalize=False)
    np.testing.assert_allclose(w3, np.take_along_axis(full, idx3, 1), rtol=1e-13)
    # k = 1: weight exactly 1
    _, w1 = O.route_topk(L, 1)
    assert np.all(w1 == 1.0)


# ---------------------------------------------------------------------------------------------
# permutation
# ---------------------------------------------------------------------------------------------
def _check_permutation(idx, E, off, ros, tor):
    T, k = idx.shape
    R = T * k
    counts = np.diff(off)
    assert off[0] == 0 and off[-1] == R and np.all(counts >= 0)
    assert np.array_equal(np.sort(ros), np.arange(R))                     # bijection
    assert np.array_equal(tor[ros], np.arange(R) // k)                    # slot -> its token
    for e in range(E):
        rows = np.arange(off[e], off[e + 1])
        slots = np.argsort(ros)[rows]
        assert np.all(idx.reshape(-1)[slots] == e)                      # row in its expert's group
        assert np.all(np.diff(tor[rows]) > 0)                            # ascending tokens
        assert counts[e] == int((idx == e).sum())                        # count conservation


@pytest.mark.parametrize("T,E,k", [(1, 1, 1), (5, 4, 4), (64, 8, 2), (300, 64, 6), (97, 256, 8)])
def test_permute_invariants(T, E, k):
    rng = np.random.default_rng(T + E + k)
    L = rng.standard_normal((T, E)).astype(np.float32)
    L[:, : E // 3] -= 1e4 if E > 3 else 0.0      # some experts never chosen (empty groups)
    idx, _ = O.route_topk(L, k)
    off, ros, tor = O.permute(idx, E)
    _check_permutation(idx, E, off, ros, tor)


def test_gather_combine_round_trip():
    rng = np.random.default_rng(4)
    T, d, E = 40, 16, 6
    X = rng.integers(-8, 9, (T, d)).astype(np.float64)
    for k in (1, 2, 3):
        idx, _ = O.route_topk(rng.standard_normal((T, E)).astype(np.float32), k)
        off, ros, tor = O.permute(idx, E)
        xp = O.gather(X, tor)
        back = O.combine(xp, None, ros, k)
        np.testing.assert_array_equal(back, k * X)


# ---------------------------------------------------------------------------------------------
# grouped GEMMs
# ---------------------------------------------------------------------------------------------
def test_dw_worked_example():
    g = _load("dw1_worked_example.json")
    cum = np.array(g["cumsum_K"])
    offsets = np.concatenate([[0], cum])
    dw = O.grouped_gemm_dw(np.array(g["X"]), np.array(g["G"]), offsets)
    np.testing.assert_array_equal(dw, np.array(g["dW1"]))


def _small_int(rng, shape, lo=-2, hi=2):
    return rng.integers(lo, hi + 1, shape).astype(np.float64)


def test_grouped_gemms_exact_vs_torch():
    """Small-integer operands make every product sum exact, so the oracle must equal torch's
    per-group matmul bit for bit (non-square shapes catch transposed operands)."""
    rng = np.random.default_rng(5)
    counts = [3, 0, 7, 1, 12]
    off = np.concatenate([[0], np.cumsum(counts)])
    R, K, N, G = off[-1], 24, 40, len(counts)
    A = _small_int(rng, (R, K))
    B = _small_int(rng, (G, K, N))
    B2 = _small_int(rng, (G, K, N))
    dC = _small_int(rng, (R, N))
    dC2 = _small_int(rng, (R, N))
    tA, tB, tB2, tdC, tdC2 = (torch.from_numpy(v) for v in (A, B, B2, dC, dC2))
    C = O.grouped_gemm(A, B, off)
    dA = O.grouped_gemm_dx(dC, B, off, dC2, B2)
    dB = O.grouped_gemm_dw(A, dC, off)
    for g in range(G):
        lo, hi = off[g], off[g + 1]
        np.testing.assert_array_equal(C[lo:hi], torch.matmul(tA[lo:hi], tB[g]).numpy())
        np.testing.assert_array_equal(
            dA[lo:hi], (torch.matmul(tdC[lo:hi], tB[g].T) + torch.matmul(tdC2[lo:hi], tB2[g].T)).numpy())
        np.testing.assert_array_equal(dB[g], torch.matmul(tA[lo:hi].T, tdC[lo:hi]).numpy())
    assert np.all(dB[1] == 0)
    # closed form: all-ones operands give K_g in every entry of dB[g]
    ones = O.grouped_gemm_dw(np.ones((R, 3)), np.ones((R, 5)), off)
    for g in range(G):
        assert np.all(ones[g] == counts[g])


def test_grouped_gemm_brute_force_loops():
    rng = np.random.default_rng(6)
    counts = [2, 3, 0, 1]
    off = np.concatenate([[0], np.cumsum(counts)])
    R, K, N = off[-1], 3, 5
    A = rng.standard_normal((R, K))
    B = rng.standard_normal((4, K, N))
    C = O.grouped_gemm(A, B, off, rnd=None)
    dB = O.grouped_gemm_dw(A, C, off)
    for g in range(4):
        for r in range(off[g], off[g + 1]):
            for n in range(N):
                assert abs(C[r, n] - sum(A[r, i] * B[g, i, n] for i in range(K))) < 1e-12
        for i in range(K):
            for n in range(N):
                ref = sum(A[r, i] * C[r, n] for r in range(off[g], off[g + 1]))
                assert abs(dB[g, i, n] - ref) < 1e-12


# ---------------------------------------------------------------------------------------------
# SwiGLU
# ---------------------------------------------------------------------------------------------
def test_swiglu_closed_forms_and_library():
    g = np.array([0.0, 50.0, -50.0, 1.0, -1.0])
    u = np.ones_like(g)
    a = O.swiglu(g, u, rnd=None)
    assert a[0] == 0.0 and abs(a[1] - 50.0) < 1e-12 and abs(a[2]) < 1e-12
    rng = np.random.default_rng(7)
    g = rng.standard_normal(1000) * 4
    u = rng.standard_normal(1000)
    ref = (torch.nn.functional.silu(torch.from_numpy(g)) * torch.from_numpy(u)).numpy()
    np.testing.assert_allclose(O.swiglu(g, u, rnd=None), ref, rtol=1e-13, atol=1e-15)
    # with bf16 storage the result is the bf16 rounding of the exact value
    np.testing.assert_array_equal(O.swiglu(g, u), O.bf16_round(O.swiglu(g, u, rnd=None)))


def test_swiglu_bwd_autograd():
    rng = np.random.default_rng(8)
    g = torch.from_numpy(rng.standard_normal(500) * 3).requires_grad_()
    u = torch.from_numpy(rng.standard_normal(500)).requires_grad_()
    da = torch.from_numpy(rng.standard_normal(500))
    (torch.nn.functional.silu(g) * u).backward(da)
    dhg, dhu = O.swiglu_bwd(g.detach().numpy(), u.detach().numpy(), da.numpy(), rnd=None)
    np.testing.assert_allclose(dhg, g.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(dhu, u.grad.numpy(), rtol=1e-12, atol=1e-14)
    # closed form: sigmoid'(x) = s (1 - s) at 0 gives d/dg silu = 1/2
    dg0, _ = O.swiglu_bwd(np.array([0.0]), np.array([1.0]), np.array([1.0]), rnd=None)
    assert dg0[0] == 0.5


# ---------------------------------------------------------------------------------------------
# whole layer: dense special case, brute-force masked dense, autograd, finite differences
# ---------------------------------------------------------------------------------------------
def _tiny_layer(rng, T=24, d=16, f=20, E=5, k=2, shared_f=0, scale=0.3):
    x = rng.standard_normal((T, d))
    logits = rng.standard_normal((T, E)).astype(np.float32)
    wg = rng.standard_normal((E, d, f)) * scale
    wu = rng.standard_normal((E, d, f)) * scale
    wd = rng.standard_normal((E, f, d)) * scale
    dy = rng.standard_normal((T, d))
    shared = None
    if shared_f:
        shared = (rng.standard_normal((d, shared_f)) * scale, rng.standard_normal((d, shared_f)) * scale,
                  rng.standard_normal((shared_f, d)) * scale)
    return x, logits, wg, wu, wd, dy, shared


def _torch_masked_dense(x, logits, wg, wu, wd, k, shared):
    """Every expert on every token, weighted by the routing weight (0 where not selected)."""
    T, E = logits.shape
    idx, w = O.route_topk(logits, k)      # routing is pinned separately; used as a fixed input
    wfull = np.zeros((T, E))
    np.put_along_axis(wfull, idx, w, 1)
    y = 0
    for e in range(E):
        h = torch.nn.functional.silu(x @ wg[e]) * (x @ wu[e])
        y = y + torch.from_numpy(wfull[:, e:e + 1]) * (h @ wd[e])
    if shared is not None:
        y = y + (torch.nn.functional.silu(x @ shared[0]) * (x @ shared[1])) @ shared[2]
    return y


@pytest.mark.parametrize("shared_f", [0, 12])
def test_layer_forward_vs_brute_force(shared_f):
    rng = np.random.default_rng(9 + shared_f)
    x, logits, wg, wu, wd, dy, shared = _tiny_layer(rng, shared_f=shared_f)
    fwd = O.layer_forward(x, logits, wg, wu, wd, 2, shared=shared, rnd=None)
    tsh = None if shared is None else tuple(torch.from_numpy(s) for s in shared)
    ref = _torch_masked_dense(torch.from_numpy(x), logits, torch.from_numpy(wg), torch.from_numpy(wu),
                              torch.from_numpy(wd), 2, tsh)
    np.testing.assert_allclose(fwd["y"], ref.numpy(), rtol=1e-11, atol=1e-12)
    # with bf16 storage: within a few bf16 ulps of the exact layer output
    fb = O.layer_forward(x, logits, wg, wu, wd, 2, shared=shared)
    assert O.rel_fro(fb["y"], ref.numpy()) < 1e-2


def test_layer_single_expert_is_dense_ffn():
    rng = np.random.default_rng(10)
    x, logits, wg, wu, wd, dy, _ = _tiny_layer(rng, E=1, k=1)
    x = O.bf16_round(x)
    wg, wu, wd = (O.bf16_round(w) for w in (wg, wu, wd))
    fwd = O.layer_forward(x, logits, wg, wu, wd, 1)
    # torch CPU fp32 dense FFN with bf16 rounding at the same stores
    tb = lambda t: t.to(torch.bfloat16).to(torch.float32)
    xt = torch.from_numpy(x).float()
    hg = tb(xt @ torch.from_numpy(wg[0]).float())
    hu = tb(xt @ torch.from_numpy(wu[0]).float())
    a = tb(torch.nn.functional.silu(hg) * hu)
    y = tb(a @ torch.from_numpy(wd[0]).float())
    assert np.all(fwd["topk_w"] == 1.0) and np.all(fwd["topk_idx"] == 0)
    assert O.rel_fro(fwd["y"], y.numpy()) < 1e-2
    assert O.rel_fro(fwd["act"], a.numpy()) < 1e-2


@pytest.mark.parametrize("shared_f", [0, 12])
def test_layer_backward_vs_autograd(shared_f):
    rng = np.random.default_rng(11 + shared_f)
    k = 2
    x, logits, wg, wu, wd, dy, shared = _tiny_layer(rng, shared_f=shared_f)
    fwd = O.layer_forward(x, logits, wg, wu, wd, k, shared=shared, rnd=None)
    bwd = O.layer_backward(fwd, x, dy, wg, wu, wd, shared=shared, rnd=None)

    tx, twg, twu, twd = (torch.from_numpy(v).requires_grad_() for v in (x, wg, wu, wd))
    tsh = None if shared is None else tuple(torch.from_numpy(s).requires_grad_() for s in shared)
    # routing weights as a differentiable input to get d_topk_w
    idx, w = O.route_topk(logits, k)
    tw = torch.from_numpy(w).requires_grad_()
    T, E = logits.shape
    y = 0
    for e in range(E):
        h = torch.nn.functional.silu(tx @ twg[e]) * (tx @ twu[e])
        sel = torch.from_numpy((idx == e).astype(np.float64))
        y = y + (tw * sel).sum(1, keepdim=True) * (h @ twd[e])
    if tsh is not None:
        y = y + (torch.nn.functional.silu(tx @ tsh[0]) * (tx @ tsh[1])) @ tsh[2]
    y.backward(torch.from_numpy(dy))
    tol = dict(rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(bwd["dx"], tx.grad.numpy(), **tol)
    np.testing.assert_allclose(bwd["dw_gate"], twg.grad.numpy(), **tol)
    np.testing.assert_allclose(bwd["dw_up"], twu.grad.numpy(), **tol)
    np.testing.assert_allclose(bwd["dw_down"], twd.grad.numpy(), **tol)
    np.testing.assert_allclose(bwd["d_topk_w"], tw.grad.numpy(), **tol)
    if tsh is not None:
        for key, t in zip(("dw_gate", "dw_up", "dw_down"), tsh):
            np.testing.assert_allclose(bwd["shared"][key], t.grad.numpy(), **tol)


def test_layer_backward_finite_differences():
    rng = np.random.default_rng(12)
    k = 2
    x, logits, wg, wu, wd, dy, shared = _tiny_layer(rng, T=10, d=8, f=6, E=3, shared_f=4)
    loss = lambda x_, wg_, wd_: float((O.layer_forward(x_, logits, wg_, wu, wd_, k, shared=shared,
                                                       rnd=None)["y"] * dy).sum())
    fwd = O.layer_forward(x, logits, wg, wu, wd, k, shared=shared, rnd=None)
    bwd = O.layer_backward(fwd, x, dy, wg, wu, wd, shared=shared, rnd=None)
    h = 1e-6
    for (arr, grad, pos) in ((x, bwd["dx"], (3, 5)), (wg, bwd["dw_gate"], (fwd["topk_idx"][0, 0], 2, 4)),
                             (wd, bwd["dw_down"], (fwd["topk_idx"][1, 1], 1, 7))):
        p, m = arr.copy(), arr.copy()
        p[pos] += h
        m[pos] -= h
        args_p = [x, wg, wd]
        args_m = [x, wg, wd]
        which = 0 if arr is x else (1 if arr is wg else 2)
        args_p[which], args_m[which] = p, m
        fd = (loss(*args_p) - loss(*args_m)) / (2 * h)
        assert abs(fd - grad[pos]) < 1e-6 * max(1.0, abs(fd))


def test_sampled_helpers_match_full_oracle():
    rng = np.random.default_rng(13)
    k = 2
    x, logits, wg, wu, wd, dy, _ = _tiny_layer(rng, T=40, d=16, f=24, E=4)
    x, wg, wu, wd, dy = (O.bf16_round(v) for v in (x, wg, wu, wd, dy))
    fwd = O.layer_forward(x, logits, wg, wu, wd, k)
    bwd = O.layer_backward(fwd, x, dy, wg, wu, wd)
    off = fwd["offsets"]
    e = int(np.argmax(np.diff(off)))
    lo, hi = off[e], off[e + 1]
    rows = np.arange(lo, hi)[::3]
    hg, hu, a, yp = O.expert_rows_forward(fwd["x_perm"][rows], wg[e], wu[e], wd[e])
    np.testing.assert_array_equal(yp, fwd["y_perm"][rows])
    da, dhg, dhu, dxp = O.expert_rows_backward(hg, hu, bwd["dy_perm"][rows], wg[e], wu[e], wd[e])
    np.testing.assert_array_equal(dxp, bwd["dx_perm"][rows])
    cols = np.array([0, 5, 23])
    np.testing.assert_allclose(O.dw_down_rows(fwd["x_perm"][lo:hi], bwd["dy_perm"][lo:hi], wg[e], wu[e], cols),
                               bwd["dw_down"][e][cols], rtol=1e-12)
    dwg, dwu = O.dw_gate_up_cols(fwd["x_perm"][lo:hi], bwd["dy_perm"][lo:hi], wg[e], wu[e], wd[e], cols)
    np.testing.assert_allclose(dwg, bwd["dw_gate"][e][:, cols], rtol=1e-12)
    np.testing.assert_allclose(dwu, bwd["dw_up"][e][:, cols], rtol=1e-12)


# ---------------------------------------------------------------------------------------------
# Router: logits, routing-weight backward, load-balancing loss, router-map backward
# ---------------------------------------------------------------------------------------------
def test_router_logits_one_hot_and_integers():
    """One-hot tokens read rows of Wr exactly; small-integer operands give exact dot products
    checked by explicit loops (no matrix routine)."""
    rng = np.random.default_rng(1)
    d, E = 12, 5
    wr = rng.normal(0, 0.02, (d, E))
    x = np.eye(d)[[3, 0, 11]]
    np.testing.assert_array_equal(O.router_logits(x, wr), wr[[3, 0, 11]])
    bias = rng.normal(size=E)
    np.testing.assert_array_equal(O.router_logits(x, wr, bias), wr[[3, 0, 11]] + bias)
    xi = rng.integers(-3, 4, (7, d)).astype(float)
    wi = rng.integers(-3, 4, (d, E)).astype(float)
    want = [[sum(xi[t, i] * wi[i, e] for i in range(d)) for e in range(E)] for t in range(7)]
    np.testing.assert_array_equal(O.router_logits(xi, wi), np.array(want))


@pytest.mark.parametrize("normalize", [True, False])
def test_route_topk_bwd_autograd(normalize):
    """dlogits against torch autograd of the routing weights (softmax over the selected logits,
    or the full softmax read at the selected experts), selection held fixed."""
    rng = np.random.default_rng(2)
    T, E, k = 9, 7, 3
    L = rng.normal(size=(T, E)) * 2
    idx, w = O.route_topk(L, k, normalize)
    g = rng.normal(size=(T, k))
    Lt = torch.tensor(L, dtype=torch.float64, requires_grad=True)
    it = torch.tensor(idx)
    if normalize:
        wt = torch.softmax(torch.gather(Lt, 1, it), dim=1)
    else:
        wt = torch.gather(torch.softmax(Lt, dim=1), 1, it)
    np.testing.assert_allclose(wt.detach().numpy(), w, rtol=1e-12)
    (wt * torch.tensor(g)).sum().backward()
    np.testing.assert_allclose(O.route_topk_bwd(L, idx, g, normalize), Lt.grad.numpy(), rtol=1e-10, atol=1e-14)


def test_route_topk_bwd_properties_and_fd():
    """Rows of the normalized-weight gradient sum to zero (the k weights sum to one) and vanish
    outside the selection; one central finite difference of sum(g * w)."""
    rng = np.random.default_rng(3)
    T, E, k = 6, 8, 2
    L = rng.normal(size=(T, E))
    idx, _ = O.route_topk(L, k)
    g = rng.normal(size=(T, k))
    dl = O.route_topk_bwd(L, idx, g)
    np.testing.assert_allclose(dl.sum(axis=1), 0, atol=1e-14)
    mask = np.zeros((T, E), bool)
    np.put_along_axis(mask, idx, True, axis=1)
    assert (dl[~mask] == 0).all()
    t, e = 4, int(idx[4, 1])
    h = 1e-6
    f = lambda LL: (g * O.route_topk(LL, k)[1]).sum()
    Lp, Lm = L.copy(), L.copy()
    Lp[t, e] += h
    Lm[t, e] -= h
    assert abs((f(Lp) - f(Lm)) / (2 * h) - dl[t, e]) < 1e-8


def test_aux_loss_closed_form_and_autograd():
    """Uniform logits give P_e = 1/E, so L = alpha * E * sum_e f_e / E = alpha whatever the counts;
    the gradient against torch autograd with the counts held constant."""
    T, E, k, alpha = 10, 6, 2, 0.01
    counts = np.array([7, 0, 3, 5, 4, 1])
    loss, grad = O.aux_loss(np.zeros((T, E)), counts, k, alpha)
    assert abs(loss - alpha) < 1e-15
    np.testing.assert_allclose(grad.sum(axis=1), 0, atol=1e-16)
    rng = np.random.default_rng(4)
    L = rng.normal(size=(T, E))
    loss, grad = O.aux_loss(L, counts, k, alpha)
    Lt = torch.tensor(L, requires_grad=True)
    f = torch.tensor(counts / (T * k))
    lt = alpha * E * (f * torch.softmax(Lt, dim=1).mean(dim=0)).sum()
    lt.backward()
    assert abs(lt.item() - loss) < 1e-14
    np.testing.assert_allclose(grad, Lt.grad.numpy(), rtol=1e-10, atol=1e-16)


def test_router_bwd_autograd():
    """dWr and the token gradient against torch autograd of logits = x . Wr; the stored-dX sum
    rounds once."""
    rng = np.random.default_rng(5)
    T, d, E = 5, 8, 4
    x, wr, g = rng.normal(size=(T, d)), rng.normal(size=(d, E)), rng.normal(size=(T, E))
    xt = torch.tensor(x, requires_grad=True)
    wt = torch.tensor(wr, requires_grad=True)
    (xt @ wt * torch.tensor(g)).sum().backward()
    dwr, dxr = O.router_bwd(x, wr, g, rnd=None)
    np.testing.assert_allclose(dwr, wt.grad.numpy(), rtol=1e-12)
    np.testing.assert_allclose(dxr, xt.grad.numpy(), rtol=1e-12)
    dx0 = O.bf16_round(rng.normal(size=(T, d)))
    _, dxs = O.router_bwd(x, wr, g, dx=dx0)
    np.testing.assert_array_equal(dxs, O.bf16_round(dx0 + xt.grad.numpy()))


# ---------------------------------------------------------------------------------------------
# FP8 (E4M3) variant
# ---------------------------------------------------------------------------------------------
def test_e4m3_decode_spec_values_and_torch():
    """Values fixed by the E4M3 format definition, and torch's float8_e4m3fn decoding of every
    code (a library routine)."""
    spec = {0x00: 0.0, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9, 0x08: 2.0 ** -6, 0x38: 1.0, 0x3C: 1.5,
            0x40: 2.0, 0x77: 240.0, 0x7E: 448.0, 0x80: -0.0, 0xB8: -1.0, 0xFE: -448.0}
    v = O.e4m3_decode(np.arange(256, dtype=np.uint8))
    for c, val in spec.items():
        assert v[c] == val and np.signbit(v[c]) == np.signbit(val), hex(c)
    assert np.isnan(v[0x7F]) and np.isnan(v[0xFF]) and np.isnan(v).sum() == 2
    t = torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn).double().numpy()
    np.testing.assert_array_equal(v, t)


def _e4m3_nearest_brute(x):
    """Nearest finite E4M3 code by exhaustive search, ties to the even code, saturating."""
    codes = np.arange(256, dtype=np.uint8)
    vals = O.e4m3_decode(codes)
    ok = ~np.isnan(vals) & ((codes & 0x80) == 0)          # non-negative codes; sign applied after
    cv, vv = codes[ok].astype(np.int64), vals[ok]
    out = []
    for xi in np.asarray(x, dtype=np.float64):
        a = min(abs(xi), 448.0)
        d = np.abs(vv - a)
        best = cv[d == d.min()]
        c = int(best[0]) if len(best) == 1 else int(best[best % 2 == 0][0])
        out.append(c | (0x80 if np.signbit(xi) else 0))
    return np.array(out, dtype=np.uint8)


def test_e4m3_encode_brute_force_and_torch():
    rng = np.random.default_rng(8)
    vals = O.e4m3_decode(np.arange(0, 0x7F, dtype=np.uint8))            # 0 .. 448
    mids = (vals[1:] + vals[:-1]) / 2                                    # exact ties
    x = np.concatenate([rng.uniform(-470, 470, 3000), rng.normal(0, 0.01, 1000), mids, -mids,
                        vals, [0.0, -0.0, 1e-12, -1e-12, 448.0, 463.9, 1e6, -1e6]])
    got = O.e4m3_encode(x)
    np.testing.assert_array_equal(got, _e4m3_nearest_brute(x))
    inr = np.abs(x) < 464                                                # torch overflows to NaN beyond
    t = torch.from_numpy(x[inr]).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    np.testing.assert_array_equal(got[inr], t)
    assert O.e4m3_encode(np.array([np.nan]))[0] == 0x7F
    assert O.e4m3_encode(np.array([1e9]))[0] == 0x7E and O.e4m3_encode(np.array([-1e9]))[0] == 0xFE


def test_quantize_rows_fp8_properties():
    rng = np.random.default_rng(9)
    x = O.bf16_round(rng.normal(0, 1, (40, 96)) * rng.uniform(0.01, 100, (40, 1)))
    x[3] = 0.0
    codes, scale = O.quantize_rows_fp8(x)
    assert codes.dtype == np.uint8 and scale.dtype == np.float32
    dec = O.e4m3_decode(codes)
    assert np.all(codes[3] == 0) and scale[3] == 1.0
    nz = np.arange(40) != 3
    # each row's largest magnitude lands on 448 (saturation absorbs the fp32 rounding of 448/amax)
    np.testing.assert_array_equal(np.abs(dec[nz]).max(axis=1), 448.0)
    # reconstruction within half an E4M3 spacing (relative 2**-4) plus the fp32 rounding of the
    # scaled value, and the subnormal spacing near zero
    rec = dec * scale[:, None].astype(np.float64)
    tol = (np.abs(x) * (2.0 ** -4 + 2.0 ** -20) + 2.0 ** -10 * scale[:, None]) * 1.0001
    assert np.all(np.abs(rec - x) <= tol)
    # the scale is amax / 448 in fp32
    amax = np.abs(x).max(axis=1).astype(np.float32)
    np.testing.assert_array_equal(scale[nz], (amax / np.float32(448))[nz])


def test_grouped_gemm_fp8_vs_library():
    """Exact on small-integer codes (torch matmul of the decoded operands, then the scales), and
    linear in each scale."""
    rng = np.random.default_rng(10)
    counts = [5, 0, 7, 1, 3]
    G, R, K, N = len(counts), sum(counts), 32, 12
    off = np.concatenate([[0], np.cumsum(counts)])
    ints = np.arange(-4, 5, dtype=np.float64)
    a = O.e4m3_encode(rng.choice(ints, (R, K)))
    w = O.e4m3_encode(rng.choice(ints, (G, N, K)))
    sa = np.float32(2.0) ** rng.integers(-3, 3, R).astype(np.float32)
    sw = np.float32(2.0) ** rng.integers(-3, 3, (G, N)).astype(np.float32)
    got = O.grouped_gemm_fp8(a, sa, w, sw, off, rnd=None)
    A = torch.from_numpy(O.e4m3_decode(a))
    W = torch.from_numpy(O.e4m3_decode(w))
    for g in range(G):
        lo, hi = off[g], off[g + 1]
        ref = (A[lo:hi] @ W[g].T).numpy() * sa[lo:hi, None] * sw[g][None, :]
        np.testing.assert_array_equal(got[lo:hi], ref)
    sa2 = sa.copy()
    sa2[2] *= 4
    np.testing.assert_array_equal(O.grouped_gemm_fp8(a, sa2, w, sw, off, rnd=None)[2], 4 * got[2])
    np.testing.assert_array_equal(O.grouped_gemm_fp8(a, sa, w, sw, off), O.bf16_round(got))


# ---------------------------------------------------------------------------------------------
# MX variant: E4M3 elements with a power-of-two scale per 32 elements
# ---------------------------------------------------------------------------------------------
def test_mx_block_exponent_hand_values():
    """The smallest e with amax <= 448 * 2**e, worked by hand; -127 at the bottom."""
    cases = {
        448.0: 0,            # exactly the largest E4M3 magnitude
        450.0: 1,            # the next bf16 above 448 no longer fits at e = 0
        224.0: -1,           # 448 / 2 fits at e = -1 (and 224 > 448 * 2**-2 = 112)
        225.0: 0,
        1.0: -8,             # 448 * 2**-8 = 1.75 >= 1 > 0.875 = 448 * 2**-9
        1.75: -8,            # equal to 448 * 2**-8
        1.7578125: -7,       # the next bf16 above 1.75
        256.0: 0,            # a power of two: 256 <= 448 (a floor(log2) - 8 rule gives 0 too)
        300.0: 0,
        500.0: 1,            # floor(log2(500)) - 8 = 0 would saturate: 500 > 448
        0.0: -127,           # an all-zero block
        2.0 ** -140: -127,   # e would be -148: raised to the smallest scale
        448.0 * 2.0 ** -127: -127,
        448.0 * 2.0 ** -126: -126,
    }
    for amax, e in cases.items():
        assert int(O.mx_block_exponent(np.array([amax]))[0]) == e, amax
    for k in (-100, -20, -1, 3, 60, 110):
        assert int(O.mx_block_exponent(np.array([448.0 * 2.0 ** k]))[0]) == k
        assert int(O.mx_block_exponent(np.array([450.0 * 2.0 ** k]))[0]) == k + 1


def test_quantize_rows_mx_worked_example():
    """One row of three blocks, every code and scale byte worked by hand.
    Block 0: amax 100 -> e = -2 (100 <= 448/4 = 112, 100 > 56), byte 125; scaled values x * 4:
      100 -> 400, halfway between 384 and 416: ties to the even mantissa, 384 = 1.5 * 2**8 ->
      exponent field 15, mantissa 4: 0x7C;  1 -> 4 = 2**2: field 9, mantissa 0: 0x48;
      -3.5 -> -14 = -1.75 * 2**3: field 10, mantissa 6, sign: 0xD6;  2**-9 -> 2**-7, a subnormal,
      4 * 2**-9: 0x04;  the rest 0.
    Block 1: all zero -> byte 0 and zero codes.
    Block 2: amax 0.4375 = 448 * 2**-10 -> byte 117; 0.4375 -> 448: 0x7E; -0.25 -> -256 =
      -2**8: field 15, mantissa 0, sign: 0xF8."""
    x = np.zeros((1, 96))
    x[0, 0], x[0, 1], x[0, 2], x[0, 3] = 100.0, 1.0, -3.5, 2.0 ** -9
    x[0, 64], x[0, 70] = 0.4375, -0.25
    codes, sb = O.quantize_rows_mx(x)
    assert codes.dtype == np.uint8 and sb.dtype == np.uint8 and sb.shape == (1, 3)
    assert sb.tolist() == [[125, 0, 117]]
    want = np.zeros(96, dtype=np.uint8)
    want[0], want[1], want[2], want[3], want[64], want[70] = 0x7C, 0x48, 0xD6, 0x04, 0x7E, 0xF8
    np.testing.assert_array_equal(codes[0], want)
    # decoded: 384 * 2**-2 = 96 for the tie, the others exact
    dec = O.mx_decode(codes, sb)[0]
    assert dec[0] == 96.0 and dec[1] == 1.0 and dec[2] == -3.5 and dec[3] == 2.0 ** -9
    assert dec[64] == 0.4375 and dec[70] == -0.25 and not np.any(dec[32:64])


def test_quantize_rows_mx_properties():
    """On rows whose blocks span many magnitudes (and all-zero and tiny blocks): the scaled block
    never exceeds 448 and a smaller exponent would (unless at -127); each code is the nearest E4M3
    value to x * 2**-e by exhaustive search; blocks are quantized independently."""
    rng = np.random.default_rng(11)
    R, C = 6, 256
    mag = 2.0 ** rng.integers(-30, 30, (R, C // 32))
    x = O.bf16_round(rng.normal(0, 1, (R, C)) * np.repeat(mag, 32, axis=1))
    x[1, 32:64] = 0.0
    x[2, 0:32] = O.bf16_round(rng.normal(0, 1, 32) * 2.0 ** -131)        # bf16 subnormals
    codes, sb = O.quantize_rows_mx(x)
    e = sb.astype(np.int64) - 127
    blocks = x.reshape(R, C // 32, 32)
    amax = np.abs(blocks).max(axis=2)
    assert sb[1, 1] == 0 and not np.any(codes[1, 32:64])
    assert np.all(amax <= np.ldexp(448.0, e))
    assert np.all((e == -127) | (amax > np.ldexp(448.0, e - 1)))
    scaled = np.ldexp(blocks, -e[..., None]).reshape(-1)
    np.testing.assert_array_equal(codes.reshape(-1), _e4m3_nearest_brute(scaled))
    # block independence: changing block 3 of row 0 changes nothing else
    x2 = x.copy()
    x2[0, 96:128] *= 1024.0
    c2, s2 = O.quantize_rows_mx(x2)
    assert s2[0, 3] == sb[0, 3] + 10
    keep = np.ones(C, dtype=bool)
    keep[96:128] = False
    np.testing.assert_array_equal(c2[0, keep], codes[0, keep])
    np.testing.assert_array_equal(np.delete(s2, 3, axis=1), np.delete(sb, 3, axis=1))


def test_grouped_gemm_mx_vs_library():
    """Exact on small-integer codes with random block scales: torch matmuls of one 32-column block
    at a time, each scaled by its two scale columns, summed over the blocks; one scale byte one
    higher doubles exactly its block's share."""
    rng = np.random.default_rng(12)
    counts = [5, 0, 7, 1, 3]
    G, R, K, N = len(counts), sum(counts), 96, 12
    off = np.concatenate([[0], np.cumsum(counts)])
    ints = np.arange(-4, 5, dtype=np.float64)
    a = O.e4m3_encode(rng.choice(ints, (R, K)))
    w = O.e4m3_encode(rng.choice(ints, (G, N, K)))
    sa = rng.integers(120, 134, (R, K // 32)).astype(np.uint8)
    sw = rng.integers(120, 134, (G, N, K // 32)).astype(np.uint8)
    got = O.grouped_gemm_mx(a, sa, w, sw, off, rnd=None)
    A = torch.from_numpy(O.e4m3_decode(a))
    W = torch.from_numpy(O.e4m3_decode(w))
    SA = torch.from_numpy(2.0 ** (sa.astype(np.float64) - 127))
    SW = torch.from_numpy(2.0 ** (sw.astype(np.float64) - 127))
    for g in range(G):
        lo, hi = off[g], off[g + 1]
        ref = torch.zeros(hi - lo, N, dtype=torch.float64)
        for b in range(K // 32):
            cols = slice(32 * b, 32 * b + 32)
            ref += (A[lo:hi, cols] @ W[g][:, cols].T) * SA[lo:hi, b][:, None] * SW[g][:, b][None, :]
        np.testing.assert_array_equal(got[lo:hi], ref.numpy())
    sa2 = sa.copy()
    sa2[2, 1] += 1
    share = (A[2, 32:64] @ W[0][:, 32:64].T).numpy() * 2.0 ** (sa[2, 1] - 127.0) * \
        (2.0 ** (sw[0][:, 1].astype(np.float64) - 127))
    np.testing.assert_array_equal(O.grouped_gemm_mx(a, sa2, w, sw, off, rnd=None)[2], got[2] + share)
    np.testing.assert_array_equal(O.grouped_gemm_mx(a, sa, w, sw, off), O.bf16_round(got))


def test_pack_groups_t_brute_force():
    """Every element placed by hand-style loops: group g's i-th row becomes column p[g] + i, the
    starts are the 128-rounded prefix of the counts (empty groups take no columns), the rest zero."""
    rng = np.random.default_rng(13)
    counts = [5, 0, 130, 128, 1]
    off = np.concatenate([[0], np.cumsum(counts)])
    x = rng.normal(0, 1, (sum(counts), 7))
    got, p = O.pack_groups_t(x, off)
    assert p.tolist() == [0, 128, 128, 384, 512, 640]
    want = np.zeros((7, 640))
    for g in range(len(counts)):
        for i in range(counts[g]):
            for c in range(7):
                want[c, p[g] + i] = x[off[g] + i, c]
    np.testing.assert_array_equal(got, want)
    got32, p32 = O.pack_groups_t(x, off, align=32)
    assert p32.tolist() == [0, 32, 32, 192, 320, 352] and got32.shape == (7, 352)


def test_grouped_gemm_dw_mx_vs_library():
    """The MX weight gradient on integer codes with random block scales: exact against torch's
    matmul of each group's un-padded token columns, one 32-token block at a time with the block's
    scales; padding columns (zero codes) add nothing; an empty group's gradient is zero."""
    rng = np.random.default_rng(14)
    counts = [40, 0, 150, 7]
    off = np.concatenate([[0], np.cumsum(counts)])
    K, N = 6, 5
    L = 128 + 0 + 256 + 128
    ints = np.arange(-4, 5, dtype=np.float64)
    at = np.zeros((K, L))
    ct = np.zeros((N, L))
    _, p = O.pack_groups_t(np.zeros((sum(counts), 1)), off)
    for g in range(len(counts)):
        at[:, p[g]:p[g] + counts[g]] = rng.choice(ints, (K, counts[g]))
        ct[:, p[g]:p[g] + counts[g]] = rng.choice(ints, (N, counts[g]))
    ac, cc = O.e4m3_encode(at), O.e4m3_encode(ct)
    sa = rng.integers(122, 132, (K, L // 32)).astype(np.uint8)
    sc = rng.integers(122, 132, (N, L // 32)).astype(np.uint8)
    got = O.grouped_gemm_dw_mx(ac, sa, cc, sc, off)
    A, C = torch.from_numpy(at), torch.from_numpy(ct)
    SA = torch.from_numpy(2.0 ** (sa.astype(np.float64) - 127))
    SC = torch.from_numpy(2.0 ** (sc.astype(np.float64) - 127))
    for g in range(len(counts)):
        ref = torch.zeros(K, N, dtype=torch.float64)
        for b in range(int(p[g]) // 32, int(p[g + 1]) // 32):
            cols = slice(32 * b, 32 * b + 32)
            ref += (A[:, cols] * SA[:, b:b + 1]) @ (C[:, cols] * SC[:, b:b + 1]).T
        np.testing.assert_array_equal(got[g], ref.numpy())
    assert not np.any(got[1])


# ---------------------------------------------------------------------------------------------
# the comparison metric every floating-point parity check goes through
# ---------------------------------------------------------------------------------------------
def test_rel_fro_hand_values():
    """rel_fro(got, ref) = ||got - ref||_F / ||ref||_F over the whole tensor, values worked by hand."""
    # ref = [[3, 0], [0, 4]] has norm 5; the difference [[1, 2], [2, 0]] has norm 3: exactly 3/5.
    # (A squared ratio gives 0.36, dividing by ||got|| = sqrt(40) gives 0.4743, no square root
    # gives 9/25 as well, a max-abs ratio gives 2/4.)
    ref = np.array([[3.0, 0.0], [0.0, 4.0]])
    got = np.array([[4.0, 2.0], [2.0, 4.0]])
    assert O.rel_fro(got, ref) == 0.6
    # not symmetric: with the roles swapped the denominator is sqrt(40)
    assert abs(O.rel_fro(ref, got) - 3.0 / math.sqrt(40.0)) < 1e-15
    # one Frobenius norm over the tensor, not a mean of per-row ratios: ref rows of norm 1 and 100,
    # an error of 1 in the first row only -> 1 / sqrt(10001) (a per-row mean would give 0.5)
    ref = np.array([[1.0, 0.0], [0.0, 100.0]])
    got = np.array([[2.0, 0.0], [0.0, 100.0]])
    assert abs(O.rel_fro(got, ref) - 1.0 / math.sqrt(10001.0)) < 1e-15
    # a 3-4-5 error on a 12-5-13 reference, in three dimensions: 5/13
    ref = np.array([12.0, 5.0, 0.0]).reshape(1, 3, 1)
    got = np.array([15.0, 9.0, 0.0]).reshape(1, 3, 1)
    assert abs(O.rel_fro(got, ref) - 5.0 / 13.0) < 1e-15
    # scale invariance, and exactness on equal inputs
    assert abs(O.rel_fro(7.0 * got, 7.0 * ref) - 5.0 / 13.0) < 1e-15
    assert O.rel_fro(ref, ref) == 0.0
    # the zero-reference conventions: 0/0 -> 0 (an exactly zero output matches), x/0 -> inf
    z = np.zeros((3, 2))
    assert O.rel_fro(z, z) == 0.0
    assert O.rel_fro(np.full((3, 2), 1e-30), z) == float("inf")
    # float64 norms: values whose squares overflow float32 still give the exact ratio
    ref = np.array([3e30, 4e30])
    got = np.array([3e30, 4e30 + 5e29])
    assert abs(O.rel_fro(got, ref) - 0.1) < 1e-15
    # inputs of any dtype are compared in float64 (bf16-valued float32 arrays here)
    ref32 = np.array([[3.0, 0.0], [0.0, 4.0]], dtype=np.float32)
    got32 = np.array([[4.0, 2.0], [2.0, 4.0]], dtype=np.float32)
    assert O.rel_fro(got32, ref32) == 0.6
