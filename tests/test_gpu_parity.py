"""GPU parity of every library entry point against the CPU oracle (same seeded inputs).

Integers (routing indices, offsets, permutation) and bit copies must match exactly; GEMMs on
small-integer operands must match exactly; every floating output must be within Frobenius-relative
2e-2 of the oracle and finite."""
import sys

import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2606_26453_amd import layer as L
from paper_2606_26453_amd import moe, workloads as W
from tests.gpu_util import FRO_TOL, check_float, f64, gpu_available, i64, poison_

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

DEV = "cuda:0"


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


# ---------------------------------------------------------------------------------------------
# routing + permutation + gather: bit exact
# ---------------------------------------------------------------------------------------------
ROUTE_CASES = [
    # T, E, k, d, normalize, special
    (256, 4, 2, 256, True, None),
    (1, 1, 1, 64, True, None),
    (63, 8, 8, 128, True, None),          # k = E
    (1, 16, 3, 64, True, None),
    (1000, 64, 6, 64, True, "ties"),
    (777, 256, 8, 64, True, None),        # E = 256
    (500, 32, 4, 128, True, "empty"),     # forced-empty experts
    (300, 64, 6, 64, False, None),        # unnormalized full-softmax weights
    (4097, 128, 4, 64, True, "ties"),
    (20000, 16, 2, 64, True, None),       # several ranges of slots
]


@pytest.mark.parametrize("case", ROUTE_CASES, ids=[f"T{c[0]}_E{c[1]}_k{c[2]}_{c[5]}_{'n' if c[4] else 'u'}" for c in ROUTE_CASES])
def test_route_permute_bit_exact(case):
    T, E, k, d, normalize, special = case
    _say("route_permute", case)
    g = torch.Generator().manual_seed(T * 7 + E)
    logits = torch.randn((T, E), generator=g)
    if special == "ties":
        logits = torch.round(logits * 2) / 2      # many exact ties
    if special == "empty":
        logits[:, :5] -= 1e4
    x = torch.randn((T, d), generator=g).to(torch.bfloat16)
    out = moe.moe_route_permute(logits.to(DEV), x.to(DEV), k, normalize)
    torch.cuda.synchronize()
    idx, w = O.route_topk(logits.numpy(), k, normalize)
    off, ros, tor = O.permute(idx, E)
    np.testing.assert_array_equal(i64(out["topk_idx"]), idx)
    np.testing.assert_array_equal(i64(out["offsets"]), off)
    np.testing.assert_array_equal(i64(out["row_of_slot"]), ros)
    np.testing.assert_array_equal(i64(out["token_of_row"]), tor)
    np.testing.assert_array_equal(out["x_perm"].cpu().view(torch.int16).numpy(),
                                  x.view(torch.int16).numpy()[tor])
    np.testing.assert_allclose(f64(out["topk_w"]), w, rtol=2e-6, atol=1e-7)


def test_route_permute_deterministic():
    T, E, k = 5000, 64, 6
    g = torch.Generator().manual_seed(3)
    logits = torch.randn((T, E), generator=g).to(DEV)
    x = torch.randn((T, 64), generator=g).to(torch.bfloat16).to(DEV)
    outs = [moe.moe_route_permute(logits, x, k) for _ in range(3)]
    torch.cuda.synchronize()
    for key in outs[0]:
        for o in outs[1:]:
            assert torch.equal(outs[0][key], o[key]), key


# ---------------------------------------------------------------------------------------------
# grouped GEMMs: exact on small-integer operands, ragged groups spanning several tiles
# ---------------------------------------------------------------------------------------------
GROUPS = [1, 63, 64, 65, 127, 0, 128, 129, 300, 513, 0, 31]


def _int_tensor(g, shape, lo=-1, hi=1):
    return torch.randint(lo, hi + 1, shape, generator=g).to(torch.bfloat16)


@pytest.mark.parametrize("K,N", [(192, 320), (256, 512), (64, 64)])
def test_grouped_gemm_fwd_exact(K, N):
    _say("gemm_fwd exact", K, N)
    g = torch.Generator().manual_seed(K + N)
    counts = GROUPS
    G, R = len(counts), sum(counts)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    A = _int_tensor(g, (R, K))
    B = _int_tensor(g, (G, K, N))
    B2 = _int_tensor(g, (G, K, N))
    C, C2, act = (poison_(torch.empty((R, N), dtype=torch.bfloat16, device=DEV)) for _ in range(3))
    moe.moe_grouped_gemm_fwd(A.to(DEV), B.to(DEV), off.to(DEV), B2.to(DEV), C, C2, act, want_act=True)
    C1 = poison_(torch.empty((R, N), dtype=torch.bfloat16, device=DEV))
    moe.moe_grouped_gemm_fwd(A.to(DEV), B.to(DEV), off.to(DEV), C=C1)
    torch.cuda.synchronize()
    refC = O.grouped_gemm(f64(A), f64(B), off.numpy())
    refC2 = O.grouped_gemm(f64(A), f64(B2), off.numpy())
    np.testing.assert_array_equal(f64(C), refC)
    np.testing.assert_array_equal(f64(C2), refC2)
    np.testing.assert_array_equal(f64(C1), refC)
    check_float("act", f64(act), O.swiglu(refC, refC2), tol=1e-2)


@pytest.mark.parametrize("K,N", [(192, 320), (320, 128)])
def test_grouped_gemm_dx_exact(K, N):
    _say("gemm_dx exact", K, N)
    g = torch.Generator().manual_seed(10 * K + N)
    counts = GROUPS
    G, R = len(counts), sum(counts)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    dC = _int_tensor(g, (R, N))
    dC2 = _int_tensor(g, (R, N))
    B = _int_tensor(g, (G, K, N))
    B2 = _int_tensor(g, (G, K, N))
    dA = poison_(torch.empty((R, K), dtype=torch.bfloat16, device=DEV))
    dA1 = poison_(torch.empty((R, K), dtype=torch.bfloat16, device=DEV))
    moe.moe_grouped_gemm_dx(dC.to(DEV), B.to(DEV), off.to(DEV), dC2.to(DEV), B2.to(DEV), dA=dA)
    moe.moe_grouped_gemm_dx(dC.to(DEV), B.to(DEV), off.to(DEV), dA=dA1)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(f64(dA), O.grouped_gemm_dx(f64(dC), f64(B), off.numpy(), f64(dC2), f64(B2)))
    np.testing.assert_array_equal(f64(dA1), O.grouped_gemm_dx(f64(dC), f64(B), off.numpy()))


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5, 6, 8, 9])
@pytest.mark.parametrize("d", [64, 576])
def test_combine_exact(k, d):
    """The weighted and unweighted combine (with and without the added token rows) and its
    backward, for every k the library specialises (1, 2, 4, 6, 8) and others (the general path),
    on small integers with power-of-two weights, where every fp32 sum is exact: bit-equal to the
    oracle.  d = 576 gives each lane several 16-byte chunks (72 per row)."""
    _say("combine exact", k, d)
    g = torch.Generator().manual_seed(1000 * k + d)
    T = 37
    R = T * k
    row_of_slot = torch.randperm(R, generator=g).to(torch.int32)
    w = (2.0 ** torch.randint(-2, 2, (T, k), generator=g)).to(torch.float32)
    y_perm = _int_tensor(g, (R, d), -8, 8)
    add = _int_tensor(g, (T, d), -8, 8)
    dy = _int_tensor(g, (T, d), -8, 8)
    dv = lambda t: t.to(DEV)
    rs = i64(row_of_slot)
    for wt, ad in ((w, None), (None, None), (w, add), (None, add)):
        y = poison_(torch.empty((T, d), dtype=torch.bfloat16, device=DEV))
        moe.moe_unpermute_combine(dv(y_perm), None if wt is None else dv(wt), dv(row_of_slot), k,
                                  add=None if ad is None else dv(ad), y=y)
        torch.cuda.synchronize()
        ref = O.combine(f64(y_perm), None if wt is None else f64(wt), rs, k, add=None if ad is None else f64(ad))
        np.testing.assert_array_equal(f64(y), ref)
    for yp in (y_perm, None):
        dy_perm = poison_(torch.empty((R, d), dtype=torch.bfloat16, device=DEV))
        d_w = poison_(torch.empty((T, k), dtype=torch.float32, device=DEV)) if yp is not None else None
        moe.moe_unpermute_combine_bwd(dv(dy), dv(w), dv(row_of_slot), k, y_perm=None if yp is None else dv(yp),
                                      dy_perm=dy_perm, d_topk_w=d_w)
        torch.cuda.synchronize()
        ref_p, ref_w = O.combine_bwd(f64(dy), f64(w), rs, None if yp is None else f64(yp), k)
        np.testing.assert_array_equal(f64(dy_perm), ref_p)
        if yp is not None:
            np.testing.assert_array_equal(f64(d_w), ref_w)


def test_combine_exact_large():
    """The weighted combine over a Y_perm larger than half the Infinity Cache (the streaming-load
    branch; 8192 tokens x top-4 x d = 4096: 256 MiB), with the added rows, and its backward: exact
    against the oracle on small integers with power-of-two weights, on 256 sampled tokens (the
    oracle reads only their slots' rows)."""
    T, k, d = 8192, 4, 4096
    _say("combine exact large", T, k, d)
    g = torch.Generator().manual_seed(4096)
    R = T * k
    row_of_slot = torch.randperm(R, generator=g).to(torch.int32)
    w = (2.0 ** torch.randint(-2, 2, (T, k), generator=g)).to(torch.float32)
    y_perm = _int_tensor(g, (R, d), -8, 8)
    add = _int_tensor(g, (T, d), -8, 8)
    dy = _int_tensor(g, (T, d), -8, 8)
    y = poison_(torch.empty((T, d), dtype=torch.bfloat16, device=DEV))
    moe.moe_unpermute_combine(y_perm.to(DEV), w.to(DEV), row_of_slot.to(DEV), k, add=add.to(DEV), y=y)
    dy_perm = poison_(torch.empty((R, d), dtype=torch.bfloat16, device=DEV))
    d_w = poison_(torch.empty((T, k), dtype=torch.float32, device=DEV))
    moe.moe_unpermute_combine_bwd(dy.to(DEV), w.to(DEV), row_of_slot.to(DEV), k, y_perm=y_perm.to(DEV),
                                  dy_perm=dy_perm, d_topk_w=d_w)
    torch.cuda.synchronize()
    sub = torch.randperm(T, generator=g)[:256].sort().values
    rows = i64(row_of_slot).reshape(T, k)[sub.numpy()]           # [256, k] rows of Y_perm
    yp_sub = f64(y_perm[torch.as_tensor(rows.reshape(-1))])        # those rows, slot by slot
    local = np.arange(rows.size)
    np.testing.assert_array_equal(f64(y[sub]), O.combine(yp_sub, f64(w[sub]), local, k, add=f64(add[sub])))
    ref_p, ref_w = O.combine_bwd(f64(dy[sub]), f64(w[sub]), local, yp_sub, k)
    np.testing.assert_array_equal(f64(dy_perm[torch.as_tensor(rows.reshape(-1)).to(DEV)]), ref_p)
    np.testing.assert_array_equal(f64(d_w[sub.to(DEV)]), ref_w)


@pytest.mark.parametrize("K,N", [(192, 320), (256, 256), (576, 64)])
def test_grouped_gemm_dw_exact(K, N):
    _say("gemm_dw exact", K, N)
    g = torch.Generator().manual_seed(100 * K + N)
    counts = GROUPS
    G, R = len(counts), sum(counts)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    A = _int_tensor(g, (R, K), -2, 2)
    dC = _int_tensor(g, (R, N), -2, 2)
    dC2 = _int_tensor(g, (R, N), -2, 2)
    dB, dB2, dB1 = (poison_(torch.empty((G, K, N), dtype=torch.float32, device=DEV)) for _ in range(3))
    moe.moe_grouped_gemm_dw(A.to(DEV), dC.to(DEV), off.to(DEV), dC2.to(DEV), dB, dB2)
    moe.moe_grouped_gemm_dw(A.to(DEV), dC.to(DEV), off.to(DEV), dB=dB1)
    torch.cuda.synchronize()
    ref = O.grouped_gemm_dw(f64(A), f64(dC), off.numpy())
    np.testing.assert_array_equal(f64(dB), ref)
    np.testing.assert_array_equal(f64(dB1), ref)
    np.testing.assert_array_equal(f64(dB2), O.grouped_gemm_dw(f64(A), f64(dC2), off.numpy()))
    assert torch.count_nonzero(dB[5]) == 0 and torch.count_nonzero(dB[10]) == 0   # empty groups


@pytest.mark.parametrize("K,N,R,dual", [(512, 256, 8192, False),      # 2 tiles: every tile split (4 pieces)
                                         (512, 256, 8192, True),
                                         (4352, 4096, 16384, False),    # 272 tiles: a round plus 16 split 8 ways
                                         (256, 256, 4000, True)])       # contraction too short to split
def test_grouped_gemm_dw_split_exact(K, N, R, dual):
    """moe_grouped_gemm_dw_split on one group (the shared experts' weight gradient): tiles of the
    last round split along the contraction, partial tiles summed in piece order; exact against
    the oracle on small-integer operands (every partial and total sum exact in fp32), twice in a
    row on the same counters and workspace; with several groups the workspace is unused and the
    result is bitwise moe_grouped_gemm_dw_persistent's."""
    _say("gemm dw split", K, N, R, dual)
    g = torch.Generator().manual_seed(K + N + R + dual)
    off = torch.tensor([0, R], dtype=torch.int32)
    A = _int_tensor(g, (R, K), -1, 1).to(DEV)
    dC = _int_tensor(g, (R, N), -1, 1).to(DEV)
    dC2 = _int_tensor(g, (R, N), -1, 1).to(DEV) if dual else None
    cnt, ws = moe.dw_counters(DEV), moe.split_workspace(DEV)
    ref = O.grouped_gemm_dw(f64(A), f64(dC), off.numpy())
    ref2 = O.grouped_gemm_dw(f64(A), f64(dC2), off.numpy()) if dual else None
    for _ in range(2):
        dB = poison_(torch.empty((1, K, N), dtype=torch.float32, device=DEV))
        dB2 = poison_(torch.empty((1, K, N), dtype=torch.float32, device=DEV)) if dual else None
        moe.moe_grouped_gemm_dw(A, dC, off.to(DEV), dC2, dB=dB, dB2=dB2, counters=cnt, workspace=ws)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(f64(dB), ref)
        if dual:
            np.testing.assert_array_equal(f64(dB2), ref2)
    # an empty group: exact zeros (nothing to split)
    z = poison_(torch.empty((1, K, N), dtype=torch.float32, device=DEV))
    moe.moe_grouped_gemm_dw(A[:0], dC[:0], torch.zeros(2, dtype=torch.int32, device=DEV), dB=z, counters=cnt,
                            workspace=ws)
    torch.cuda.synchronize()
    assert torch.count_nonzero(z) == 0
    # several groups: no split, bitwise the persistent kernel
    off3 = torch.tensor([0, R // 3, R // 3, R], dtype=torch.int32, device=DEV)
    a, _ = moe.moe_grouped_gemm_dw(A, dC, off3, counters=cnt, workspace=ws)
    b, _ = moe.moe_grouped_gemm_dw(A, dC, off3, counters=cnt)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_grouped_gemm_256_groups_exact():
    """The maximum group count (G = 256, empty groups included) with more row tiles than CUs, so
    the persistent dX kernel walks several tiles per workgroup: every product exact on
    small-integer operands, and the fused dX + SwiGLU backward bitwise equal to the two calls."""
    _say("gemm 256 groups exact")
    rng = np.random.default_rng(256)
    counts = rng.integers(0, 400, 256)
    counts[rng.choice(256, 20, replace=False)] = 0
    G, R = 256, int(counts.sum())
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    offd = off.to(DEV)
    g = torch.Generator().manual_seed(256)
    # fwd: C = A B[g] (K = 64, N = 512), dual with SwiGLU
    A = _int_tensor(g, (R, 64))
    B, B2 = _int_tensor(g, (G, 64, 512)), _int_tensor(g, (G, 64, 512))
    C, C2, act = moe.moe_grouped_gemm_fwd(A.to(DEV), B.to(DEV), offd, B2.to(DEV), want_act=True)
    C1 = moe.moe_grouped_gemm_fwd(A.to(DEV), B.to(DEV), offd)[0]
    torch.cuda.synchronize()
    refC = O.grouped_gemm(f64(A), f64(B), off.numpy())
    np.testing.assert_array_equal(f64(C), refC)
    np.testing.assert_array_equal(f64(C1), refC)
    np.testing.assert_array_equal(f64(C2), O.grouped_gemm(f64(A), f64(B2), off.numpy()))
    # dX: dA = dC B[g]^T (K = 512 output columns, N = 64 contraction), single and dual
    dC, dC2 = _int_tensor(g, (R, 64)), _int_tensor(g, (R, 64))
    Bx, Bx2 = _int_tensor(g, (G, 512, 64)), _int_tensor(g, (G, 512, 64))
    dA = moe.moe_grouped_gemm_dx(dC.to(DEV), Bx.to(DEV), offd)
    dA2 = moe.moe_grouped_gemm_dx(dC.to(DEV), Bx.to(DEV), offd, dC2.to(DEV), Bx2.to(DEV))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(f64(dA), O.grouped_gemm_dx(f64(dC), f64(Bx), off.numpy()))
    np.testing.assert_array_equal(f64(dA2), O.grouped_gemm_dx(f64(dC), f64(Bx), off.numpy(), f64(dC2), f64(Bx2)))
    hg = (torch.randn((R, 512), generator=g) * 2).to(torch.bfloat16).to(DEV)
    hu = torch.randn((R, 512), generator=g).to(torch.bfloat16).to(DEV)
    ref_g, ref_u = moe.moe_swiglu_bwd(hg, hu, dA)
    fg, fu = moe.moe_grouped_gemm_dx_swiglu_bwd(dC.to(DEV), Bx.to(DEV), offd, hg, hu)
    torch.cuda.synchronize()
    assert torch.equal(fg.view(torch.int16), ref_g.view(torch.int16))
    assert torch.equal(fu.view(torch.int16), ref_u.view(torch.int16))
    # dW: dB[g] = A_g^T dC_g (64 x 128 per group), empty groups exactly zero
    dCw = _int_tensor(g, (R, 128), -2, 2)
    dB = moe.moe_grouped_gemm_dw(A.to(DEV), dCw.to(DEV), offd)[0]
    dBt = moe.moe_grouped_gemm_dw_t(moe.moe_transpose_grouped(A.to(DEV), offd),
                                    moe.moe_transpose_grouped(dCw.to(DEV), offd), offd, R)[0]
    torch.cuda.synchronize()
    refw = O.grouped_gemm_dw(f64(A), f64(dCw), off.numpy())
    np.testing.assert_array_equal(f64(dB), refw)
    np.testing.assert_array_equal(f64(dBt), refw)
    for e in np.flatnonzero(counts == 0):
        assert torch.count_nonzero(dB[int(e)]) == 0 and torch.count_nonzero(dBt[int(e)]) == 0


@pytest.mark.parametrize("K,N,counts", [
    (192, 320, GROUPS),
    (1024, 2048, [700, 0, 3000, 1, 255, 257, 4096, 64, 1900, 0, 33, 2500]),   # several tiles per CU
    (256, 128, [0] * 200 + [37] * 40 + [600] * 16),                           # G = 256, mostly empty
])
def test_grouped_gemm_dw_persistent_bitwise(K, N, counts):
    """The persistent dW entry points (tiles handed out through per-XCD claim counters) against
    the one-workgroup-per-tile ones: bit-identical fp32 and bf16 results, single and dual, empty
    groups included, and twice in a row on the same counters (each call resets them)."""
    _say("gemm dw persistent", K, N, len(counts))
    g = torch.Generator(device=DEV).manual_seed(K + N + len(counts))
    G, R = len(counts), sum(counts)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32, device=DEV)
    A = (torch.randn((R, K), generator=g, device=DEV)).to(torch.bfloat16)
    dC = (torch.randn((R, N), generator=g, device=DEV)).to(torch.bfloat16)
    dC2 = (torch.randn((R, N), generator=g, device=DEV)).to(torch.bfloat16)
    cnt = moe.dw_counters(DEV)
    ref1, ref2 = moe.moe_grouped_gemm_dw(A, dC, off, dC2)
    ref_s, _ = moe.moe_grouped_gemm_dw(A, dC, off)
    ref16, ref16b = moe.moe_grouped_gemm_dw_bf16(A, dC, off, dC2)
    for _ in range(2):
        got1, got2 = moe.moe_grouped_gemm_dw(A, dC, off, dC2, dB=poison_(torch.empty_like(ref1)),
                                             dB2=poison_(torch.empty_like(ref2)), counters=cnt)
        got_s, _ = moe.moe_grouped_gemm_dw(A, dC, off, dB=poison_(torch.empty_like(ref_s)), counters=cnt)
        got16, got16b = moe.moe_grouped_gemm_dw_bf16(A, dC, off, dC2, dB=poison_(torch.empty_like(ref16)),
                                                     dB2=poison_(torch.empty_like(ref16b)), counters=cnt)
        torch.cuda.synchronize()
        for name, a, b in (("dB", got1, ref1), ("dB2", got2, ref2), ("dB single", got_s, ref_s),
                           ("dB bf16", got16, ref16), ("dB2 bf16", got16b, ref16b)):
            assert torch.equal(a, b), f"{name}: persistent and one-per-tile results differ"
    empty = [i for i, c in enumerate(counts) if c == 0]
    if empty:
        assert torch.count_nonzero(got1[empty]) == 0 and torch.count_nonzero(got16[empty]) == 0


@pytest.mark.parametrize("K,N", [(320, 192), (256, 256)])
def test_grouped_gemm_dw_bf16_exact(K, N):
    """bf16-output dW: the fp32 sum of small integers is exact, so every output equals the
    round-to-nearest-even of the exact sum (group sums above 256 do round); empty groups zero."""
    _say("gemm_dw_bf16 exact", K, N)
    g = torch.Generator().manual_seed(7 * K + N)
    counts = GROUPS
    G, R = len(counts), sum(counts)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    A = _int_tensor(g, (R, K), -2, 2)
    dC, dC2 = _int_tensor(g, (R, N), -2, 2), _int_tensor(g, (R, N), -2, 2)
    dB, dB2, dB1 = (poison_(torch.empty((G, K, N), dtype=torch.bfloat16, device=DEV)) for _ in range(3))
    moe.moe_grouped_gemm_dw_bf16(A.to(DEV), dC.to(DEV), off.to(DEV), dC2.to(DEV), dB, dB2)
    moe.moe_grouped_gemm_dw_bf16(A.to(DEV), dC.to(DEV), off.to(DEV), dB=dB1)
    torch.cuda.synchronize()
    ref = O.bf16_round(O.grouped_gemm_dw(f64(A), f64(dC), off.numpy()))
    np.testing.assert_array_equal(f64(dB), ref)
    np.testing.assert_array_equal(f64(dB1), ref)
    np.testing.assert_array_equal(f64(dB2), O.bf16_round(O.grouped_gemm_dw(f64(A), f64(dC2), off.numpy())))
    assert torch.count_nonzero(dB[5]) == 0 and torch.count_nonzero(dB2[10]) == 0


def _padded_starts(counts):
    pad = [(c + 31) // 32 * 32 for c in counts]
    return np.concatenate([[0], np.cumsum(pad)]).astype(np.int64)


@pytest.mark.parametrize("C", [64, 320])
def test_transpose_grouped_exact(C):
    """The contraction-major copy: a bit copy of every row into its group's padded segment, zero
    padding up to the next multiple of 32 (and to the end of the last 64-column block)."""
    _say("transpose_grouped", C)
    g = torch.Generator().manual_seed(C)
    counts = GROUPS
    G, R = len(counts), sum(counts)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32)
    src = torch.randn((R, C), generator=g).to(torch.bfloat16)
    ld = moe.transposed_cols(R, G)
    dst = poison_(torch.empty((C, ld), dtype=torch.bfloat16, device=DEV))
    moe.moe_transpose_grouped(src.to(DEV), off.to(DEV), dst=dst)
    torch.cuda.synchronize()
    ps = _padded_starts(counts)
    want = np.zeros((C, int(ps[-1])), dtype=np.int16)
    sb = src.view(torch.int16).numpy()
    o = off.numpy()
    for gi in range(G):
        want[:, ps[gi]:ps[gi] + counts[gi]] = sb[o[gi]:o[gi + 1]].T
    got = dst.view(torch.int16).cpu().numpy()
    np.testing.assert_array_equal(got[:, :ps[-1]], want)
    end = (int(ps[-1]) + 63) // 64 * 64
    assert (got[:, ps[-1]:end] == 0).all()


@pytest.mark.parametrize("K,N", [(192, 320), (256, 256), (576, 64)])
def test_grouped_gemm_dw_t_exact(K, N):
    """dW from contraction-major copies: exact on small-integer operands (fp32 and bf16 outputs,
    single and dual), empty groups zero, and bitwise equal to moe_grouped_gemm_dw on Gaussian
    operands (same per-element reduction order; padding adds exact zeros)."""
    _say("gemm_dw_t exact", K, N)
    g = torch.Generator().manual_seed(100 * K + N + 1)
    counts = GROUPS
    G, R = len(counts), sum(counts)
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32).to(DEV)
    A = _int_tensor(g, (R, K), -2, 2).to(DEV)
    dC, dC2 = _int_tensor(g, (R, N), -2, 2).to(DEV), _int_tensor(g, (R, N), -2, 2).to(DEV)
    At, dCt, dC2t = (moe.moe_transpose_grouped(t, off) for t in (A, dC, dC2))
    dB, dB2 = moe.moe_grouped_gemm_dw_t(At, dCt, off, R, dC2t)
    dB1 = moe.moe_grouped_gemm_dw_t(At, dCt, off, R)[0]
    hB, hB2 = moe.moe_grouped_gemm_dw_t(At, dCt, off, R, dC2t, out_bf16=True)
    torch.cuda.synchronize()
    offn = off.cpu().numpy()
    ref = O.grouped_gemm_dw(f64(A), f64(dC), offn)
    ref2 = O.grouped_gemm_dw(f64(A), f64(dC2), offn)
    np.testing.assert_array_equal(f64(dB), ref)
    np.testing.assert_array_equal(f64(dB1), ref)
    np.testing.assert_array_equal(f64(dB2), ref2)
    np.testing.assert_array_equal(f64(hB), O.bf16_round(ref))
    np.testing.assert_array_equal(f64(hB2), O.bf16_round(ref2))
    assert torch.count_nonzero(dB[5]) == 0 and torch.count_nonzero(dB2[10]) == 0
    # Gaussian operands: bitwise equal to the row-major dW kernel
    Ag = torch.randn((R, K), generator=g).to(torch.bfloat16).to(DEV)
    dCg = torch.randn((R, N), generator=g).to(torch.bfloat16).to(DEV)
    d_rm = moe.moe_grouped_gemm_dw(Ag, dCg, off)[0]
    d_t = moe.moe_grouped_gemm_dw_t(moe.moe_transpose_grouped(Ag, off), moe.moe_transpose_grouped(dCg, off), off, R)[0]
    torch.cuda.synchronize()
    assert torch.equal(d_rm.view(torch.int32), d_t.view(torch.int32))


def _sampled_rows(counts, n, seed):
    """n rows spread over the groups (sorted), with the sub-problem's exclusive offsets."""
    off = np.concatenate([[0], np.cumsum(counts)])
    rows = np.sort(np.random.default_rng(seed).choice(int(off[-1]), size=n, replace=False))
    grp = np.searchsorted(off, rows, side="right") - 1
    sub = np.concatenate([[0], np.cumsum(np.bincount(grp, minlength=len(counts)))])
    return rows, sub


def _int_dev(g, shape):
    return torch.randint(-1, 2, shape, generator=g, device=DEV).to(torch.bfloat16)


def test_grouped_gemm_fwd_split_tail():
    """The forward product with a split workspace, on a shape whose tile count is a few tiles past
    a multiple of the CU count and whose contraction (K = 8192: 256 steps) is long enough to split
    (non-dual 264 tiles, dual 528: the last round's tiles in 4 pieces each).  Small-integer operands
    make every sum exact, so the split results equal the unsplit ones bit for bit (also the fused
    SwiGLU, computed from the same summed tile) and the oracle on sampled rows; Gaussian operands
    give bitwise-repeatable results within tolerance of the unsplit ones."""
    _say("gemm fwd split tail")
    counts = [2048] * 7 + [2400]                      # 66 row tiles
    G, R, K, N = len(counts), sum(counts), 8192, 1024
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32, device=DEV)
    g = torch.Generator(device=DEV).manual_seed(12)
    ws = moe.split_workspace(DEV)
    A, B, B2 = _int_dev(g, (R, K)), _int_dev(g, (G, K, N)), _int_dev(g, (G, K, N))
    c1 = moe.moe_grouped_gemm_fwd(A, B, off)[0]
    s1 = moe.moe_grouped_gemm_fwd(A, B, off, workspace=ws)[0]
    c2 = moe.moe_grouped_gemm_fwd(A, B, off, B2, want_act=True)
    s2 = moe.moe_grouped_gemm_fwd(A, B, off, B2, want_act=True, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(c1.view(torch.int16), s1.view(torch.int16))
    for u, v in zip(c2, s2):
        assert torch.equal(u.view(torch.int16), v.view(torch.int16))
    rows, sub = _sampled_rows(counts, 96, 3)
    ridx = torch.tensor(rows, device=DEV)
    Bf, B2f = f64(B), f64(B2)
    np.testing.assert_array_equal(f64(s1[ridx]), O.grouped_gemm(f64(A[ridx]), Bf, sub))
    np.testing.assert_array_equal(f64(s2[1][ridx]), O.grouped_gemm(f64(A[ridx]), B2f, sub))
    Ag = torch.randn((R, K), generator=g, device=DEV).to(torch.bfloat16)
    Bg = (torch.randn((G, K, N), generator=g, device=DEV) * 0.02).to(torch.bfloat16)
    x1 = moe.moe_grouped_gemm_fwd(Ag, Bg, off, workspace=ws)[0]
    x2 = moe.moe_grouped_gemm_fwd(Ag, Bg, off, workspace=ws)[0]
    x0 = moe.moe_grouped_gemm_fwd(Ag, Bg, off)[0]
    torch.cuda.synchronize()
    assert torch.equal(x1.view(torch.int16), x2.view(torch.int16))
    check_float("C split vs unsplit", f64(x1), f64(x0), 1e-3)
    check_float("C split (sampled rows)", f64(x1[ridx]), O.grouped_gemm(f64(Ag[ridx]), f64(Bg), sub))


def test_grouped_gemm_dx_split_tail():
    """The persistent dX products with a split workspace: a tile count just past a full round
    (131 row tiles x 2 column tiles) and a contraction long enough to split (N = 4096: 128 steps,
    256 in the dual product) -- bitwise equal to the unsplit kernels on small-integer operands and
    equal to the oracle on sampled rows; the fused SwiGLU backward likewise; Gaussian operands
    deterministic and within tolerance."""
    _say("gemm dx split tail")
    counts = [4096] * 7 + [4700]                      # 131 row tiles
    G, R, K, N = len(counts), sum(counts), 512, 4096
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32, device=DEV)
    g = torch.Generator(device=DEV).manual_seed(9)
    ws = moe.split_workspace(DEV)
    dC, dC2 = _int_dev(g, (R, N)), _int_dev(g, (R, N))
    B, B2 = _int_dev(g, (G, K, N)), _int_dev(g, (G, K, N))
    ref_s = moe.moe_grouped_gemm_dx(dC, B, off, dC2, B2)
    got_s = moe.moe_grouped_gemm_dx(dC, B, off, dC2, B2, workspace=ws)
    ref_1 = moe.moe_grouped_gemm_dx(dC, B, off)
    got_1 = moe.moe_grouped_gemm_dx(dC, B, off, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(got_s.view(torch.int16), ref_s.view(torch.int16))
    assert torch.equal(got_1.view(torch.int16), ref_1.view(torch.int16))
    rows, sub = _sampled_rows(counts, 96, 4)
    ridx = torch.tensor(rows, device=DEV)
    np.testing.assert_array_equal(f64(got_s[ridx]), O.grouped_gemm_dx(f64(dC[ridx]), f64(B), sub, f64(dC2[ridx]),
                                                                        f64(B2)))
    np.testing.assert_array_equal(f64(got_1[ridx]), O.grouped_gemm_dx(f64(dC[ridx]), f64(B), sub))
    hg = (torch.randn((R, K), generator=g, device=DEV) * 2).to(torch.bfloat16)
    hu = torch.randn((R, K), generator=g, device=DEV).to(torch.bfloat16)
    a_g, a_u = moe.moe_grouped_gemm_dx_swiglu_bwd(dC, B, off, hg, hu)
    b_g, b_u = moe.moe_grouped_gemm_dx_swiglu_bwd(dC, B, off, hg, hu, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(a_g.view(torch.int16), b_g.view(torch.int16))
    assert torch.equal(a_u.view(torch.int16), b_u.view(torch.int16))
    dCg = torch.randn((R, N), generator=g, device=DEV).to(torch.bfloat16)
    Bg = (torch.randn((G, K, N), generator=g, device=DEV) * 0.05).to(torch.bfloat16)
    x1 = moe.moe_grouped_gemm_dx(dCg, Bg, off, workspace=ws)
    x2 = moe.moe_grouped_gemm_dx(dCg, Bg, off, workspace=ws)
    x0 = moe.moe_grouped_gemm_dx(dCg, Bg, off)
    torch.cuda.synchronize()
    assert torch.equal(x1.view(torch.int16), x2.view(torch.int16))
    check_float("dA split vs unsplit", f64(x1), f64(x0), 1e-3)
    check_float("dA split (sampled rows)", f64(x1[ridx]), O.grouped_gemm_dx(f64(dCg[ridx]), f64(Bg), sub))


# Host replica of the fwd/dX products' dispatch order (blocks round-robin over the 8 XCDs, each XCD
# walking a contiguous logical range in bands of 4 column tiles): used only to check the premise of
# the ragged split-tail tests, i.e. that the last partial round really holds ragged tiles.
def _xcd_remap(bid, n):
    q, r, x, l = n >> 3, n & 7, bid & 7, bid >> 3
    return x * q + (x if x < r else r) + l


def _band_order(i, mt, nt, bw=4):
    full, span = nt // bw, mt * bw
    if i < full * span:
        band, rem = divmod(i, span)
        return rem // bw, band * bw + rem % bw
    rem, w = i - full * span, nt - full * bw
    return rem // w, full * bw + rem % w


def _tail_tile_rows(counts, n_tiles, slots, tm=256):
    """Rows of each tile that the last partial round of `slots` workgroups computes."""
    pre = np.cumsum([(c + tm - 1) // tm for c in counts])
    mtotal = int(pre[-1])
    nall = mtotal * n_tiles
    out = []
    for it in range((nall // slots) * slots, nall):
        m, _ = _band_order(_xcd_remap(it, nall), mtotal, n_tiles)
        g = int(np.sum(pre <= m))
        mt = m - (int(pre[g - 1]) if g else 0)
        out.append(min(tm, counts[g] - mt * tm))
    return out


# groups of 0 to 255 rows, one row tile each (empty groups between them): every tile is ragged,
# the ones of the split round included
_RAGGED = [1, 63, 0, 129, 255, 70, 0, 193, 2, 64, 0, 200, 31, 250, 128, 97]


def _ragged_counts(n_row_tiles, rot=0):
    pat = _RAGGED[rot:] + _RAGGED[:rot]
    c, i = [], 0
    while sum(1 for x in c if x > 0) < n_row_tiles:
        c.append(pat[i % len(pat)])
        i += 1
    return c


def _cu_slots():
    return torch.cuda.get_device_properties(0).multi_processor_count


def test_grouped_gemm_fwd_split_tail_ragged():
    """Split tail over ragged groups: 66 one-tile groups of 1..255 rows with empty groups between
    them (264 tiles, dual 528), so the last partial round splits tiles of 1, 2, 128, 129, 193, 200,
    250 and 255 rows (dual: 1, 2, 250, 255) along K = 8192.  Small-integer operands: bitwise equal
    to the unsplit product and exactly equal to the oracle on every row."""
    _say("gemm fwd split tail, ragged groups")
    counts = _ragged_counts(66)
    slots = _cu_slots()
    G, R, K, N = len(counts), sum(counts), 8192, 1024
    for nt in (N // 256, N // 128):
        tail = _tail_tile_rows(counts, nt, slots)
        assert 0 < len(tail) <= slots // 2 and sum(1 for r in tail if r < 256) >= 3, tail
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32, device=DEV)
    g = torch.Generator(device=DEV).manual_seed(21)
    ws = moe.split_workspace(DEV)
    A, B, B2 = _int_dev(g, (R, K)), _int_dev(g, (G, K, N)), _int_dev(g, (G, K, N))
    c1 = moe.moe_grouped_gemm_fwd(A, B, off)[0]
    s1 = moe.moe_grouped_gemm_fwd(A, B, off, workspace=ws)[0]
    c2 = moe.moe_grouped_gemm_fwd(A, B, off, B2, want_act=True)
    s2 = moe.moe_grouped_gemm_fwd(A, B, off, B2, want_act=True, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(c1.view(torch.int16), s1.view(torch.int16))
    for u, v in zip(c2, s2):
        assert torch.equal(u.view(torch.int16), v.view(torch.int16))
    offn = np.concatenate([[0], np.cumsum(counts)])
    Af = f64(A)
    np.testing.assert_array_equal(f64(s1), O.grouped_gemm(Af, f64(B), offn))
    np.testing.assert_array_equal(f64(s2[0]), O.grouped_gemm(Af, f64(B), offn))
    np.testing.assert_array_equal(f64(s2[1]), O.grouped_gemm(Af, f64(B2), offn))


def test_grouped_gemm_dx_split_tail_ragged():
    """The persistent dX products' split tail over ragged groups: 131 one-tile groups of 1..255
    rows with empty groups between them (262 tiles), so the split round holds tiles of 1, 2, 31,
    97, 129 and 255 rows.  Small-integer operands: the plain and dual products bitwise equal to the
    unsplit kernels and exactly equal to the oracle on every row; the fused SwiGLU backward bitwise
    equal to the unsplit kernel's."""
    _say("gemm dx split tail, ragged groups")
    counts = _ragged_counts(131, rot=12)
    slots = _cu_slots() & ~7
    G, R, K, N = len(counts), sum(counts), 512, 4096
    tail = _tail_tile_rows(counts, K // 256, slots)
    assert 0 < len(tail) <= slots // 2 and sum(1 for r in tail if r < 256) >= 3, tail
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32, device=DEV)
    g = torch.Generator(device=DEV).manual_seed(22)
    ws = moe.split_workspace(DEV)
    dC, dC2 = _int_dev(g, (R, N)), _int_dev(g, (R, N))
    B, B2 = _int_dev(g, (G, K, N)), _int_dev(g, (G, K, N))
    ref_s = moe.moe_grouped_gemm_dx(dC, B, off, dC2, B2)
    got_s = moe.moe_grouped_gemm_dx(dC, B, off, dC2, B2, workspace=ws)
    ref_1 = moe.moe_grouped_gemm_dx(dC, B, off)
    got_1 = moe.moe_grouped_gemm_dx(dC, B, off, workspace=ws)
    hg = (torch.randn((R, K), generator=g, device=DEV) * 2).to(torch.bfloat16)
    hu = torch.randn((R, K), generator=g, device=DEV).to(torch.bfloat16)
    a_g, a_u = moe.moe_grouped_gemm_dx_swiglu_bwd(dC, B, off, hg, hu)
    b_g, b_u = moe.moe_grouped_gemm_dx_swiglu_bwd(dC, B, off, hg, hu, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(got_s.view(torch.int16), ref_s.view(torch.int16))
    assert torch.equal(got_1.view(torch.int16), ref_1.view(torch.int16))
    assert torch.equal(a_g.view(torch.int16), b_g.view(torch.int16))
    assert torch.equal(a_u.view(torch.int16), b_u.view(torch.int16))
    offn = np.concatenate([[0], np.cumsum(counts)])
    np.testing.assert_array_equal(f64(got_s), O.grouped_gemm_dx(f64(dC), f64(B), offn, f64(dC2), f64(B2)))
    np.testing.assert_array_equal(f64(got_1), O.grouped_gemm_dx(f64(dC), f64(B), offn))


def test_grouped_gemm_dw_worked_example():
    """The hand-evaluated dW1 example of Appendix H's definition, zero-padded to 64-multiples."""
    import json, os
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "dw1_worked_example.json")))
    X = torch.zeros((3, 64)); X[:, :2] = torch.tensor(gold["X"])
    Gm = torch.zeros((3, 64)); Gm[:, :3] = torch.tensor(gold["G"])
    off = torch.tensor([0] + gold["cumsum_K"], dtype=torch.int32)
    dB, _ = moe.moe_grouped_gemm_dw(X.to(torch.bfloat16).to(DEV), Gm.to(torch.bfloat16).to(DEV), off.to(DEV))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(dB[:, :2, :3].cpu().numpy(), np.array(gold["dW1"], dtype=np.float32))
    assert torch.count_nonzero(dB[:, 2:, :]) == 0 and torch.count_nonzero(dB[:, :, 3:]) == 0


# ---------------------------------------------------------------------------------------------
# elementwise kernels vs oracle
# ---------------------------------------------------------------------------------------------
def test_swiglu_fwd_bwd():
    g = torch.Generator().manual_seed(5)
    rows, f = 333, 448
    hg = (torch.randn((rows, f), generator=g) * 3).to(torch.bfloat16)
    hu = torch.randn((rows, f), generator=g).to(torch.bfloat16)
    da = torch.randn((rows, f), generator=g).to(torch.bfloat16)
    act = moe.moe_swiglu(hg.to(DEV), hu.to(DEV))
    dhg, dhu = moe.moe_swiglu_bwd(hg.to(DEV), hu.to(DEV), da.to(DEV))
    torch.cuda.synchronize()
    ref_a = O.swiglu(f64(hg), f64(hu))
    rg, ru = O.swiglu_bwd(f64(hg), f64(hu), f64(da))
    check_float("act", f64(act), ref_a)
    check_float("dh_gate", f64(dhg), rg)
    check_float("dh_up", f64(dhu), ru)
    # elementwise: at most one bf16 ulp from the oracle's rounding of the exact value
    for got, ref in ((f64(act), ref_a), (f64(dhg), rg), (f64(dhu), ru)):
        ulp = np.abs(ref) * 2.0 ** -7 + 1e-30
        assert np.all(np.abs(got - ref) <= ulp * 1.01)


# ---------------------------------------------------------------------------------------------
# whole layer, small configs: every tensor vs the oracle
# ---------------------------------------------------------------------------------------------
def _layer_parity(cfg, seed=0, expert_bias=None, log=None, fuse=True, dw_t=False, split=True):
    inp = W.make_inputs(cfg, seed, "cpu", expert_bias=expert_bias)
    dinp = {k_: v.to(DEV) for k_, v in inp.items()}
    lay = L.MoELayer(cfg, dinp, fuse_swiglu_bwd=fuse, dw_transposed=dw_t, split_tail=split)
    for t in lay.buf.values():
        if t.dtype != torch.uint8:
            poison_(t)
    lay.step()
    torch.cuda.synchronize()
    b = lay.buf
    np_ = {k_: f64(v) for k_, v in inp.items()}
    shared = None
    if cfg.f_shared:
        shared = (np_["w_gate_sh"], np_["w_up_sh"], np_["w_down_sh"])
    fwd = O.layer_forward(np_["x"], inp["logits"].numpy(), np_["w_gate"], np_["w_up"], np_["w_down"], cfg.k,
                          shared=shared)
    bwd = O.layer_backward(fwd, np_["x"], np_["dy"], np_["w_gate"], np_["w_up"], np_["w_down"], shared=shared)
    for key in ("topk_idx", "offsets", "row_of_slot", "token_of_row"):
        np.testing.assert_array_equal(i64(b[key]), fwd[key])
    np.testing.assert_array_equal(f64(b["x_perm"]), fwd["x_perm"])
    check_float("topk_w", f64(b["topk_w"]), fwd["topk_w"], 1e-5, log)
    for key in ("h_gate", "h_up", "act", "y_perm", "y"):
        check_float(key, f64(b[key]), fwd[key], log=log)
    for key in ("dy_perm", "d_topk_w", "dw_down", "dh_gate", "dh_up", "dx_perm", "dw_gate", "dw_up", "dx"):
        check_float(key, f64(b[key]), bwd[key], log=log)
    if not fuse:
        check_float("d_act", f64(b["d_act"]), bwd["d_act"], log=log)
    if cfg.f_shared:
        for key in ("h_gate", "h_up", "act", "y"):
            check_float(key + "_sh", f64(b[key + "_sh" if key != "y" else "y_sh"]), fwd["shared"][key], log=log)
        for key in ("dw_gate", "dw_up", "dw_down"):
            check_float(key + "_sh", f64(b[key + "_sh"])[0], bwd["shared"][key], log=log)
        check_float("dx_sh", f64(b["dx_sh"]), bwd["shared"]["dx"], log=log)
        for key in ("dh_gate", "dh_up"):
            check_float(key + "_sh", f64(b[key + "_sh"]), bwd["shared"][key], log=log)
    return lay


@pytest.mark.parametrize("fuse", [True, False], ids=["fused_swiglu_bwd", "unfused"])
def test_layer_config0_parity(fuse):
    _say("layer parity cfg0", "fused" if fuse else "unfused")
    log = {}
    _layer_parity(W.CONFIGS[0], log=log, fuse=fuse)
    _say({k_: f"{v:.2e}" for k_, v in log.items()})


@pytest.mark.parametrize("cfg_id", [1, 3])
def test_layer_split_tail_consistent(cfg_id):
    """The layer with the split tail (the default) against the same layer without it, at full size:
    config 1 splits all four fwd/dX products (each a few tiles past a full round, with 128-896
    contraction steps), config 3 its dX gate/up.  Integer outputs equal, floating outputs within
    1e-3 (a split tile groups its fp32 sum differently: last-place bf16 differences), and the
    unsplit products' outputs bitwise equal where nothing upstream was split.  The split path's
    oracle parity at full size is the full-size layer test (which runs the default)."""
    cfg = W.CONFIGS[cfg_id]
    _say("layer split tail vs unsplit", cfg)
    inp = W.make_inputs(cfg, 0, DEV)
    lay_s = L.MoELayer(cfg, inp)
    lay_u = L.MoELayer(cfg, inp, split_tail=False)
    lay_s.step()
    lay_u.step()
    torch.cuda.synchronize()
    for key, t in lay_u.buf.items():
        if key in ("workspace", "d_act", "d_act_sh"):   # scratch, and dA (not stored when fused)
            continue
        u = lay_s.buf[key]
        if not t.dtype.is_floating_point:
            assert torch.equal(t, u), key
        else:
            check_float(key + " split vs unsplit", f64(u), f64(t), 1e-3)


@pytest.mark.parametrize("cfg_id", [0, 2, 3])
def test_layer_dw_transposed(cfg_id):
    """The layer with its weight gradients computed from contraction-major copies: oracle parity,
    and every dW bitwise equal to the row-major path's on the same inputs.  Configs 2 and 3 run
    at 512 tokens (their shapes otherwise)."""
    import dataclasses
    cfg = W.CONFIGS[cfg_id]
    if cfg_id:
        cfg = dataclasses.replace(cfg, T=512)
    _say("layer dw transposed", cfg)
    lay_t = _layer_parity(cfg, dw_t=True)
    inp = W.make_inputs(cfg, 0, "cpu")
    lay = L.MoELayer(cfg, {k_: v.to(DEV) for k_, v in inp.items()})
    lay.step()
    torch.cuda.synchronize()
    for key in ("dw_gate", "dw_up", "dw_down"):
        assert torch.equal(lay.buf[key].view(torch.int32), lay_t.buf[key].view(torch.int32)), key


@pytest.mark.parametrize("T,d,E,k,N", [(300, 256, 8, 2, 320), (1000, 512, 16, 4, 256), (64, 64, 4, 1, 64)])
def test_grouped_gemm_fwd_gather(T, d, E, k, N):
    """The gate/up product reading its rows through token_of_row equals the product on the
    gathered X_perm bit for bit (single, dual, dual + SwiGLU; with and without a split
    workspace), and equals the oracle exactly on small-integer operands; moe_gather_rows equals
    the oracle's gather bit for bit."""
    _say("gemm fwd gather", T, d, E, k, N)
    g = torch.Generator().manual_seed(T + d)
    logits = torch.randn((T, E), generator=g)
    x = _int_tensor(g, (T, d)).to(DEV)
    B, B2 = _int_tensor(g, (E, d, N)).to(DEV), _int_tensor(g, (E, d, N)).to(DEV)
    r = moe.moe_route_permute(logits.to(DEV), x, k)
    xg = poison_(torch.empty((T * k, d), dtype=torch.bfloat16, device=DEV))
    moe.moe_gather_rows(x, r["row_of_slot"], k, xg)
    torch.cuda.synchronize()
    tor = i64(r["token_of_row"])
    np.testing.assert_array_equal(f64(xg), f64(x)[tor])
    assert torch.equal(xg.view(torch.int16), r["x_perm"].view(torch.int16))
    off = r["offsets"]
    ws = moe.split_workspace(DEV)
    for w in (None, ws):
        a1 = moe.moe_grouped_gemm_fwd(r["x_perm"], B, off)[0]
        b1 = moe.moe_grouped_gemm_fwd_gather(x, r["token_of_row"], B, off, workspace=w)[0]
        a3 = moe.moe_grouped_gemm_fwd(r["x_perm"], B, off, B2, want_act=True)
        b3 = moe.moe_grouped_gemm_fwd_gather(x, r["token_of_row"], B, off, B2, want_act=True, workspace=w)
        torch.cuda.synchronize()
        assert torch.equal(a1.view(torch.int16), b1.view(torch.int16))
        for u, v in zip(a3, b3):
            assert torch.equal(u.view(torch.int16), v.view(torch.int16))
    np.testing.assert_array_equal(f64(b1), O.grouped_gemm(f64(x)[tor], f64(B), i64(off)))


@pytest.mark.parametrize("cfg_id", [0, 2])
def test_layer_gather_fused_bitwise(cfg_id):
    """The layer with the gather folded into the gate/up product gives bitwise the outputs of the
    default layer (X_perm, gathered in the backward instead, included), over two steps."""
    import dataclasses
    cfg = W.CONFIGS[cfg_id]
    if cfg_id:
        cfg = dataclasses.replace(cfg, T=1024)
    _say("layer gather fused", cfg)
    inp = W.make_inputs(cfg, 0, "cpu")
    dinp = {k_: v.to(DEV) for k_, v in inp.items()}
    ref = L.MoELayer(cfg, dinp)
    gat = L.MoELayer(cfg, dinp, gather_fused=True)
    ref.step()
    for _ in range(2):
        for t in gat.buf.values():
            poison_(t)
        gat.step()
    torch.cuda.synchronize()
    for key, t in ref.buf.items():
        if key in ("workspace", "d_act", "d_act_sh"):
            continue
        assert torch.equal(t.view(torch.uint8), gat.buf[key].view(torch.uint8)), key


def _routing(g, T, E, k):
    """Seeded top-k choices over distinct experts and the stable expert-ordered packing they imply
    (built here with torch sorting: offsets, row_of_slot, token_of_row)."""
    idx = torch.stack([torch.randperm(E, generator=g)[:k] for _ in range(T)])
    flat = idx.reshape(-1)
    order = torch.sort(flat, stable=True).indices
    row_of_slot = torch.empty(T * k, dtype=torch.int64)
    row_of_slot[order] = torch.arange(T * k)
    off = torch.zeros(E + 1, dtype=torch.int64)
    off[1:] = torch.cumsum(torch.bincount(flat, minlength=E), 0)
    return off.to(torch.int32), row_of_slot.to(torch.int32), (order // k).to(torch.int32)


@pytest.mark.parametrize("k,N,shared,split", [(2, 320, False, False), (2, 512, True, True), (1, 256, False, True),
                                              (4, 192, True, False), (6, 128, False, True), (8, 64, True, True)])
def test_grouped_gemm_fwd_combine_exact(k, N, shared, split):
    """The down product with the weighted combine fused into its epilogue, on small integers with
    power-of-two routing weights (every sum exact): Y_perm and Y exact against the oracle's product
    and combine, for every k the combine specialises and a general one, with and without the shared
    output, with and without the split tail, several column tiles (N = 320: a partial one); called
    twice (the arrival counters are re-zeroed by each call)."""
    _say("fwd combine exact", k, N, shared, split)
    g = torch.Generator().manual_seed(77 * k + N)
    T, E, K = 300, 8, 192
    R = T * k
    off, ros, tor = _routing(g, T, E, k)
    a = _int_tensor(g, (R, K))
    b = _int_tensor(g, (E, K, N))
    w = (2.0 ** torch.randint(-2, 2, (T, k), generator=g)).to(torch.float32)
    add = _int_tensor(g, (T, N), -8, 8) if shared else None
    ref_perm = O.grouped_gemm(f64(a), f64(b), i64(off))
    ref_y = O.combine(ref_perm, f64(w), i64(ros), k, add=None if add is None else f64(add))
    dv = lambda t: None if t is None else t.to(DEV)
    ws = moe.split_workspace(DEV) if split else None
    cnt = moe.combine_counters(T, N, DEV)
    for _ in range(2):
        yp = poison_(torch.empty((R, N), dtype=torch.bfloat16, device=DEV))
        y = poison_(torch.empty((T, N), dtype=torch.bfloat16, device=DEV))
        moe.moe_grouped_gemm_fwd_combine(dv(a), dv(b), dv(off), dv(w), dv(ros), dv(tor), add=dv(add), y_perm=yp,
                                         y=y, counters=cnt, workspace=ws)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(f64(yp), ref_perm)
        np.testing.assert_array_equal(f64(y), ref_y)


@pytest.mark.parametrize("cfg_id", [0, 2])
def test_layer_combine_fused_bitwise(cfg_id):
    """The layer with the combine fused into the down product gives bitwise the outputs of the
    default layer (Y, Y_perm and everything the backward derives from them), over two steps."""
    import dataclasses
    cfg = W.CONFIGS[cfg_id]
    if cfg_id:
        cfg = dataclasses.replace(cfg, T=1024)
    _say("layer combine fused", cfg)
    inp = W.make_inputs(cfg, 0, "cpu")
    dinp = {k_: v.to(DEV) for k_, v in inp.items()}
    ref = L.MoELayer(cfg, dinp)
    fus = L.MoELayer(cfg, dinp, combine_fused=True)
    ref.step()
    for _ in range(2):
        for t in fus.buf.values():
            poison_(t)
        fus.step()
    torch.cuda.synchronize()
    for key, t in ref.buf.items():
        if key in ("workspace", "d_act", "d_act_sh"):
            continue
        assert torch.equal(t.view(torch.uint8), fus.buf[key].view(torch.uint8)), key


@pytest.mark.parametrize("cfg_id", [0, 2])
def test_layer_concurrent_bitwise(cfg_id):
    """The two-stream schedule (weight gradients and the shared FFN beside the main chain) gives
    bitwise the same outputs as one stream: every kernel is deterministic and the joins order
    every dependency.  Two steps in a row (the second reuses every buffer)."""
    import dataclasses
    cfg = W.CONFIGS[cfg_id]
    if cfg_id:
        cfg = dataclasses.replace(cfg, T=1024)
    _say("layer concurrent", cfg)
    inp = W.make_inputs(cfg, 0, "cpu")
    dinp = {k_: v.to(DEV) for k_, v in inp.items()}
    seq = L.MoELayer(cfg, dinp)
    con = L.MoELayer(cfg, dinp, concurrent=True)
    seq.step()
    for _ in range(2):
        for t in con.buf.values():
            poison_(t)
        con.step()
    torch.cuda.synchronize()
    for key, t in seq.buf.items():
        if key in ("workspace", "d_act", "d_act_sh"):
            continue
        u = con.buf[key]
        assert torch.equal(t.view(torch.uint8), u.view(torch.uint8)), key


def test_dx_swiglu_bwd_fusion_bitwise():
    """The fused dX+SwiGLU-backward epilogue equals moe_grouped_gemm_dx then moe_swiglu_bwd bit for
    bit (same rounding of dA, same elementwise arithmetic), on ragged groups spanning tiles."""
    g = torch.Generator().manual_seed(21)
    counts = GROUPS
    G, R = len(counts), sum(counts)
    K, N = 320, 192
    off = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32).to(DEV)
    dC = torch.randn((R, N), generator=g).to(torch.bfloat16).to(DEV)
    B = (torch.randn((G, K, N), generator=g) * 0.1).to(torch.bfloat16).to(DEV)
    hg = (torch.randn((R, K), generator=g) * 2).to(torch.bfloat16).to(DEV)
    hu = torch.randn((R, K), generator=g).to(torch.bfloat16).to(DEV)
    dA = moe.moe_grouped_gemm_dx(dC, B, off)
    ref_g, ref_u = moe.moe_swiglu_bwd(hg, hu, dA)
    fg, fu = (poison_(torch.empty((R, K), dtype=torch.bfloat16, device=DEV)) for _ in range(2))
    moe.moe_grouped_gemm_dx_swiglu_bwd(dC, B, off, hg, hu, fg, fu)
    torch.cuda.synchronize()
    assert torch.equal(fg.view(torch.int16), ref_g.view(torch.int16))
    assert torch.equal(fu.view(torch.int16), ref_u.view(torch.int16))
    og, ou = O.swiglu_bwd(f64(hg), f64(hu), O.grouped_gemm_dx(f64(dC), f64(B), off.cpu().numpy()))
    check_float("dh_gate", f64(fg), og)
    check_float("dh_up", f64(fu), ou)


@pytest.mark.parametrize("name,cfg,bias", [
    ("single_expert", W.custom(T=200, d=128, f=192, E=1, k=1), None),
    ("fine_grained_shared_small", W.custom(T=512, d=256, f=192, E=64, k=6, f_shared=384), None),
    ("zipf_small", W.custom(T=1024, d=256, f=256, E=32, k=4, zipf_s=1.2, zipf_beta=1.5), None),
    ("forced_empty", W.custom(T=300, d=192, f=320, E=8, k=2), [0, -1e4, 0, 0, -1e4, 0, 0, 0]),
    ("k_equals_E", W.custom(T=130, d=128, f=128, E=4, k=4), None),
])
def test_layer_small_parity(name, cfg, bias):
    _say("layer parity", name)
    _layer_parity(cfg, seed=1, expert_bias=bias)


def test_layer_deterministic():
    cfg = W.custom(T=600, d=256, f=320, E=16, k=3, f_shared=128)
    inp = {k_: v.to(DEV) for k_, v in W.make_inputs(cfg, 2, "cpu").items()}
    lay = L.MoELayer(cfg, inp)
    snaps = []
    for _ in range(3):
        lay.step()
        torch.cuda.synchronize()
        snaps.append({k_: v.clone() for k_, v in lay.buf.items() if k_ != "workspace"})
    for key in snaps[0]:
        for s in snaps[1:]:
            assert torch.equal(snaps[0][key].view(torch.uint8) if snaps[0][key].dtype == torch.bfloat16 else snaps[0][key],
                               s[key].view(torch.uint8) if s[key].dtype == torch.bfloat16 else s[key]), key
