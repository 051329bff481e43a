"""CPU oracle of the MoE expert-FFN training layer (forward and backward).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the benchmark's CPU-baseline
leg import this module.  The library's compute path never calls it, and the two share no code:
this file uses numpy alone.

Arithmetic is float64.  A value that the layer stores as a bf16 tensor (H_gate, H_up, the SwiGLU
output, Y_perm, Y, dY_perm, dA, dH_gate, dH_up, dX_perm, dX) is rounded to bf16 with
round-to-nearest-even exactly where it is stored, by `bf16_round`; every other value (softmax
weights, d_topk_w, the weight gradients) stays float64.  Every function takes `rnd`, the rounding
applied at those stores: `bf16_round` by default, `None` for exact float64 math (used to pin the
backward against automatic differentiation).

What the paper defines.  The paper (section 5.4 and Appendix H, "What the kernel computes")
defines one step of this layer: routed tokens are packed into one buffer ordered by expert, the
per-expert row counts are given as a cumulative sum, and for every expert the weight gradient of
the first FFN projection is dW1_e = X_e^T G_e, a contraction over that expert's K_e rows (K_e may
be zero).  `grouped_gemm_dw` is that definition.  The paper states no routing rule, row order,
activation, combine, router or other backward formula; the readings used for those are the
standard MoE layer (and, for the router's load-balancing loss, the Switch-style auxiliary loss) and
are named at each function.  The FP8 and MX functions at the end serve variants the paper does not
describe (OCP E4M3 operands with fp32 scales, or with a power-of-two scale per 32 elements); their
reading is stated there.

Parity: every function here is pinned by the CPU test suite against closed forms, library
routines, brute force, hand-worked values or automatic differentiation, and the suite plants
plausible mistakes in each to show that a pin catches them.  That includes `rel_fro`, the
comparison metric every floating-point parity check uses (pinned on hand-computed ratios and its
zero-reference conventions).  No function is "parity unpinned".
"""
from __future__ import annotations

import numpy as np

BF16_MAX = float.fromhex("0x1.fe00000000000p+127")


# --------------------------------------------------------------------------------------------
# bf16 storage
# --------------------------------------------------------------------------------------------
def bf16_round(x):
    """Round float64 values to the nearest bfloat16 value, ties to even.

    bfloat16 keeps 8 significant bits and float32's exponent range.  With x = m * 2**e and
    0.5 <= |m| < 1, the spacing of bf16 values around x is 2**(e - 8); below the normal range
    (|x| < 2**-126) the spacing stays 2**-133.  Results beyond the largest finite bf16 become inf.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    e = np.maximum(e, -125)
    q = np.ldexp(np.rint(np.ldexp(x, 8 - e)), e - 8)
    big = np.abs(q) > BF16_MAX
    if np.any(big):
        q = np.where(big, np.copysign(np.inf, q), q)
    return q


def _r(rnd, x):
    return x if rnd is None else rnd(x)


def bf16_bits_to_f64(bits):
    """uint16 bf16 bit patterns -> float64 values (exact)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x):
    """float64 values that are already bf16-representable -> uint16 bit patterns."""
    bits = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32)).view(np.uint32)
    if np.any(bits & 0xFFFF):
        raise ValueError("value is not representable in bf16")
    return (bits >> 16).astype(np.uint16)


# --------------------------------------------------------------------------------------------
# A1: routing
# --------------------------------------------------------------------------------------------
def route_topk(logits, k, normalize=True):
    """Top-k routing on router logits [T, E] (section 5.4 names top-k routing; the rule is not
    stated).  Reading: the k experts with the largest logits, ordered by descending logit with
    ties going to the lower expert id; weights are the softmax over the k selected logits
    (normalize=True), or the softmax probability over all E experts (normalize=False).

    Returns topk_idx [T, k] int64 and topk_w [T, k] float64.
    """
    L = np.asarray(logits, dtype=np.float64)
    T, E = L.shape
    if not 1 <= k <= E:
        raise ValueError("need 1 <= k <= E")
    ids = np.broadcast_to(np.arange(E), (T, E))
    order = np.lexsort((ids, -L), axis=-1)          # primary: -logit ascending, then id
    idx = order[:, :k]
    sel = np.take_along_axis(L, idx, axis=1)
    if normalize:
        ex = np.exp(sel - sel[:, :1])
        w = ex / ex.sum(axis=1, keepdims=True)
    else:
        M = L.max(axis=1, keepdims=True)
        w = np.exp(sel - M) / np.exp(L - M).sum(axis=1, keepdims=True)
    return idx.astype(np.int64), w


# --------------------------------------------------------------------------------------------
# A2-A4: grouping, permutation, gather
# --------------------------------------------------------------------------------------------
def permute(topk_idx, E):
    """Pack the T*k routed slots into one buffer ordered by expert (Appendix H: one contiguous
    buffer ordered by expert, per-expert row counts as a cumulative sum).

    Slot s = t*k + j is token t's j-th choice.  Reading for the order inside a group (the paper
    leaves it open): a stable counting sort, i.e. slots keep their slot order, so rows of one
    group hold ascending token ids.

    Returns offsets [E+1] (exclusive prefix sum of the per-expert counts, offsets[e+1] equals the
    paper's cumsum_K[e]), row_of_slot [T*k] and token_of_row [T*k], all int64.
    """
    idx = np.asarray(topk_idx)
    T, k = idx.shape
    flat = idx.reshape(-1)
    counts = np.bincount(flat, minlength=E)
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    order = np.argsort(flat, kind="stable")          # order[row] = slot stored at that row
    row_of_slot = np.empty(T * k, dtype=np.int64)
    row_of_slot[order] = np.arange(T * k)
    token_of_row = order // k
    return offsets, row_of_slot, token_of_row


def gather(x, token_of_row):
    """X_perm[r] = X[token_of_row[r]] (a copy; values unchanged)."""
    return np.asarray(x)[np.asarray(token_of_row)]


# --------------------------------------------------------------------------------------------
# B, D, G, J: grouped GEMMs over ragged row groups
# --------------------------------------------------------------------------------------------
def grouped_gemm(A, B, offsets, rnd=bf16_round):
    """C[r, :] = A[r, :] @ B[g] for offsets[g] <= r < offsets[g+1]; A [R, K], B [G, K, N]."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    G, K, N = B.shape
    C = np.zeros((A.shape[0], N))
    for g in range(G):
        lo, hi = int(offsets[g]), int(offsets[g + 1])
        if hi > lo:
            C[lo:hi] = A[lo:hi] @ B[g]
    return _r(rnd, C)


def grouped_gemm_dx(dC, B, offsets, dC2=None, B2=None, rnd=bf16_round):
    """dA[r, :] = dC[r, :] @ B[g]^T (+ dC2[r, :] @ B2[g]^T), one sum before rounding.

    Gradient of grouped_gemm with respect to its row operand; B [G, K, N], dC [R, N] -> [R, K].
    """
    dC = np.asarray(dC, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    G, K, N = B.shape
    out = np.zeros((dC.shape[0], K))
    for g in range(G):
        lo, hi = int(offsets[g]), int(offsets[g + 1])
        if hi > lo:
            out[lo:hi] = dC[lo:hi] @ B[g].T
            if dC2 is not None:
                out[lo:hi] += np.asarray(dC2[lo:hi], dtype=np.float64) @ np.asarray(B2[g], dtype=np.float64).T
    return _r(rnd, out)


def grouped_gemm_dw(A, dC, offsets, G=None):
    """dB[g] = A_g^T @ dC_g over the rows of group g: the paper's dW1_e = X_e^T G_e (section 5.4,
    Appendix H), a contraction over a ragged number K_g of rows.  An empty group (K_g = 0) gives
    an all-zero [K, N] block.  A [R, K], dC [R, N] -> [G, K, N], not rounded (float32 on the GPU).
    """
    A = np.asarray(A, dtype=np.float64)
    dC = np.asarray(dC, dtype=np.float64)
    if G is None:
        G = len(offsets) - 1
    out = np.zeros((G, A.shape[1], dC.shape[1]))
    for g in range(G):
        lo, hi = int(offsets[g]), int(offsets[g + 1])
        if hi > lo:
            out[g] = A[lo:hi].T @ dC[lo:hi]
    return out


# --------------------------------------------------------------------------------------------
# C, I: SwiGLU
# --------------------------------------------------------------------------------------------
def sigmoid(x):
    """1 / (1 + exp(-x)), evaluated without overflow: for x < 0 as exp(x) / (1 + exp(x))."""
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def swiglu(h_gate, h_up, rnd=bf16_round):
    """act = silu(g) * u with silu(g) = g * sigmoid(g), from the stored gate/up values.
    (Reading: plain SwiGLU, no bias, clamp or scale; the paper does not state the activation.)"""
    g = np.asarray(h_gate, dtype=np.float64)
    u = np.asarray(h_up, dtype=np.float64)
    return _r(rnd, g * sigmoid(g) * u)


def swiglu_bwd(h_gate, h_up, d_act, rnd=bf16_round):
    """Derivative of swiglu: d/du = silu(g); d/dg = u * s * (1 + g * (1 - s)), s = sigmoid(g).
    Returns (dh_gate, dh_up)."""
    g = np.asarray(h_gate, dtype=np.float64)
    u = np.asarray(h_up, dtype=np.float64)
    da = np.asarray(d_act, dtype=np.float64)
    s = sigmoid(g)
    dh_up = da * g * s
    dh_gate = da * u * s * (1.0 + g * (1.0 - s))
    return _r(rnd, dh_gate), _r(rnd, dh_up)


# --------------------------------------------------------------------------------------------
# E, F, L: combine and its backward
# --------------------------------------------------------------------------------------------
def combine(y_perm, topk_w, row_of_slot, k, add=None, rnd=bf16_round):
    """Y[t] = sum_j w[t, j] * Y_perm[row_of_slot[t*k + j]] (+ add[t]), summed over j = 0..k-1 and
    then add, rounded once.  topk_w = None means weight 1 (the unpermute-sum of dX_perm)."""
    y_perm = np.asarray(y_perm, dtype=np.float64)
    rows = np.asarray(row_of_slot).reshape(-1, k)
    T = rows.shape[0]
    acc = np.zeros((T, y_perm.shape[1]))
    for j in range(k):
        term = y_perm[rows[:, j]]
        if topk_w is not None:
            term = np.asarray(topk_w, dtype=np.float64)[:, j:j + 1] * term
        acc += term
    if add is not None:
        acc += np.asarray(add, dtype=np.float64)
    return _r(rnd, acc)


def combine_bwd(dy, topk_w, row_of_slot, y_perm, k, rnd=bf16_round):
    """Backward of the weighted combine.  Reading: the routing weight is applied while permuting
    dY, so dY_perm[row_of_slot[t*k+j]] = w[t, j] * dY[t]; the weight gradient is
    d_topk_w[t, j] = <dY[t], Y_perm[row_of_slot[t*k+j]]>.  Returns (dy_perm [R, d], d_topk_w [T, k]).
    """
    dy = np.asarray(dy, dtype=np.float64)
    rows = np.asarray(row_of_slot).reshape(-1, k)
    T, d = dy.shape
    dy_perm = np.zeros((T * k, d))
    d_w = np.zeros((T, k))
    for j in range(k):
        w = 1.0 if topk_w is None else np.asarray(topk_w, dtype=np.float64)[:, j:j + 1]
        dy_perm[rows[:, j]] = w * dy
        if y_perm is not None:
            d_w[:, j] = (dy * np.asarray(y_perm, dtype=np.float64)[rows[:, j]]).sum(axis=1)
    return _r(rnd, dy_perm), d_w


# --------------------------------------------------------------------------------------------
# Router: logits, the backward through the routing weights, the load-balancing loss
# --------------------------------------------------------------------------------------------
def router_logits(x, wr, bias=None):
    """Router logits [T, E] = x [T, d] . Wr [d, E] (+ a per-expert bias).  The paper names top-k
    routing (section 5.4) but not the router; reading: one linear map of the token, computed in
    float32 by the layer (exactly here)."""
    L = np.asarray(x, dtype=np.float64) @ np.asarray(wr, dtype=np.float64)
    if bias is not None:
        L = L + np.asarray(bias, dtype=np.float64)
    return L


def route_topk_bwd(logits, topk_idx, d_topk_w, normalize=True):
    """Gradient of the routing weights with respect to the logits (the selection itself is
    piecewise constant and passes no gradient).  With p the probabilities the weights are read
    from (the softmax over the k selected logits when normalize, zero elsewhere; else the softmax
    over all E) and G[t, e] = d_topk_w[t, j] where e = topk_idx[t, j] (0 for unselected e):
        dlogits[t, e] = p[t, e] * (G[t, e] - sum_j d_topk_w[t, j] * p[t, topk_idx[t, j]]).
    Returns dlogits [T, E] float64."""
    L = np.asarray(logits, dtype=np.float64)
    idx = np.asarray(topk_idx)
    g = np.asarray(d_topk_w, dtype=np.float64)
    T, E = L.shape
    if normalize:
        sel = np.take_along_axis(L, idx, axis=1)
        ex = np.exp(sel - sel.max(axis=1, keepdims=True))
        p = np.zeros((T, E))
        np.put_along_axis(p, idx, ex / ex.sum(axis=1, keepdims=True), axis=1)
    else:
        ex = np.exp(L - L.max(axis=1, keepdims=True))
        p = ex / ex.sum(axis=1, keepdims=True)
    G = np.zeros((T, E))
    np.put_along_axis(G, idx, g, axis=1)
    s = (g * np.take_along_axis(p, idx, axis=1)).sum(axis=1, keepdims=True)
    return p * (G - s)


def aux_loss(logits, counts, k, alpha):
    """Load-balancing loss of Switch-style MoE training (not in the paper; a standard companion
    of top-k routing): L = alpha * E * sum_e f_e * P_e with f_e = counts[e] / (T * k), the share
    of routed slots expert e received (held constant: counts are not differentiable), and P_e the
    mean over tokens of the full softmax probability of e.  Returns (L, dL/dlogits [T, E]):
        dL/dlogits[t, e] = alpha * E / T * p[t, e] * (f_e - sum_e' f_e' * p[t, e'])."""
    L = np.asarray(logits, dtype=np.float64)
    T, E = L.shape
    ex = np.exp(L - L.max(axis=1, keepdims=True))
    p = ex / ex.sum(axis=1, keepdims=True)
    f = np.asarray(counts, dtype=np.float64) / (T * k)
    loss = alpha * E * float((f * p.mean(axis=0)).sum())
    grad = alpha * E / T * p * (f[None, :] - (p * f[None, :]).sum(axis=1, keepdims=True))
    return loss, grad


def router_bwd(x, wr, dlogits, dx=None, rnd=bf16_round):
    """Backward of the router map: dWr [d, E] = x^T . dlogits (float64), and the router's share
    of the token gradient, dlogits . Wr^T [T, d].  Reading: the router runs after the experts'
    unpermute-sum has stored dX in bf16, so its share is added to that stored value and rounded
    once more: returns (dWr, rnd(dx + dlogits . Wr^T)) (dx = None: the share alone, rounded)."""
    x = np.asarray(x, dtype=np.float64)
    g = np.asarray(dlogits, dtype=np.float64)
    wr = np.asarray(wr, dtype=np.float64)
    share = g @ wr.T
    if dx is not None:
        share = np.asarray(dx, dtype=np.float64) + share
    return x.T @ g, _r(rnd, share)


# --------------------------------------------------------------------------------------------
# The whole layer
# --------------------------------------------------------------------------------------------
def dense_ffn_forward(x, w_gate, w_up, w_down, rnd=bf16_round):
    """An always-on (shared) SwiGLU FFN: the grouped path with one group holding every row."""
    T = np.asarray(x).shape[0]
    off = np.array([0, T])
    hg = grouped_gemm(x, np.asarray(w_gate)[None], off, rnd)
    hu = grouped_gemm(x, np.asarray(w_up)[None], off, rnd)
    a = swiglu(hg, hu, rnd)
    y = grouped_gemm(a, np.asarray(w_down)[None], off, rnd)
    return {"h_gate": hg, "h_up": hu, "act": a, "y": y}


def dense_ffn_backward(fwd, x, dy, w_gate, w_up, w_down, rnd=bf16_round):
    T = np.asarray(x).shape[0]
    off = np.array([0, T])
    da = grouped_gemm_dx(dy, np.asarray(w_down)[None], off, rnd=rnd)
    dwd = grouped_gemm_dw(fwd["act"], dy, off)[0]
    dhg, dhu = swiglu_bwd(fwd["h_gate"], fwd["h_up"], da, rnd)
    dx = grouped_gemm_dx(dhg, np.asarray(w_gate)[None], off, dhu, np.asarray(w_up)[None], rnd)
    dwg = grouped_gemm_dw(x, dhg, off)[0]
    dwu = grouped_gemm_dw(x, dhu, off)[0]
    return {"d_act": da, "dh_gate": dhg, "dh_up": dhu, "dx": dx,
            "dw_gate": dwg, "dw_up": dwu, "dw_down": dwd}


def layer_forward(x, logits, w_gate, w_up, w_down, k, shared=None, normalize=True,
                  rnd=bf16_round):
    """Forward of the MoE expert-FFN layer.  `shared` = (w_gate_sh, w_up_sh, w_down_sh) or None.

    route -> permute -> gather -> gate/up grouped GEMMs -> SwiGLU -> down grouped GEMM ->
    weighted combine (+ shared FFN output).
    """
    E = np.asarray(w_gate).shape[0]
    idx, w = route_topk(logits, k, normalize)
    offsets, row_of_slot, token_of_row = permute(idx, E)
    x_perm = gather(x, token_of_row)
    hg = grouped_gemm(x_perm, w_gate, offsets, rnd)
    hu = grouped_gemm(x_perm, w_up, offsets, rnd)
    a = swiglu(hg, hu, rnd)
    y_perm = grouped_gemm(a, w_down, offsets, rnd)
    out = {"topk_idx": idx, "topk_w": w, "offsets": offsets, "row_of_slot": row_of_slot,
           "token_of_row": token_of_row, "x_perm": x_perm, "h_gate": hg, "h_up": hu, "act": a,
           "y_perm": y_perm, "k": k}
    y_sh = None
    if shared is not None:
        out["shared"] = dense_ffn_forward(x, *shared, rnd=rnd)
        y_sh = out["shared"]["y"]
    out["y"] = combine(y_perm, w, row_of_slot, k, add=y_sh, rnd=rnd)
    return out


def layer_backward(fwd, x, dy, w_gate, w_up, w_down, shared=None, rnd=bf16_round):
    """Backward of layer_forward for upstream gradient dy [T, d] (routing held fixed).

    Returns dY_perm, d_topk_w, dA, dW_down, dH_gate, dH_up, dX_perm, dW_gate, dW_up, dX
    (+ the shared FFN's gradients).
    """
    k = fwd["k"]
    off = fwd["offsets"]
    dy_perm, d_w = combine_bwd(dy, fwd["topk_w"], fwd["row_of_slot"], fwd["y_perm"], k, rnd)
    da = grouped_gemm_dx(dy_perm, w_down, off, rnd=rnd)
    dwd = grouped_gemm_dw(fwd["act"], dy_perm, off)
    dhg, dhu = swiglu_bwd(fwd["h_gate"], fwd["h_up"], da, rnd)
    dx_perm = grouped_gemm_dx(dhg, w_gate, off, dhu, w_up, rnd)
    dwg = grouped_gemm_dw(fwd["x_perm"], dhg, off)
    dwu = grouped_gemm_dw(fwd["x_perm"], dhu, off)
    out = {"dy_perm": dy_perm, "d_topk_w": d_w, "d_act": da, "dw_down": dwd, "dh_gate": dhg,
           "dh_up": dhu, "dx_perm": dx_perm, "dw_gate": dwg, "dw_up": dwu}
    dx_sh = None
    if shared is not None:
        out["shared"] = dense_ffn_backward(fwd["shared"], x, dy, *shared, rnd=rnd)
        dx_sh = out["shared"]["dx"]
    out["dx"] = combine(dx_perm, None, fwd["row_of_slot"], k, add=dx_sh, rnd=rnd)
    return out


# --------------------------------------------------------------------------------------------
# Sampled evaluation for large shapes: the same definitions restricted to chosen rows/columns
# --------------------------------------------------------------------------------------------
def expert_rows_forward(x_rows, w_gate_e, w_up_e, w_down_e, rnd=bf16_round):
    """Gate/up, SwiGLU and down for some rows of one expert (rows are independent)."""
    off = np.array([0, np.asarray(x_rows).shape[0]])
    hg = grouped_gemm(x_rows, np.asarray(w_gate_e)[None], off, rnd)
    hu = grouped_gemm(x_rows, np.asarray(w_up_e)[None], off, rnd)
    a = swiglu(hg, hu, rnd)
    y = grouped_gemm(a, np.asarray(w_down_e)[None], off, rnd)
    return hg, hu, a, y


def expert_rows_backward(hg, hu, dy_perm_rows, w_gate_e, w_up_e, w_down_e, rnd=bf16_round):
    """dA, dH_gate, dH_up and dX_perm for some rows of one expert."""
    off = np.array([0, np.asarray(hg).shape[0]])
    da = grouped_gemm_dx(dy_perm_rows, np.asarray(w_down_e)[None], off, rnd=rnd)
    dhg, dhu = swiglu_bwd(hg, hu, da, rnd)
    dxp = grouped_gemm_dx(dhg, np.asarray(w_gate_e)[None], off, dhu, np.asarray(w_up_e)[None], rnd)
    return da, dhg, dhu, dxp


def dw_down_rows(x_perm_e, dy_perm_e, w_gate_e, w_up_e, rows_f, rnd=bf16_round):
    """Rows `rows_f` of dW_down[e] = act_e^T dY_perm_e; needs only those columns of act_e."""
    off = np.array([0, np.asarray(x_perm_e).shape[0]])
    hg = grouped_gemm(x_perm_e, np.asarray(w_gate_e)[None, :, rows_f], off, rnd)
    hu = grouped_gemm(x_perm_e, np.asarray(w_up_e)[None, :, rows_f], off, rnd)
    a = swiglu(hg, hu, rnd)
    return grouped_gemm_dw(a, dy_perm_e, off)[0]


def dw_gate_up_cols(x_perm_e, dy_perm_e, w_gate_e, w_up_e, w_down_e, cols_f, rnd=bf16_round):
    """Columns `cols_f` of dW_gate[e] and dW_up[e] = X_perm_e^T dH_{gate,up}; needs only those
    columns of H_gate, H_up and dA."""
    off = np.array([0, np.asarray(x_perm_e).shape[0]])
    hg = grouped_gemm(x_perm_e, np.asarray(w_gate_e)[None, :, cols_f], off, rnd)
    hu = grouped_gemm(x_perm_e, np.asarray(w_up_e)[None, :, cols_f], off, rnd)
    da = grouped_gemm_dx(dy_perm_e, np.asarray(w_down_e)[None, cols_f, :], off, rnd=rnd)
    dhg, dhu = swiglu_bwd(hg, hu, da, rnd)
    return grouped_gemm_dw(x_perm_e, dhg, off)[0], grouped_gemm_dw(x_perm_e, dhu, off)[0]


# --------------------------------------------------------------------------------------------
# FP8 variant of the forward products (a variant beyond the paper, which is silent on it; the
# reading: the OCP 8-bit floating-point format E4M3, activations scaled per row and weights per
# output channel by fp32 factors, products accumulated exactly and rounded once to bf16)
# --------------------------------------------------------------------------------------------
E4M3_MAX = 448.0


def e4m3_decode(codes):
    """E4M3 codes (uint8) -> float64, exactly.

    Bit 7 is the sign, bits 6..3 the exponent field E (bias 7), bits 2..0 the mantissa M.  E = 0
    encodes the subnormals M/8 * 2**-6; otherwise the value is (1 + M/8) * 2**(E - 7).  The code
    with E = 15 and M = 7 (either sign) is NaN; the format has no infinities, so the largest finite
    magnitude is 1.75 * 2**8 = 448.
    """
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * np.ldexp(1.0, e - 7))
    mag = np.where((e == 15) & (c & 0x7 == 7), np.nan, mag)
    return np.where(c & 0x80, -mag, mag)


def e4m3_encode(x):
    """float -> E4M3 codes: round to the nearest representable magnitude, ties to the even
    mantissa; magnitudes beyond 448 saturate to 448; NaN -> 0x7F; the sign bit is x's (so values
    that round to zero keep their sign).

    A magnitude a in [2**n, 2**(n+1)) with n >= -6 has representable neighbours 2**(n-3) apart; below
    2**-6 (the subnormals) the spacing is 2**-9.  Rounding a / spacing to the nearest integer with
    ties to even gives the neighbour with the even mantissa.
    """
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(np.where(np.isnan(x), 0.0, x)), E4M3_MAX)
    _, fe = np.frexp(a)                       # a = f * 2**fe, 0.5 <= f < 1
    n = np.maximum(fe - 1, -6)                # binade exponent, clamped to the subnormal range
    q = np.ldexp(np.rint(np.ldexp(a, 3 - n)), n - 3)   # the rounded magnitude
    _, qe = np.frexp(q)
    qn = qe - 1
    normal = q >= 2.0 ** -6
    mant = np.where(normal, np.rint(np.ldexp(q, 3 - np.where(normal, qn, 0))) - 8, np.rint(q * 2.0 ** 9))
    code = np.where(normal, ((np.where(normal, qn, 0) + 7) << 3) + mant.astype(np.int64), mant.astype(np.int64))
    code = code.astype(np.int64) | np.where(np.signbit(x), 0x80, 0)
    code = np.where(np.isnan(x), 0x7F, code)
    return code.astype(np.uint8)


def quantize_rows_fp8(x):
    """Per-row E4M3 quantization: with amax = max |x[r, :]| (fp32), scale[r] = amax / 448 and
    codes[r, :] = e4m3_encode(x[r, :] * (448 / amax)), both quotients and the product taken in fp32
    (the precision the device kernel decides the codes in), so that the row's largest magnitude
    lands on 448; an all-zero row gets scale 1 and zero codes.  x ~= e4m3_decode(codes) * scale."""
    x32 = np.asarray(x, dtype=np.float32)
    amax = np.max(np.abs(x32), axis=-1)
    big = amax > 0
    scale = np.ones_like(amax)
    np.divide(amax, np.float32(E4M3_MAX), out=scale, where=big)
    inv = np.ones_like(amax)
    np.divide(np.float32(E4M3_MAX), amax, out=inv, where=big)
    y = (x32 * inv[..., None]).astype(np.float32)
    return e4m3_encode(y.astype(np.float64)), scale.astype(np.float32)


def grouped_gemm_fp8(a_codes, a_scale, wt_codes, w_scale, offsets, rnd=bf16_round):
    """The forward grouped product on E4M3 operands: for rows r of group g,
    C[r, n] = a_scale[r] * w_scale[g, n] * sum_k dec(A[r, k]) * dec(Wt[g, n, k]), rounded once to
    bf16.  A [R, K] codes with per-row scales [R]; Wt [G, N, K] codes (the weight in the layout
    [output channel, contraction]) with per-channel scales [G, N]."""
    A = e4m3_decode(a_codes)
    W = e4m3_decode(wt_codes)
    sa = np.asarray(a_scale, dtype=np.float64)
    sw = np.asarray(w_scale, dtype=np.float64)
    G, N, _ = W.shape
    C = np.zeros((A.shape[0], N))
    for g in range(G):
        lo, hi = int(offsets[g]), int(offsets[g + 1])
        if hi > lo:
            C[lo:hi] = (A[lo:hi] @ W[g].T) * sa[lo:hi, None] * sw[g][None, :]
    return _r(rnd, C)


# --------------------------------------------------------------------------------------------
# MX (microscaling) variant of the FP8 products, also beyond the paper.  The reading: the OCP
# microscaling formats' block structure, E4M3 elements sharing one power-of-two scale (an E8M0
# byte, value 2**(byte - 127)) per 32 consecutive contraction elements of a row; the shared
# exponent is the smallest one that keeps every element of the block within E4M3's range (no
# element saturates), and an all-zero block gets the smallest scale, byte 0.
# --------------------------------------------------------------------------------------------
MX_BLOCK = 32


def mx_block_exponent(amax):
    """The smallest integer e with amax <= 448 * 2**e, raised to -127 where it is below (the
    smallest E8M0 value; every all-zero block gets it).  amax >= 0, finite."""
    amax = np.asarray(amax, dtype=np.float64)
    pos = amax > 0
    e = np.where(pos, np.ceil(np.log2(np.where(pos, amax, 1.0) / E4M3_MAX)), -127.0).astype(np.int64)
    # the logarithm may be off by one ulp next to a power of two: settle e on the definition
    e = np.where(pos & (amax > np.ldexp(E4M3_MAX, e)), e + 1, e)
    e = np.where(pos & (amax <= np.ldexp(E4M3_MAX, e - 1)), e - 1, e)
    return np.maximum(e, -127)


def quantize_rows_mx(x):
    """MX quantization along the last axis (its length a multiple of 32): for each block of 32
    consecutive elements, e = mx_block_exponent(max |block|), scale byte e + 127 and codes
    e4m3_encode(x * 2**-e) (an exact scaling, so the codes round x itself to the E4M3 grid times
    2**e).  Returns codes (x's shape, uint8) and scale bytes (x's shape with the last axis / 32,
    uint8); x ~= e4m3_decode(codes) * 2**(bytes - 127) per block."""
    x = np.asarray(x, dtype=np.float64)
    C = x.shape[-1]
    assert C % MX_BLOCK == 0
    blocks = x.reshape(x.shape[:-1] + (C // MX_BLOCK, MX_BLOCK))
    e = mx_block_exponent(np.max(np.abs(blocks), axis=-1))
    codes = e4m3_encode(np.ldexp(blocks, -e[..., None]))
    return codes.reshape(x.shape), (e + 127).astype(np.uint8)


def mx_decode(codes, scale_bytes):
    """MX operand -> float64: e4m3_decode(codes) times 2**(byte - 127) of each element's block."""
    v = e4m3_decode(codes)
    s = np.asarray(scale_bytes, dtype=np.int64) - 127
    return np.ldexp(v, np.repeat(s, MX_BLOCK, axis=-1))


def grouped_gemm_mx(a_codes, a_scale, wt_codes, w_scale, offsets, rnd=bf16_round):
    """The grouped product on MX operands: for rows r of group g,
    C[r, n] = sum_k mx(A)[r, k] * mx(Wt[g])[n, k], accumulated exactly and rounded once to bf16.
    A [R, K] codes with scale bytes [R, K/32]; Wt [G, N, K] codes (the weight in the layout
    [output channel, contraction]) with scale bytes [G, N, K/32]."""
    A = mx_decode(a_codes, a_scale)
    W = mx_decode(wt_codes, w_scale)
    G, N, _ = W.shape
    C = np.zeros((A.shape[0], N))
    for g in range(G):
        lo, hi = int(offsets[g]), int(offsets[g + 1])
        if hi > lo:
            C[lo:hi] = A[lo:hi] @ W[g].T
    return _r(rnd, C)


def pack_groups_t(x, offsets, align=128):
    """The contraction-major form of a routed buffer for the weight gradient on MX operands: x
    [R, C] rows grouped by offsets -> [C, L], group g's rows as columns p[g] .. p[g] + K_g - 1 with
    p[g] = sum over h < g of K_h rounded up to a multiple of `align`, zeros elsewhere (so that no
    32-element block of a row spans two groups).  Returns the packed matrix and p [G+1]."""
    x = np.asarray(x, dtype=np.float64)
    off = np.asarray(offsets, dtype=np.int64)
    cnt = off[1:] - off[:-1]
    p = np.zeros(len(cnt) + 1, dtype=np.int64)
    p[1:] = np.cumsum((cnt + align - 1) // align * align)
    out = np.zeros((x.shape[1], int(p[-1])))
    for g in range(len(cnt)):
        out[:, p[g]:p[g] + cnt[g]] = x[off[g]:off[g + 1]].T
    return out, p


def grouped_gemm_dw_mx(at_codes, at_scale, ct_codes, ct_scale, offsets, align=128):
    """The ragged weight gradient on MX operands (Appendix H's dW_e = X_e^T G_e with both operands
    quantized along the token axis): At [K, L] and Ct [N, L] codes in the layout of pack_groups_t
    with scale bytes [K, L/32] and [N, L/32]; dW[g] = sum over the group's K_g token columns of
    mx(At)[:, t] mx(Ct)[:, t]^T, float64 (fp32 storage is not modelled: the result stays exact)."""
    A = mx_decode(at_codes, at_scale)
    C = mx_decode(ct_codes, ct_scale)
    off = np.asarray(offsets, dtype=np.int64)
    cnt = off[1:] - off[:-1]
    G = len(cnt)
    p = np.zeros(G + 1, dtype=np.int64)
    p[1:] = np.cumsum((cnt + align - 1) // align * align)
    out = np.zeros((G, A.shape[0], C.shape[0]))
    for g in range(G):
        cols = slice(int(p[g]), int(p[g] + cnt[g]))
        out[g] = A[:, cols] @ C[:, cols].T
    return out


def rel_fro(got, ref):
    """||got - ref||_F / ||ref||_F in float64 (0 if both are zero, inf if only ref is zero)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.linalg.norm((got - ref).ravel())
    den = np.linalg.norm(ref.ravel())
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return float(num / den)
