"""Planted mistakes in the oracle (on the CPU only): each plausible mistake must make at least one
of the oracle's pins fail, which shows the pins constrain every part of it."""
import numpy as np
import pytest

from oracle import moe_oracle as O
from tests import test_oracle as P

PINS = [
    P.test_bf16_round_matches_torch_random,
    P.test_bf16_round_ties_and_edges,
    P.test_route_permute_worked_example,
    lambda: P.test_route_brute_force_with_ties(8, 3),
    P.test_route_weights_library_softmax,
    lambda: P.test_permute_invariants(64, 8, 2),
    P.test_gather_combine_round_trip,
    P.test_dw_worked_example,
    P.test_grouped_gemms_exact_vs_torch,
    P.test_grouped_gemm_brute_force_loops,
    P.test_swiglu_closed_forms_and_library,
    P.test_swiglu_bwd_autograd,
    lambda: P.test_layer_forward_vs_brute_force(12),
    P.test_layer_single_expert_is_dense_ffn,
    lambda: P.test_layer_backward_vs_autograd(12),
    P.test_layer_backward_finite_differences,
    P.test_router_logits_one_hot_and_integers,
    lambda: P.test_route_topk_bwd_autograd(True),
    lambda: P.test_route_topk_bwd_autograd(False),
    P.test_route_topk_bwd_properties_and_fd,
    P.test_aux_loss_closed_form_and_autograd,
    P.test_router_bwd_autograd,
    P.test_e4m3_decode_spec_values_and_torch,
    P.test_e4m3_encode_brute_force_and_torch,
    P.test_quantize_rows_fp8_properties,
    P.test_grouped_gemm_fp8_vs_library,
    P.test_mx_block_exponent_hand_values,
    P.test_quantize_rows_mx_worked_example,
    P.test_quantize_rows_mx_properties,
    P.test_grouped_gemm_mx_vs_library,
    P.test_pack_groups_t_brute_force,
    P.test_grouped_gemm_dw_mx_vs_library,
    P.test_rel_fro_hand_values,
]


def _gg(A, B, offsets, rnd=O.bf16_round):                      # wrong expert's weights
    A = np.asarray(A, dtype=np.float64)
    G = B.shape[0]
    C = np.zeros((A.shape[0], B.shape[2]))
    for g in range(G):
        lo, hi = int(offsets[g]), int(offsets[g + 1])
        C[lo:hi] = A[lo:hi] @ B[(g + 1) % G]
    return O._r(rnd, C)


def _dw_drop_last(A, dC, offsets, G=None):                      # ragged bound off by one
    G = len(offsets) - 1 if G is None else G
    out = np.zeros((G, A.shape[1], dC.shape[1]))
    for g in range(G):
        lo, hi = int(offsets[g]), int(offsets[g + 1])
        if hi - 1 > lo:
            out[g] = np.asarray(A[lo:hi - 1]).T @ np.asarray(dC[lo:hi - 1])
    return out


def _dx_b_twice(dC, B, offsets, dC2=None, B2=None, rnd=O.bf16_round):   # second pair uses B
    return O.__dict__["_orig_dx"](dC, B, offsets, dC2, B if B2 is not None else None, rnd)


def _swiglu_bwd_dropped(h_gate, h_up, d_act, rnd=O.bf16_round):         # dropped term
    s = O.sigmoid(h_gate)
    return O._r(rnd, d_act * h_up * s), O._r(rnd, d_act * h_gate * s)


def _swiglu_bwd_sign(h_gate, h_up, d_act, rnd=O.bf16_round):            # wrong sign
    g, u, da = (np.asarray(v, dtype=np.float64) for v in (h_gate, h_up, d_act))
    s = O.sigmoid(g)
    return O._r(rnd, da * u * s * (1.0 - g * (1.0 - s))), O._r(rnd, da * g * s)


def _combine_bwd_unweighted(dy, topk_w, row_of_slot, y_perm, k, rnd=O.bf16_round):
    return O.__dict__["_orig_cb"](dy, None, row_of_slot, y_perm, k, rnd)


def _route_ties_high(logits, k, normalize=True):                        # ties -> higher id
    L = np.asarray(logits, dtype=np.float64)
    T, E = L.shape
    ids = np.broadcast_to(np.arange(E), (T, E))
    idx = np.lexsort((-ids, -L), axis=-1)[:, :k]
    sel = np.take_along_axis(L, idx, 1)
    ex = np.exp(sel - sel[:, :1])
    return idx, ex / ex.sum(1, keepdims=True)


def _permute_desc(topk_idx, E):                                          # wrong in-group order
    off, ros, tor = O.__dict__["_orig_perm"](topk_idx, E)
    ros2 = ros.copy()
    for e in range(E):
        lo, hi = off[e], off[e + 1]
        sel = (ros >= lo) & (ros < hi)
        ros2[sel] = lo + hi - 1 - ros[sel]
    tor2 = np.empty_like(tor)
    tor2[ros2] = np.arange(len(ros2)) // topk_idx.shape[1]
    return off, ros2, tor2


def _bf16_truncate(x):                                                   # truncation, not RNE
    x = np.asarray(x, dtype=np.float64)
    b = x.astype(np.float32).view(np.uint32) & np.uint32(0xFFFF0000)
    return b.view(np.float32).astype(np.float64)


def _combine_weighted_add(y_perm, topk_w, row_of_slot, k, add=None, rnd=O.bf16_round):
    out = O.__dict__["_orig_comb"](y_perm, topk_w, row_of_slot, k, None, None)
    if add is not None:
        out = out + 0.5 * np.asarray(add)
    return O._r(rnd, out)


def _logits_no_bias(x, wr, bias=None):                                   # bias dropped
    return np.asarray(x, dtype=np.float64) @ np.asarray(wr, dtype=np.float64)


def _topk_bwd_no_mean(logits, topk_idx, d_topk_w, normalize=True):       # dropped subtraction
    L = np.asarray(logits, dtype=np.float64)
    idx = np.asarray(topk_idx)
    sel = np.take_along_axis(L, idx, axis=1)
    ex = np.exp(sel - sel.max(axis=1, keepdims=True))
    p = np.zeros(L.shape)
    np.put_along_axis(p, idx, ex / ex.sum(axis=1, keepdims=True), axis=1)
    G = np.zeros(L.shape)
    np.put_along_axis(G, idx, np.asarray(d_topk_w, dtype=np.float64), axis=1)
    return p * G


def _topk_bwd_full_softmax(logits, topk_idx, d_topk_w, normalize=True):  # wrong probabilities
    return O.__dict__["_orig_tkb"](logits, topk_idx, d_topk_w, False)


def _aux_no_E(logits, counts, k, alpha):                                   # missing factor E
    loss, grad = O.__dict__["_orig_aux"](logits, counts, k, alpha)
    E = np.asarray(logits).shape[1]
    return loss / E, grad / E


def _router_bwd_misaligned(x, wr, dlogits, dx=None, rnd=O.bf16_round):     # token rows misaligned
    x = np.asarray(x, dtype=np.float64)
    g = np.asarray(dlogits, dtype=np.float64)
    share = g @ np.asarray(wr, dtype=np.float64).T
    if dx is not None:
        share = np.asarray(dx, dtype=np.float64) + share
    return x.T @ np.roll(g, 1, axis=0), O._r(rnd, share)


def _e4m3_ties_away(x):                                                   # ties away from zero
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), 448.0)
    _, fe = np.frexp(a)
    n = np.maximum(fe - 1, -6)
    q = np.ldexp(np.floor(np.ldexp(a, 3 - n) + 0.5), n - 3)
    return O.__dict__["_orig_enc"](np.copysign(q, x))


def _e4m3_decode_bias8(codes):                                            # exponent bias off by one
    return O.__dict__["_orig_dec"](codes) * 0.5


def _fp8_gemm_no_weight_scale(a_codes, a_scale, wt_codes, w_scale, offsets, rnd=O.bf16_round):
    return O.__dict__["_orig_f8"](a_codes, a_scale, wt_codes, np.ones_like(w_scale), offsets, rnd)


def _quant_inverted_scale(x):                                             # scale = 448 / amax
    codes, scale = O.__dict__["_orig_q8"](x)
    return codes, np.where(scale != 1, (np.float32(448.0) ** 2 / 448.0) / (scale * 448.0), scale).astype(np.float32)


def _mx_exponent_floor_rule(amax):                                      # e = floor(log2 amax) - 8
    amax = np.asarray(amax, dtype=np.float64)
    pos = amax > 0
    _, fe = np.frexp(np.where(pos, amax, 1.0))
    return np.where(pos, np.maximum(fe - 1 - 8, -127), -127).astype(np.int64)


def _mx_exponent_no_clamp(amax):                                          # no floor at -127
    amax = np.asarray(amax, dtype=np.float64)
    pos = amax > 0
    e = np.ceil(np.log2(np.where(pos, amax, 1.0) / 448.0)).astype(np.int64)
    return np.where(pos, e, -127)


def _quant_mx_blocks_of_16(x):                                             # 16-element blocks
    x = np.asarray(x, dtype=np.float64)
    blocks = x.reshape(x.shape[:-1] + (x.shape[-1] // 16, 16))
    e = O.mx_block_exponent(np.max(np.abs(blocks), axis=-1))
    codes = O.e4m3_encode(np.ldexp(blocks, -e[..., None]))
    return codes.reshape(x.shape), (e[..., ::2] + 127).astype(np.uint8)


def _mx_decode_tiled_scales(codes, scale_bytes):                           # scales tiled, not repeated
    v = O.e4m3_decode(codes)
    s = np.asarray(scale_bytes, dtype=np.int64) - 127
    return np.ldexp(v, np.tile(s, (1,) * (s.ndim - 1) + (32,)))


def _mx_gemm_scale_negated(a_codes, a_scale, wt_codes, w_scale, offsets, rnd=O.bf16_round):   # 2**(127 - byte)
    return O.__dict__["_orig_mxg"](a_codes, (254 - np.asarray(a_scale, dtype=np.int64)).astype(np.uint8),
                                   wt_codes, w_scale, offsets, rnd)


def _pack_groups_t_align32(x, offsets, align=128):                        # padding to 32, not 128
    return O.__dict__["_orig_pgt"](x, offsets, 32)


def _pack_groups_t_drop_last(x, offsets, align=128):                      # each group's last row lost
    out, p = O.__dict__["_orig_pgt"](x, offsets, align)
    off = np.asarray(offsets)
    for g in range(len(off) - 1):
        if off[g + 1] > off[g]:
            out[:, p[g] + off[g + 1] - off[g] - 1] = 0.0
    return out, p


def _dw_mx_next_group_scales(at_codes, at_scale, ct_codes, ct_scale, offsets, align=128):   # scales shifted a block
    return O.__dict__["_orig_dwmx"](at_codes, np.roll(at_scale, 1, axis=1), ct_codes, ct_scale, offsets, align)


def _rel_fro_squared(got, ref):                                           # squared ratio
    r = O.__dict__["_orig_rf"](got, ref)
    return r * r


def _rel_fro_got_norm(got, ref):                                          # ||got|| denominator
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(got.ravel())
    num = np.linalg.norm((got - ref).ravel())
    return 0.0 if num == 0.0 else (float("inf") if den == 0.0 else float(num / den))


def _rel_fro_row_mean(got, ref):                                          # mean of per-row ratios
    got = np.atleast_2d(np.asarray(got, dtype=np.float64))
    ref = np.atleast_2d(np.asarray(ref, dtype=np.float64))
    g2 = got.reshape(got.shape[0], -1)
    r2 = ref.reshape(ref.shape[0], -1)
    vals = [O.__dict__["_orig_rf"](a, b) for a, b in zip(g2, r2)]
    return float(np.mean(vals))


def _rel_fro_zero(got, ref):                                              # always passes
    return 0.0


MUTANTS = {
    "rel_fro squared": ("rel_fro", _rel_fro_squared),
    "rel_fro divides by the norm of got": ("rel_fro", _rel_fro_got_norm),
    "rel_fro averages per-row ratios": ("rel_fro", _rel_fro_row_mean),
    "rel_fro returns zero": ("rel_fro", _rel_fro_zero),
    "e4m3 ties away from zero": ("e4m3_encode", _e4m3_ties_away),
    "e4m3 exponent bias 8": ("e4m3_decode", _e4m3_decode_bias8),
    "fp8 gemm ignores the weight scale": ("grouped_gemm_fp8", _fp8_gemm_no_weight_scale),
    "fp8 quantization stores the inverse scale": ("quantize_rows_fp8", _quant_inverted_scale),
    "mx exponent by floor(log2 amax) - 8": ("mx_block_exponent", _mx_exponent_floor_rule),
    "mx exponent not raised to -127": ("mx_block_exponent", _mx_exponent_no_clamp),
    "mx blocks of 16": ("quantize_rows_mx", _quant_mx_blocks_of_16),
    "mx decode tiles the scales": ("mx_decode", _mx_decode_tiled_scales),
    "mx gemm negated activation scale": ("grouped_gemm_mx", _mx_gemm_scale_negated),
    "pack_groups_t pads to 32": ("pack_groups_t", _pack_groups_t_align32),
    "pack_groups_t drops each group's last row": ("pack_groups_t", _pack_groups_t_drop_last),
    "mx dW ignores the scales of a shifted block": ("grouped_gemm_dw_mx", _dw_mx_next_group_scales),
    "router logits drop the bias": ("router_logits", _logits_no_bias),
    "route_topk_bwd drops the weighted mean": ("route_topk_bwd", _topk_bwd_no_mean),
    "route_topk_bwd uses the full softmax": ("route_topk_bwd", _topk_bwd_full_softmax),
    "aux loss without the factor E": ("aux_loss", _aux_no_E),
    "router_bwd pairs x and dlogits of different tokens": ("router_bwd", _router_bwd_misaligned),
    "grouped_gemm wrong expert": ("grouped_gemm", _gg),
    "dw ragged bound off by one": ("grouped_gemm_dw", _dw_drop_last),
    "dx second pair uses first weights": ("grouped_gemm_dx", _dx_b_twice),
    "swiglu_bwd dropped term": ("swiglu_bwd", _swiglu_bwd_dropped),
    "swiglu_bwd sign": ("swiglu_bwd", _swiglu_bwd_sign),
    "combine_bwd unweighted": ("combine_bwd", _combine_bwd_unweighted),
    "route ties to higher id": ("route_topk", _route_ties_high),
    "permute descending tokens": ("permute", _permute_desc),
    "bf16 truncation": ("bf16_round", _bf16_truncate),
    "combine weights the shared add": ("combine", _combine_weighted_add),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setitem(O.__dict__, "_orig_dx", O.grouped_gemm_dx)
    monkeypatch.setitem(O.__dict__, "_orig_cb", O.combine_bwd)
    monkeypatch.setitem(O.__dict__, "_orig_perm", O.permute)
    monkeypatch.setitem(O.__dict__, "_orig_comb", O.combine)
    monkeypatch.setitem(O.__dict__, "_orig_tkb", O.route_topk_bwd)
    monkeypatch.setitem(O.__dict__, "_orig_aux", O.aux_loss)
    monkeypatch.setitem(O.__dict__, "_orig_enc", O.e4m3_encode)
    monkeypatch.setitem(O.__dict__, "_orig_dec", O.e4m3_decode)
    monkeypatch.setitem(O.__dict__, "_orig_f8", O.grouped_gemm_fp8)
    monkeypatch.setitem(O.__dict__, "_orig_q8", O.quantize_rows_fp8)
    monkeypatch.setitem(O.__dict__, "_orig_rf", O.rel_fro)
    monkeypatch.setitem(O.__dict__, "_orig_mxg", O.grouped_gemm_mx)
    monkeypatch.setitem(O.__dict__, "_orig_pgt", O.pack_groups_t)
    monkeypatch.setitem(O.__dict__, "_orig_dwmx", O.grouped_gemm_dw_mx)
    monkeypatch.setattr(O, attr, fn)
    if attr == "bf16_round":
        # default arguments captured the original function; patch the module-level users too
        monkeypatch.setattr(O, "_r", lambda rnd, x: x if rnd is None else _bf16_truncate(x))
    failures = 0
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            failures += 1
        except (ValueError, IndexError):
            failures += 1
    assert failures > 0, f"no pin caught the planted mistake '{name}'"
