"""Python binding of libmoe_mi355x.so: one function per C entry point, same names.

Argument marshalling only: tensors become device pointers, the stream defaults to torch's
current stream, and missing outputs are allocated with torch (device memory is torch's job).
Every computation runs in the library's HIP kernels; if the library is missing this module
raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os

import torch

from .build import LIB_PATH

_lib = None

MOE_SUCCESS = 0
STATUS_NAMES = {0: "MOE_SUCCESS", 1: "MOE_ERROR_INVALID_VALUE", 2: "MOE_ERROR_NOT_SUPPORTED",
                3: "MOE_ERROR_WORKSPACE", 4: "MOE_ERROR_HIP"}


class MoEError(RuntimeError):
    def __init__(self, fn, status, detail):
        super().__init__(f"{fn}: {STATUS_NAMES.get(status, status)}: {detail}")
        self.status = status


_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
_SIG = {
    "moe_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "moe_last_error": (ctypes.c_char_p, []),
    "moe_route_permute_workspace_bytes": (ctypes.c_size_t, [_I64, _I32, _I32]),
    "moe_route_permute": (ctypes.c_int, [_P, _P, _I64, _I64, _I32, _I32, _I32, _P, _P, _P, _P, _P,
                                         _P, _P, ctypes.c_size_t, _P]),
    "moe_grouped_gemm_fwd": (ctypes.c_int, [_P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P, _P]),
    "moe_grouped_gemm_fwd_split": (ctypes.c_int, [_P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P, _P,
                                                  ctypes.c_size_t, _P]),
    "moe_grouped_gemm_fwd_combine_workspace_bytes": (ctypes.c_size_t, [_I64, _I64]),
    "moe_grouped_gemm_fwd_combine": (ctypes.c_int, [_P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P, _I64, _I32, _P,
                                                    _P, _P, _P, ctypes.c_size_t, _P, ctypes.c_size_t, _P]),
    "moe_grouped_gemm_fwd_gather": (ctypes.c_int, [_P, _I64, _P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P,
                                                   _P, ctypes.c_size_t, _P]),
    "moe_gather_rows": (ctypes.c_int, [_P, _I64, _I64, _I32, _P, _P, _P]),
    "moe_route_permute_noalloc_max_scratch_bytes": (ctypes.c_size_t, []),
    "moe_route_permute_noalloc": (ctypes.c_int, [_P, _P, _I64, _I64, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P]),
    "moe_quantize_fp8_rows": (ctypes.c_int, [_P, _I64, _I64, _P, _P, _P]),
    "moe_quantize_fp8_rows2": (ctypes.c_int, [_P, _P, _I64, _I64, _P, _P, _P]),
    "moe_grouped_gemm_dx_swiglu_bwd_fp8": (ctypes.c_int, [_P, _P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P,
                                                          _P, _P, ctypes.c_size_t, _P]),
    "moe_quantize_fp8_weight": (ctypes.c_int, [_P, _P, _I64, _I64, _I64, _P, _P, _P]),
    "moe_grouped_gemm_fwd_fp8": (ctypes.c_int, [_P, _P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P,
                                                ctypes.c_size_t, _P]),
    "moe_grouped_gemm_fwd_fp8_gate_up": (ctypes.c_int, [_P, _P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P, _P,
                                                        ctypes.c_size_t, _P]),
    "moe_mx_scale_bytes": (_I64, [_I64, _I64]),
    "moe_mx_tokens_cols_bound": (_I64, [_I64, _I32]),
    "moe_quantize_mx_tokens_t": (ctypes.c_int, [_P, _P, _I32, _I64, _I64, _P, _P, _I64, _P]),
    "moe_quantize_mx_tokens": (ctypes.c_int, [_P, _P, _I32, _I64, _I64, _P, _P, _I64, _P, _P, _I64, _I64, _P]),
    "moe_grouped_gemm_dw_mx": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _I32, _I64, _I64, _I64, _I64, _P, _P,
                                              _I32, _P, _P]),
    "moe_quantize_mx_rows": (ctypes.c_int, [_P, _P, _I64, _I64, _P, _P, _P]),
    "moe_quantize_mx_weight": (ctypes.c_int, [_P, _P, _I64, _I64, _I64, _P, _P, _P, _P, _P]),
    "moe_grouped_gemm_fwd_mx": (ctypes.c_int, [_P, _P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P,
                                               ctypes.c_size_t, _P]),
    "moe_grouped_gemm_fwd_mx_gate_up": (ctypes.c_int, [_P, _P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P, _P,
                                                       ctypes.c_size_t, _P]),
    "moe_grouped_gemm_dx_swiglu_bwd_mx": (ctypes.c_int, [_P, _P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P,
                                                         _P, _P, ctypes.c_size_t, _P]),
    "moe_swiglu": (ctypes.c_int, [_P, _P, _P, _I64, _I64, _P]),
    "moe_swiglu_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _I64, _I64, _P]),
    "moe_unpermute_combine": (ctypes.c_int, [_P, _P, _P, _P, _I64, _I64, _I32, _P, _P]),
    "moe_unpermute_combine_bwd": (ctypes.c_int, [_P, _P, _P, _P, _I64, _I64, _I32, _P, _P, _P]),
    "moe_grouped_gemm_dx": (ctypes.c_int, [_P, _P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P]),
    "moe_grouped_gemm_dw": (ctypes.c_int, [_P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P]),
    "moe_grouped_gemm_dw_bf16": (ctypes.c_int, [_P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P]),
    "moe_grouped_gemm_dw_persistent": (ctypes.c_int, [_P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P, _P]),
    "moe_grouped_gemm_dw_bf16_persistent": (ctypes.c_int, [_P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P, _P]),
    "moe_grouped_gemm_dw_split": (ctypes.c_int, [_P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P, _P,
                                                 ctypes.c_size_t, _P]),
    "moe_grouped_gemm_split_workspace_bytes": (ctypes.c_size_t, []),
    "moe_grouped_gemm_dx_split": (ctypes.c_int, [_P, _P, _P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, ctypes.c_size_t,
                                                 _P]),
    "moe_grouped_gemm_dx_swiglu_bwd_split": (ctypes.c_int, [_P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P, _P, _P,
                                                            ctypes.c_size_t, _P]),
    "moe_grouped_gemm_dw_t": (ctypes.c_int, [_P, _P, _P, _P, _I32, _I64, _I64, _I64, _I64, _P, _P, _I32, _P]),
    "moe_transposed_cols_bound": (ctypes.c_int64, [_I64, _I32]),
    "moe_transpose_grouped": (ctypes.c_int, [_P, _P, _I32, _I64, _I64, _P, _I64, _P]),
    "moe_router_logits": (ctypes.c_int, [_P, _P, _P, _I64, _I64, _I32, _P, _P]),
    "moe_router_bwd_workspace_bytes": (ctypes.c_size_t, [_I64, _I64, _I32]),
    "moe_router_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I32, _I32, _I32, ctypes.c_float,
                                      _P, ctypes.c_size_t, _P, _P, _P, _P]),
    "moe_unpermute_router_dx": (ctypes.c_int, [_P, _P, _P, _P, _P, _I64, _I64, _I32, _I32, _P, _P]),
    "moe_router_aux_loss_workspace_bytes": (ctypes.c_size_t, [_I64, _I32]),
    "moe_router_aux_loss": (ctypes.c_int, [_P, _P, _I64, _I32, _I32, ctypes.c_float, _P, ctypes.c_size_t, _P, _P]),
    "moe_grouped_gemm_dx_swiglu_bwd": (ctypes.c_int, [_P, _P, _P, _I32, _I64, _I64, _I64, _P, _P, _P, _P, _P]),
}


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_26453_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIG.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(fn, status):
    if status != MOE_SUCCESS:
        raise MoEError(fn, status, lib().moe_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("tensors passed to the MoE library must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors passed to the MoE library must be contiguous")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _need(t, dtype, shape, name):
    if t is None:
        return
    if t.dtype != dtype or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected {dtype} {tuple(shape)}, got {t.dtype} {tuple(t.shape)}")


def moe_route_permute_workspace_bytes(T, E, k):
    return lib().moe_route_permute_workspace_bytes(T, E, k)


def moe_route_permute(logits, x, k, normalize_topk=True, topk_idx=None, topk_w=None, offsets=None,
                      row_of_slot=None, token_of_row=None, x_perm=None, workspace=None, stream=None):
    T, E = logits.shape
    dev = logits.device
    _need(logits, torch.float32, (T, E), "logits")
    d = x.shape[1] if x is not None else 0
    if x is not None:
        _need(x, torch.bfloat16, (T, d), "x")
    R = T * k
    topk_idx = torch.empty((T, k), dtype=torch.int32, device=dev) if topk_idx is None else topk_idx
    topk_w = torch.empty((T, k), dtype=torch.float32, device=dev) if topk_w is None else topk_w
    offsets = torch.empty(E + 1, dtype=torch.int32, device=dev) if offsets is None else offsets
    row_of_slot = torch.empty(R, dtype=torch.int32, device=dev) if row_of_slot is None else row_of_slot
    token_of_row = torch.empty(R, dtype=torch.int32, device=dev) if token_of_row is None else token_of_row
    if x is not None and x_perm is None:
        x_perm = torch.empty((R, d), dtype=torch.bfloat16, device=dev)
    _need(topk_idx, torch.int32, (T, k), "topk_idx")
    _need(topk_w, torch.float32, (T, k), "topk_w")
    _need(offsets, torch.int32, (E + 1,), "offsets")
    _need(row_of_slot, torch.int32, (R,), "row_of_slot")
    _need(token_of_row, torch.int32, (R,), "token_of_row")
    _need(x_perm, torch.bfloat16, (R, d), "x_perm")
    ws_bytes = moe_route_permute_workspace_bytes(T, E, k)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=dev)
    st = lib().moe_route_permute(_ptr(logits), _ptr(x), T, d, E, k, int(bool(normalize_topk)),
                                 _ptr(topk_idx), _ptr(topk_w), _ptr(offsets), _ptr(row_of_slot),
                                 _ptr(token_of_row), _ptr(x_perm), _ptr(workspace),
                                 workspace.numel() * workspace.element_size(), _stream(stream))
    _check("moe_route_permute", st)
    return {"topk_idx": topk_idx, "topk_w": topk_w, "offsets": offsets, "row_of_slot": row_of_slot,
            "token_of_row": token_of_row, "x_perm": x_perm}


def moe_route_permute_noalloc(logits, x, k, normalize_topk=True, topk_idx=None, topk_w=None, offsets=None,
                              row_of_slot=None, token_of_row=None, x_perm=None, stream=None):
    """moe_route_permute without a workspace: the library's own device scratch holds the
    per-range histogram (calls on one device must not overlap)."""
    T, E = logits.shape
    dev = logits.device
    _need(logits, torch.float32, (T, E), "logits")
    d = x.shape[1] if x is not None else 0
    if x is not None:
        _need(x, torch.bfloat16, (T, d), "x")
    R = T * k
    topk_idx = torch.empty((T, k), dtype=torch.int32, device=dev) if topk_idx is None else topk_idx
    topk_w = torch.empty((T, k), dtype=torch.float32, device=dev) if topk_w is None else topk_w
    offsets = torch.empty(E + 1, dtype=torch.int32, device=dev) if offsets is None else offsets
    row_of_slot = torch.empty(R, dtype=torch.int32, device=dev) if row_of_slot is None else row_of_slot
    token_of_row = torch.empty(R, dtype=torch.int32, device=dev) if token_of_row is None else token_of_row
    if x is not None and x_perm is None:
        x_perm = torch.empty((R, d), dtype=torch.bfloat16, device=dev)
    _need(topk_idx, torch.int32, (T, k), "topk_idx")
    _need(topk_w, torch.float32, (T, k), "topk_w")
    _need(offsets, torch.int32, (E + 1,), "offsets")
    _need(row_of_slot, torch.int32, (R,), "row_of_slot")
    _need(token_of_row, torch.int32, (R,), "token_of_row")
    _need(x_perm, torch.bfloat16, (R, d), "x_perm")
    st = lib().moe_route_permute_noalloc(_ptr(logits), _ptr(x), T, d, E, k, int(bool(normalize_topk)),
                                         _ptr(topk_idx), _ptr(topk_w), _ptr(offsets), _ptr(row_of_slot),
                                         _ptr(token_of_row), _ptr(x_perm), _stream(stream))
    _check("moe_route_permute_noalloc", st)
    return {"topk_idx": topk_idx, "topk_w": topk_w, "offsets": offsets, "row_of_slot": row_of_slot,
            "token_of_row": token_of_row, "x_perm": x_perm}


def moe_grouped_gemm_fwd(A, B, offsets, B2=None, C=None, C2=None, act=None, want_act=False,
                         stream=None, workspace=None):
    R, K = A.shape
    G, K2, N = B.shape
    if K2 != K:
        raise ValueError("A and B disagree on K")
    _need(A, torch.bfloat16, (R, K), "A")
    _need(B, torch.bfloat16, (G, K, N), "B")
    _need(B2, torch.bfloat16, (G, K, N), "B2")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    dev = A.device
    C = torch.empty((R, N), dtype=torch.bfloat16, device=dev) if C is None else C
    if B2 is not None and C2 is None:
        C2 = torch.empty((R, N), dtype=torch.bfloat16, device=dev)
    if want_act and act is None:
        act = torch.empty((R, N), dtype=torch.bfloat16, device=dev)
    for t, n in ((C, "C"), (C2, "C2"), (act, "act")):
        _need(t, torch.bfloat16, (R, N), n)
    if workspace is None:
        st = lib().moe_grouped_gemm_fwd(_ptr(A), _ptr(B), _ptr(B2), _ptr(offsets), G, R, K, N, _ptr(C),
                                        _ptr(C2), _ptr(act), _stream(stream))
        _check("moe_grouped_gemm_fwd", st)
    else:
        st = lib().moe_grouped_gemm_fwd_split(_ptr(A), _ptr(B), _ptr(B2), _ptr(offsets), G, R, K, N, _ptr(C),
                                              _ptr(C2), _ptr(act), _ptr(workspace), workspace.numel(),
                                              _stream(stream))
        _check("moe_grouped_gemm_fwd_split", st)
    return C, C2, act


def moe_grouped_gemm_fwd_gather(X, row_src, B, offsets, B2=None, C=None, C2=None, act=None, want_act=False,
                                stream=None, workspace=None):
    """moe_grouped_gemm_fwd on the rows X[row_src[r]] (the gather folded into the product)."""
    T, K = X.shape
    (R,) = row_src.shape
    G, K2, N = B.shape
    if K2 != K:
        raise ValueError("X and B disagree on K")
    _need(X, torch.bfloat16, (T, K), "X")
    _need(row_src, torch.int32, (R,), "row_src")
    _need(B, torch.bfloat16, (G, K, N), "B")
    _need(B2, torch.bfloat16, (G, K, N), "B2")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    dev = X.device
    C = torch.empty((R, N), dtype=torch.bfloat16, device=dev) if C is None else C
    if B2 is not None and C2 is None:
        C2 = torch.empty((R, N), dtype=torch.bfloat16, device=dev)
    if want_act and act is None:
        act = torch.empty((R, N), dtype=torch.bfloat16, device=dev)
    for t, n in ((C, "C"), (C2, "C2"), (act, "act")):
        _need(t, torch.bfloat16, (R, N), n)
    st = lib().moe_grouped_gemm_fwd_gather(_ptr(X), T, _ptr(row_src), _ptr(B), _ptr(B2), _ptr(offsets), G, R, K, N,
                                           _ptr(C), _ptr(C2), _ptr(act), _ptr(workspace),
                                           0 if workspace is None else workspace.numel(), _stream(stream))
    _check("moe_grouped_gemm_fwd_gather", st)
    return C, C2, act


def moe_gather_rows(x, row_of_slot, k, x_perm=None, stream=None):
    """x_perm[row_of_slot[t*k + j]] = x[t] (the gather step alone)."""
    T, d = x.shape
    _need(x, torch.bfloat16, (T, d), "x")
    _need(row_of_slot, torch.int32, (T * k,), "row_of_slot")
    x_perm = torch.empty((T * k, d), dtype=torch.bfloat16, device=x.device) if x_perm is None else x_perm
    _need(x_perm, torch.bfloat16, (T * k, d), "x_perm")
    _check("moe_gather_rows", lib().moe_gather_rows(_ptr(x), T, d, k, _ptr(row_of_slot), _ptr(x_perm),
                                                    _stream(stream)))
    return x_perm


def moe_quantize_fp8_rows(x, q=None, scale=None, stream=None):
    """Per-row E4M3 codes (uint8) and fp32 scales of the rows of x (any leading shape)."""
    K = x.shape[-1]
    M = x.numel() // K
    if x.dtype != torch.bfloat16 or not x.is_contiguous():
        raise ValueError("x must be a contiguous bf16 tensor")
    q = torch.empty(x.shape, dtype=torch.uint8, device=x.device) if q is None else q
    scale = torch.empty(x.shape[:-1], dtype=torch.float32, device=x.device) if scale is None else scale
    _need(q, torch.uint8, tuple(x.shape), "q")
    _need(scale, torch.float32, tuple(x.shape[:-1]), "scale")
    _check("moe_quantize_fp8_rows", lib().moe_quantize_fp8_rows(_ptr(x), M, K, _ptr(q), _ptr(scale), _stream(stream)))
    return q, scale


def moe_quantize_fp8_rows2(x, x2, q=None, scale=None, stream=None):
    """E4M3 codes [.., 2K] and fp32 scales of the rows [x | x2] (x and x2 of one shape [.., K]), one
    scale per joined row."""
    K = x.shape[-1]
    M = x.numel() // K
    for t, n in ((x, "x"), (x2, "x2")):
        if t.dtype != torch.bfloat16 or not t.is_contiguous():
            raise ValueError(f"{n} must be a contiguous bf16 tensor")
    if tuple(x2.shape) != tuple(x.shape):
        raise ValueError("x and x2 must have one shape")
    qshape = tuple(x.shape[:-1]) + (2 * K,)
    q = torch.empty(qshape, dtype=torch.uint8, device=x.device) if q is None else q
    scale = torch.empty(x.shape[:-1], dtype=torch.float32, device=x.device) if scale is None else scale
    _need(q, torch.uint8, qshape, "q")
    _need(scale, torch.float32, tuple(x.shape[:-1]), "scale")
    _check("moe_quantize_fp8_rows2",
           lib().moe_quantize_fp8_rows2(_ptr(x), _ptr(x2), M, K, _ptr(q), _ptr(scale), _stream(stream)))
    return q, scale


def moe_quantize_fp8_weight(w, w2=None, q=None, scale=None, stream=None):
    """E4M3 codes and per-channel scales of a weight [G, K, N] (contraction K, channels N), written
    as [G, N, K] (or, with w2, [G, 2N, K] with the two weights' channels interleaved by 128)."""
    G, K, N = w.shape
    _need(w, torch.bfloat16, (G, K, N), "w")
    _need(w2, torch.bfloat16, (G, K, N), "w2")
    if not w.is_contiguous() or (w2 is not None and not w2.is_contiguous()):
        raise ValueError("w and w2 must be contiguous")
    n_out = 2 * N if w2 is not None else N
    q = torch.empty((G, n_out, K), dtype=torch.uint8, device=w.device) if q is None else q
    scale = torch.empty((G, n_out), dtype=torch.float32, device=w.device) if scale is None else scale
    _need(q, torch.uint8, (G, n_out, K), "q")
    _need(scale, torch.float32, (G, n_out), "scale")
    _check("moe_quantize_fp8_weight",
           lib().moe_quantize_fp8_weight(_ptr(w), _ptr(w2), G, K, N, _ptr(q), _ptr(scale), _stream(stream)))
    return q, scale


def moe_grouped_gemm_fwd_fp8(A, a_scale, Wt, w_scale, offsets, C=None, stream=None, workspace=None):
    """C = (A . Wt[g]^T) * a_scale * w_scale per group, bf16; A [R,K] and Wt [G,N,K] E4M3 codes."""
    R, K = A.shape
    G, N, K2 = Wt.shape
    if K2 != K:
        raise ValueError("A and Wt disagree on K")
    _need(A, torch.uint8, (R, K), "A")
    _need(a_scale, torch.float32, (R,), "a_scale")
    _need(Wt, torch.uint8, (G, N, K), "Wt")
    _need(w_scale, torch.float32, (G, N), "w_scale")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    C = torch.empty((R, N), dtype=torch.bfloat16, device=A.device) if C is None else C
    _need(C, torch.bfloat16, (R, N), "C")
    st = lib().moe_grouped_gemm_fwd_fp8(_ptr(A), _ptr(a_scale), _ptr(Wt), _ptr(w_scale), _ptr(offsets), G, R, K, N,
                                        _ptr(C), _ptr(workspace), 0 if workspace is None else workspace.numel(),
                                        _stream(stream))
    _check("moe_grouped_gemm_fwd_fp8", st)
    return C


def moe_grouped_gemm_dx_swiglu_bwd_fp8(A, a_scale, Wt, w_scale, offsets, h_gate, h_up, dh_gate=None, dh_up=None,
                                       stream=None, workspace=None):
    """dA = (A . Wt[g]^T) * a_scale * w_scale (bf16) and its SwiGLU backward: (dh_gate, dh_up) from
    h_gate, h_up [R, N]; A [R, K] and Wt [G, N, K] E4M3 codes."""
    R, K = A.shape
    G, N, K2 = Wt.shape
    if K2 != K:
        raise ValueError("A and Wt disagree on K")
    _need(A, torch.uint8, (R, K), "A")
    _need(a_scale, torch.float32, (R,), "a_scale")
    _need(Wt, torch.uint8, (G, N, K), "Wt")
    _need(w_scale, torch.float32, (G, N), "w_scale")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    _need(h_gate, torch.bfloat16, (R, N), "h_gate")
    _need(h_up, torch.bfloat16, (R, N), "h_up")
    dh_gate = torch.empty((R, N), dtype=torch.bfloat16, device=A.device) if dh_gate is None else dh_gate
    dh_up = torch.empty((R, N), dtype=torch.bfloat16, device=A.device) if dh_up is None else dh_up
    _need(dh_gate, torch.bfloat16, (R, N), "dh_gate")
    _need(dh_up, torch.bfloat16, (R, N), "dh_up")
    st = lib().moe_grouped_gemm_dx_swiglu_bwd_fp8(_ptr(A), _ptr(a_scale), _ptr(Wt), _ptr(w_scale), _ptr(offsets), G,
                                                  R, K, N, _ptr(h_gate), _ptr(h_up), _ptr(dh_gate), _ptr(dh_up),
                                                  _ptr(workspace), 0 if workspace is None else workspace.numel(),
                                                  _stream(stream))
    _check("moe_grouped_gemm_dx_swiglu_bwd_fp8", st)
    return dh_gate, dh_up


def interleave_gate_up(w_gate_t, w_up_t):
    """[G, F, K] gate and up weights (output channel, contraction) -> [G, 2F, K] with the channels
    interleaved by 128 (rows 256t .. 256t+127: gate channels 128t ..; the next 128: up channels),
    the layout moe_grouped_gemm_fwd_fp8_gate_up reads (a one-off weight preparation)."""
    G, F, K = w_gate_t.shape
    if F % 128:
        raise ValueError("F must be a multiple of 128")
    g = w_gate_t.reshape(G, F // 128, 128, K)
    u = w_up_t.reshape(G, F // 128, 128, K)
    return torch.cat([g, u], dim=2).reshape(G, 2 * F, K).contiguous()


def moe_grouped_gemm_fwd_fp8_gate_up(A, a_scale, Wt_gu, w_scale_gu, offsets, h_gate=None, h_up=None, act=None,
                                     want_act=True, stream=None, workspace=None):
    """Gate and up projections from one E4M3 weight interleaved by 128 channels, + SwiGLU."""
    R, K = A.shape
    G, F2, K2 = Wt_gu.shape
    if K2 != K or F2 % 256:
        raise ValueError("bad shapes")
    F = F2 // 2
    _need(A, torch.uint8, (R, K), "A")
    _need(a_scale, torch.float32, (R,), "a_scale")
    _need(Wt_gu, torch.uint8, (G, F2, K), "Wt_gu")
    _need(w_scale_gu, torch.float32, (G, F2), "w_scale_gu")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    dev = A.device
    h_gate = torch.empty((R, F), dtype=torch.bfloat16, device=dev) if h_gate is None else h_gate
    h_up = torch.empty((R, F), dtype=torch.bfloat16, device=dev) if h_up is None else h_up
    if want_act and act is None:
        act = torch.empty((R, F), dtype=torch.bfloat16, device=dev)
    for t, n in ((h_gate, "h_gate"), (h_up, "h_up"), (act, "act")):
        _need(t, torch.bfloat16, (R, F), n)
    st = lib().moe_grouped_gemm_fwd_fp8_gate_up(_ptr(A), _ptr(a_scale), _ptr(Wt_gu), _ptr(w_scale_gu), _ptr(offsets),
                                                G, R, K, F, _ptr(h_gate), _ptr(h_up), _ptr(act), _ptr(workspace),
                                                0 if workspace is None else workspace.numel(), _stream(stream))
    _check("moe_grouped_gemm_fwd_fp8_gate_up", st)
    return h_gate, h_up, act


def mx_groups(C):
    """128-element scale groups of a row of C elements (the leading extent of an MX scale array)."""
    return (C + 127) // 128


def mx_scales_by_row(s, C):
    """An MX scale array [groups, *rows, 4] (the library's layout) as [*rows, C/32]: block b of a row
    in column b (a view-and-copy for inspection and tests; the kernels read the first form)."""
    t = s.movedim(0, -2)
    return t.reshape(t.shape[:-2] + (t.shape[-2] * 4,))[..., : C // 32].contiguous()


def mx_scales_from_rows(sb, C, pad=0):
    """[*rows, C/32] scale bytes -> the library's MX scale array [groups, *rows, 4] (padding bytes
    set to `pad`)."""
    P = mx_groups(C)
    out = torch.full(sb.shape[:-1] + (4 * P,), pad, dtype=torch.uint8, device=sb.device)
    out[..., : C // 32] = sb
    return out.reshape(sb.shape[:-1] + (P, 4)).movedim(-2, 0).contiguous()


def moe_quantize_mx_rows(x, x2=None, q=None, scale=None, stream=None):
    """MX codes [.., C] and E8M0 block scales (the MX scale layout, [ceil(C/128), .., 4]) of the rows
    of x, or of the joined rows [x | x2] (C = 2K) when x2 is given."""
    K = x.shape[-1]
    M = x.numel() // K
    for t, n in ((x, "x"), (x2, "x2")):
        if t is not None and (t.dtype != torch.bfloat16 or not t.is_contiguous()):
            raise ValueError(f"{n} must be a contiguous bf16 tensor")
    if x2 is not None and tuple(x2.shape) != tuple(x.shape):
        raise ValueError("x and x2 must have one shape")
    C = 2 * K if x2 is not None else K
    qshape = tuple(x.shape[:-1]) + (C,)
    sshape = (mx_groups(C),) + tuple(x.shape[:-1]) + (4,)
    q = torch.empty(qshape, dtype=torch.uint8, device=x.device) if q is None else q
    scale = torch.empty(sshape, dtype=torch.uint8, device=x.device) if scale is None else scale
    _need(q, torch.uint8, qshape, "q")
    _need(scale, torch.uint8, sshape, "scale")
    _check("moe_quantize_mx_rows",
           lib().moe_quantize_mx_rows(_ptr(x), _ptr(x2), M, K, _ptr(q), _ptr(scale), _stream(stream)))
    return q, scale


def moe_quantize_mx_weight(w, w2=None, want_t=True, want_r=True, qt=None, st=None, qr=None, sr=None,
                           stream=None):
    """MX codes and block scales of a weight [G, K, N] in both orientations from one read:
    (qt [G, N', K], st [ceil(K/128), G, N', 4]) the forward operand (N' = 2N with w2, channels
    interleaved by 128) and (qr [G, K, N''], sr [ceil(N''/128), G, K, 4]) the data-gradient operand
    (N'' = 2N with w2: rows [W | W2]).  Returns (qt, st, qr, sr), None for an orientation not asked
    for."""
    G, K, N = w.shape
    _need(w, torch.bfloat16, (G, K, N), "w")
    _need(w2, torch.bfloat16, (G, K, N), "w2")
    if not w.is_contiguous() or (w2 is not None and not w2.is_contiguous()):
        raise ValueError("w and w2 must be contiguous")
    n2 = 2 * N if w2 is not None else N
    dev = w.device
    if want_t:
        qt = torch.empty((G, n2, K), dtype=torch.uint8, device=dev) if qt is None else qt
        st = torch.empty((mx_groups(K), G, n2, 4), dtype=torch.uint8, device=dev) if st is None else st
        _need(qt, torch.uint8, (G, n2, K), "qt")
        _need(st, torch.uint8, (mx_groups(K), G, n2, 4), "st")
    else:
        qt = st = None
    if want_r:
        qr = torch.empty((G, K, n2), dtype=torch.uint8, device=dev) if qr is None else qr
        sr = torch.empty((mx_groups(n2), G, K, 4), dtype=torch.uint8, device=dev) if sr is None else sr
        _need(qr, torch.uint8, (G, K, n2), "qr")
        _need(sr, torch.uint8, (mx_groups(n2), G, K, 4), "sr")
    else:
        qr = sr = None
    _check("moe_quantize_mx_weight",
           lib().moe_quantize_mx_weight(_ptr(w), _ptr(w2), G, K, N, _ptr(qt), _ptr(st), _ptr(qr), _ptr(sr),
                                        _stream(stream)))
    return qt, st, qr, sr


def _need_mx(A, a_scale, Wt, w_scale, offsets):
    R, K = A.shape
    G, N, K2 = Wt.shape
    if K2 != K:
        raise ValueError("A and Wt disagree on K")
    P = mx_groups(K)
    _need(A, torch.uint8, (R, K), "A")
    _need(a_scale, torch.uint8, (P, R, 4), "a_scale")
    _need(Wt, torch.uint8, (G, N, K), "Wt")
    _need(w_scale, torch.uint8, (P, G, N, 4), "w_scale")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    return R, K, G, N


def moe_grouped_gemm_fwd_mx(A, a_scale, Wt, w_scale, offsets, C=None, stream=None, workspace=None):
    """C = A . Wt[g]^T per group on MX operands (E4M3 codes with E8M0 scales per 32 of K, in the MX
    scale layout: a_scale [ceil(K/128), R, 4], w_scale [ceil(K/128), G, N, 4]), bf16."""
    R, K, G, N = _need_mx(A, a_scale, Wt, w_scale, offsets)
    C = torch.empty((R, N), dtype=torch.bfloat16, device=A.device) if C is None else C
    _need(C, torch.bfloat16, (R, N), "C")
    st = lib().moe_grouped_gemm_fwd_mx(_ptr(A), _ptr(a_scale), _ptr(Wt), _ptr(w_scale), _ptr(offsets), G, R, K, N,
                                       _ptr(C), _ptr(workspace), 0 if workspace is None else workspace.numel(),
                                       _stream(stream))
    _check("moe_grouped_gemm_fwd_mx", st)
    return C


def moe_grouped_gemm_fwd_mx_gate_up(A, a_scale, Wt_gu, w_scale_gu, offsets, h_gate=None, h_up=None, act=None,
                                    want_act=True, stream=None, workspace=None):
    """Gate and up projections on MX operands from one weight interleaved by 128 channels, + SwiGLU."""
    R, K, G, F2 = _need_mx(A, a_scale, Wt_gu, w_scale_gu, offsets)
    if F2 % 256:
        raise ValueError("bad shapes")
    F = F2 // 2
    dev = A.device
    h_gate = torch.empty((R, F), dtype=torch.bfloat16, device=dev) if h_gate is None else h_gate
    h_up = torch.empty((R, F), dtype=torch.bfloat16, device=dev) if h_up is None else h_up
    if want_act and act is None:
        act = torch.empty((R, F), dtype=torch.bfloat16, device=dev)
    for t, n in ((h_gate, "h_gate"), (h_up, "h_up"), (act, "act")):
        _need(t, torch.bfloat16, (R, F), n)
    st = lib().moe_grouped_gemm_fwd_mx_gate_up(_ptr(A), _ptr(a_scale), _ptr(Wt_gu), _ptr(w_scale_gu), _ptr(offsets),
                                               G, R, K, F, _ptr(h_gate), _ptr(h_up), _ptr(act), _ptr(workspace),
                                               0 if workspace is None else workspace.numel(), _stream(stream))
    _check("moe_grouped_gemm_fwd_mx_gate_up", st)
    return h_gate, h_up, act


def moe_grouped_gemm_dx_swiglu_bwd_mx(A, a_scale, Wt, w_scale, offsets, h_gate, h_up, dh_gate=None, dh_up=None,
                                      stream=None, workspace=None):
    """dA = A . Wt[g]^T on MX operands (bf16) and its SwiGLU backward: (dh_gate, dh_up) from
    h_gate, h_up [R, N]."""
    R, K, G, N = _need_mx(A, a_scale, Wt, w_scale, offsets)
    _need(h_gate, torch.bfloat16, (R, N), "h_gate")
    _need(h_up, torch.bfloat16, (R, N), "h_up")
    dh_gate = torch.empty((R, N), dtype=torch.bfloat16, device=A.device) if dh_gate is None else dh_gate
    dh_up = torch.empty((R, N), dtype=torch.bfloat16, device=A.device) if dh_up is None else dh_up
    _need(dh_gate, torch.bfloat16, (R, N), "dh_gate")
    _need(dh_up, torch.bfloat16, (R, N), "dh_up")
    st = lib().moe_grouped_gemm_dx_swiglu_bwd_mx(_ptr(A), _ptr(a_scale), _ptr(Wt), _ptr(w_scale), _ptr(offsets), G,
                                                 R, K, N, _ptr(h_gate), _ptr(h_up), _ptr(dh_gate), _ptr(dh_up),
                                                 _ptr(workspace), 0 if workspace is None else workspace.numel(),
                                                 _stream(stream))
    _check("moe_grouped_gemm_dx_swiglu_bwd_mx", st)
    return dh_gate, dh_up


def combine_counters(T, N, device):
    """Arrival counters for moe_grouped_gemm_fwd_combine (allocated once, zeroed by each call)."""
    n = int(lib().moe_grouped_gemm_fwd_combine_workspace_bytes(T, N))
    return torch.empty(max(16, n), dtype=torch.uint8, device=device)


def moe_grouped_gemm_fwd_combine(A, B, offsets, topk_w, row_of_slot, token_of_row, add=None, y_perm=None, y=None,
                                 counters=None, workspace=None, stream=None):
    """Down product with the weighted combine fused: (y_perm [R, N], y [T, N]) bit for bit as
    moe_grouped_gemm_fwd followed by moe_unpermute_combine."""
    R, K = A.shape
    G, K2, N = B.shape
    T, k = topk_w.shape
    if K2 != K or R != T * k:
        raise ValueError("bad shapes")
    _need(A, torch.bfloat16, (R, K), "A")
    _need(B, torch.bfloat16, (G, K, N), "B")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    _need(topk_w, torch.float32, (T, k), "topk_w")
    _need(row_of_slot, torch.int32, (R,), "row_of_slot")
    _need(token_of_row, torch.int32, (R,), "token_of_row")
    _need(add, torch.bfloat16, (T, N), "add")
    y_perm = torch.empty((R, N), dtype=torch.bfloat16, device=A.device) if y_perm is None else y_perm
    y = torch.empty((T, N), dtype=torch.bfloat16, device=A.device) if y is None else y
    _need(y_perm, torch.bfloat16, (R, N), "y_perm")
    _need(y, torch.bfloat16, (T, N), "y")
    counters = combine_counters(T, N, A.device) if counters is None else counters
    st = lib().moe_grouped_gemm_fwd_combine(_ptr(A), _ptr(B), _ptr(offsets), G, R, K, N, _ptr(topk_w),
                                            _ptr(row_of_slot), _ptr(token_of_row), T, k, _ptr(add), _ptr(y_perm),
                                            _ptr(y), _ptr(counters), counters.numel(), _ptr(workspace),
                                            0 if workspace is None else workspace.numel(), _stream(stream))
    _check("moe_grouped_gemm_fwd_combine", st)
    return y_perm, y


def mx_tokens_cols(R, G):
    """Row length of the token-major MX operands of R routed rows in G groups (a multiple of 128)."""
    return int(lib().moe_mx_tokens_cols_bound(R, G))


def moe_quantize_mx_tokens_t(x, offsets, qt=None, st=None, stream=None):
    """MX codes qt [C, ld] and scales st [ld/128, C, 4] of the routed buffer x [R, C] along its
    token axis: expert g's rows as columns from a 128-aligned start, zero codes in the padding."""
    R, C = x.shape
    G = offsets.numel() - 1
    _need(x, torch.bfloat16, (R, C), "x")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    ld = mx_tokens_cols(R, G)
    qt = torch.empty((C, ld), dtype=torch.uint8, device=x.device) if qt is None else qt
    st = torch.empty((ld // 128, C, 4), dtype=torch.uint8, device=x.device) if st is None else st
    _need(qt, torch.uint8, (C, ld), "qt")
    _need(st, torch.uint8, (ld // 128, C, 4), "st")
    _check("moe_quantize_mx_tokens_t", lib().moe_quantize_mx_tokens_t(_ptr(x), _ptr(offsets), G, R, C, _ptr(qt),
                                                                      _ptr(st), ld, _stream(stream)))
    return qt, st


def moe_quantize_mx_tokens(x, offsets, qt=None, st=None, qr=None, sr=None, ldr=None, col0=0, want_t=True,
                           want_r=True, stream=None):
    """Both MX orientations of the routed buffer x [R, C] from one read: token-major (qt [C, ld],
    st [ld/128, C, 4]) and row-wise codes written at column col0 of rows of ldr bytes (qr [R, ldr],
    sr [ceil(ldr/128), R, 4]; ldr defaults to C).  Returns (qt, st, qr, sr), None where not asked."""
    R, C = x.shape
    G = offsets.numel() - 1
    _need(x, torch.bfloat16, (R, C), "x")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    ld = mx_tokens_cols(R, G)
    dev = x.device
    if want_t:
        qt = torch.empty((C, ld), dtype=torch.uint8, device=dev) if qt is None else qt
        st = torch.empty((ld // 128, C, 4), dtype=torch.uint8, device=dev) if st is None else st
        _need(qt, torch.uint8, (C, ld), "qt")
        _need(st, torch.uint8, (ld // 128, C, 4), "st")
    else:
        qt = st = None
    if want_r:
        ldr = (qr.shape[1] if qr is not None else C) if ldr is None else ldr
        qr = torch.empty((R, ldr), dtype=torch.uint8, device=dev) if qr is None else qr
        sr = torch.empty((mx_groups(ldr), R, 4), dtype=torch.uint8, device=dev) if sr is None else sr
        _need(qr, torch.uint8, (R, ldr), "qr")
        _need(sr, torch.uint8, (mx_groups(ldr), R, 4), "sr")
    else:
        qr = sr = None
        ldr = 0
    _check("moe_quantize_mx_tokens", lib().moe_quantize_mx_tokens(_ptr(x), _ptr(offsets), G, R, C, _ptr(qt), _ptr(st),
                                                                  ld, _ptr(qr), _ptr(sr), ldr, col0, _stream(stream)))
    return qt, st, qr, sr


def moe_grouped_gemm_dw_mx(At, a_scale, dCt, c_scale, offsets, R, dC2t=None, c2_scale=None, dB=None, dB2=None,
                           out_bf16=False, counters=None, stream=None):
    """The weight gradient on token-major MX operands (moe_quantize_mx_tokens_t): dB [G, K, N]
    (dB2 from dC2t), fp32 or bf16; with counters (dw_counters), a persistent grid claiming tiles."""
    K, ld = At.shape
    N = dCt.shape[0]
    G = offsets.numel() - 1
    _need(At, torch.uint8, (K, ld), "At")
    _need(a_scale, torch.uint8, (ld // 128, K, 4), "a_scale")
    _need(dCt, torch.uint8, (N, ld), "dCt")
    _need(c_scale, torch.uint8, (ld // 128, N, 4), "c_scale")
    _need(dC2t, torch.uint8, (N, ld), "dC2t")
    _need(c2_scale, torch.uint8, (ld // 128, N, 4), "c2_scale")
    dt = torch.bfloat16 if out_bf16 else torch.float32
    dB = torch.empty((G, K, N), dtype=dt, device=At.device) if dB is None else dB
    _need(dB, dt, (G, K, N), "dB")
    if dC2t is not None:
        dB2 = torch.empty((G, K, N), dtype=dt, device=At.device) if dB2 is None else dB2
        _need(dB2, dt, (G, K, N), "dB2")
    _check("moe_grouped_gemm_dw_mx",
           lib().moe_grouped_gemm_dw_mx(_ptr(At), _ptr(a_scale), _ptr(dCt), _ptr(c_scale), _ptr(dC2t), _ptr(c2_scale),
                                        _ptr(offsets), G, R, K, N, ld, _ptr(dB), _ptr(dB2) if dC2t is not None else None,
                                        int(out_bf16), _ptr(counters), _stream(stream)))
    return (dB, dB2) if dC2t is not None else dB


def moe_swiglu(h_gate, h_up, act=None, stream=None):
    rows, f = h_gate.shape
    _need(h_gate, torch.bfloat16, (rows, f), "h_gate")
    _need(h_up, torch.bfloat16, (rows, f), "h_up")
    act = torch.empty_like(h_gate) if act is None else act
    _need(act, torch.bfloat16, (rows, f), "act")
    _check("moe_swiglu", lib().moe_swiglu(_ptr(h_gate), _ptr(h_up), _ptr(act), rows, f, _stream(stream)))
    return act


def moe_swiglu_bwd(h_gate, h_up, d_act, dh_gate=None, dh_up=None, stream=None):
    rows, f = h_gate.shape
    for t, n in ((h_gate, "h_gate"), (h_up, "h_up"), (d_act, "d_act")):
        _need(t, torch.bfloat16, (rows, f), n)
    dh_gate = torch.empty_like(h_gate) if dh_gate is None else dh_gate
    dh_up = torch.empty_like(h_gate) if dh_up is None else dh_up
    _need(dh_gate, torch.bfloat16, (rows, f), "dh_gate")
    _need(dh_up, torch.bfloat16, (rows, f), "dh_up")
    _check("moe_swiglu_bwd", lib().moe_swiglu_bwd(_ptr(h_gate), _ptr(h_up), _ptr(d_act), _ptr(dh_gate),
                                                  _ptr(dh_up), rows, f, _stream(stream)))
    return dh_gate, dh_up


def moe_unpermute_combine(y_perm, topk_w, row_of_slot, k, add=None, y=None, stream=None):
    R, d = y_perm.shape
    T = R // k
    _need(y_perm, torch.bfloat16, (T * k, d), "y_perm")
    _need(topk_w, torch.float32, (T, k), "topk_w")
    _need(row_of_slot, torch.int32, (R,), "row_of_slot")
    _need(add, torch.bfloat16, (T, d), "add")
    y = torch.empty((T, d), dtype=torch.bfloat16, device=y_perm.device) if y is None else y
    _need(y, torch.bfloat16, (T, d), "y")
    _check("moe_unpermute_combine",
           lib().moe_unpermute_combine(_ptr(y_perm), _ptr(topk_w), _ptr(row_of_slot), _ptr(add), T, d, k,
                                       _ptr(y), _stream(stream)))
    return y


def moe_unpermute_router_dx(dx_perm, row_of_slot, k, dlogits, wr, add=None, dx=None, stream=None):
    R, d = dx_perm.shape
    T = R // k
    E = wr.shape[1]
    _need(dx_perm, torch.bfloat16, (T * k, d), "dx_perm")
    _need(row_of_slot, torch.int32, (R,), "row_of_slot")
    _need(add, torch.bfloat16, (T, d), "add")
    _need(dlogits, torch.float32, (T, E), "dlogits")
    _need(wr, torch.float32, (d, E), "wr")
    dx = torch.empty((T, d), dtype=torch.bfloat16, device=dx_perm.device) if dx is None else dx
    _need(dx, torch.bfloat16, (T, d), "dx")
    _check("moe_unpermute_router_dx",
           lib().moe_unpermute_router_dx(_ptr(dx_perm), _ptr(row_of_slot), _ptr(add), _ptr(dlogits), _ptr(wr),
                                         T, d, k, E, _ptr(dx), _stream(stream)))
    return dx


def moe_unpermute_combine_bwd(dy, topk_w, row_of_slot, k, y_perm=None, dy_perm=None, d_topk_w=None,
                              stream=None):
    T, d = dy.shape
    _need(dy, torch.bfloat16, (T, d), "dy")
    _need(topk_w, torch.float32, (T, k), "topk_w")
    _need(row_of_slot, torch.int32, (T * k,), "row_of_slot")
    _need(y_perm, torch.bfloat16, (T * k, d), "y_perm")
    dy_perm = torch.empty((T * k, d), dtype=torch.bfloat16, device=dy.device) if dy_perm is None else dy_perm
    if y_perm is not None and d_topk_w is None:
        d_topk_w = torch.empty((T, k), dtype=torch.float32, device=dy.device)
    _need(dy_perm, torch.bfloat16, (T * k, d), "dy_perm")
    _need(d_topk_w, torch.float32, (T, k), "d_topk_w")
    _check("moe_unpermute_combine_bwd",
           lib().moe_unpermute_combine_bwd(_ptr(dy), _ptr(topk_w), _ptr(row_of_slot), _ptr(y_perm), T, d, k,
                                           _ptr(dy_perm), _ptr(d_topk_w), _stream(stream)))
    return dy_perm, d_topk_w


def split_workspace(device):
    """A workspace for the split-tail variants of the fwd and persistent dX products and of the
    single-group persistent dW."""
    return torch.empty(lib().moe_grouped_gemm_split_workspace_bytes(), dtype=torch.uint8, device=device)


def moe_grouped_gemm_dx(dC, B, offsets, dC2=None, B2=None, dA=None, stream=None, workspace=None):
    R, N = dC.shape
    G, K, N2 = B.shape
    if N2 != N:
        raise ValueError("dC and B disagree on N")
    _need(dC, torch.bfloat16, (R, N), "dC")
    _need(dC2, torch.bfloat16, (R, N), "dC2")
    _need(B, torch.bfloat16, (G, K, N), "B")
    _need(B2, torch.bfloat16, (G, K, N), "B2")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    dA = torch.empty((R, K), dtype=torch.bfloat16, device=dC.device) if dA is None else dA
    _need(dA, torch.bfloat16, (R, K), "dA")
    if workspace is None:
        _check("moe_grouped_gemm_dx",
               lib().moe_grouped_gemm_dx(_ptr(dC), _ptr(B), _ptr(dC2), _ptr(B2), _ptr(offsets), G, R, K, N,
                                         _ptr(dA), _stream(stream)))
    else:
        _check("moe_grouped_gemm_dx_split",
               lib().moe_grouped_gemm_dx_split(_ptr(dC), _ptr(B), _ptr(dC2), _ptr(B2), _ptr(offsets), G, R, K, N,
                                               _ptr(dA), _ptr(workspace), workspace.numel(), _stream(stream)))
    return dA


def dw_counters(device):
    """Claim counters for the persistent dW entry points (8 int32; each call zeroes them)."""
    return torch.zeros(8, dtype=torch.int32, device=device)


def moe_grouped_gemm_dw(A, dC, offsets, dC2=None, dB=None, dB2=None, stream=None, counters=None, workspace=None):
    """dB[g] = A_g^T dC_g (and dB2 from dC2) in fp32.  counters (from dw_counters): run the
    persistent entry point, which hands out tiles through them (bit-identical results); with a
    split workspace as well (split_workspace), moe_grouped_gemm_dw_split, which splits a single
    group's last-round tiles along the contraction."""
    R, K = A.shape
    N = dC.shape[1]
    G = offsets.numel() - 1
    _need(A, torch.bfloat16, (R, K), "A")
    _need(dC, torch.bfloat16, (R, N), "dC")
    _need(dC2, torch.bfloat16, (R, N), "dC2")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    dB = torch.empty((G, K, N), dtype=torch.float32, device=A.device) if dB is None else dB
    if dC2 is not None and dB2 is None:
        dB2 = torch.empty((G, K, N), dtype=torch.float32, device=A.device)
    _need(dB, torch.float32, (G, K, N), "dB")
    _need(dB2, torch.float32, (G, K, N), "dB2")
    if workspace is not None and counters is None:
        raise ValueError("moe_grouped_gemm_dw: a split workspace needs counters (the persistent form)")
    if counters is not None:
        _need(counters, torch.int32, (8,), "counters")
        if workspace is not None:
            _check("moe_grouped_gemm_dw_split",
                   lib().moe_grouped_gemm_dw_split(_ptr(A), _ptr(dC), _ptr(dC2), _ptr(offsets), G, R, K, N,
                                                   _ptr(dB), _ptr(dB2), _ptr(counters), _ptr(workspace),
                                                   workspace.numel(), _stream(stream)))
            return dB, dB2
        _check("moe_grouped_gemm_dw_persistent",
               lib().moe_grouped_gemm_dw_persistent(_ptr(A), _ptr(dC), _ptr(dC2), _ptr(offsets), G, R, K, N,
                                                    _ptr(dB), _ptr(dB2), _ptr(counters), _stream(stream)))
        return dB, dB2
    _check("moe_grouped_gemm_dw",
           lib().moe_grouped_gemm_dw(_ptr(A), _ptr(dC), _ptr(dC2), _ptr(offsets), G, R, K, N, _ptr(dB),
                                     _ptr(dB2), _stream(stream)))
    return dB, dB2


def moe_grouped_gemm_dw_bf16(A, dC, offsets, dC2=None, dB=None, dB2=None, stream=None, counters=None):
    """moe_grouped_gemm_dw with bf16 results (one rounding of the fp32 sum); counters as there."""
    R, K = A.shape
    N = dC.shape[1]
    G = offsets.numel() - 1
    _need(A, torch.bfloat16, (R, K), "A")
    _need(dC, torch.bfloat16, (R, N), "dC")
    _need(dC2, torch.bfloat16, (R, N), "dC2")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    dB = torch.empty((G, K, N), dtype=torch.bfloat16, device=A.device) if dB is None else dB
    if dC2 is not None and dB2 is None:
        dB2 = torch.empty((G, K, N), dtype=torch.bfloat16, device=A.device)
    _need(dB, torch.bfloat16, (G, K, N), "dB")
    _need(dB2, torch.bfloat16, (G, K, N), "dB2")
    if counters is not None:
        _need(counters, torch.int32, (8,), "counters")
        _check("moe_grouped_gemm_dw_bf16_persistent",
               lib().moe_grouped_gemm_dw_bf16_persistent(_ptr(A), _ptr(dC), _ptr(dC2), _ptr(offsets), G, R, K,
                                                         N, _ptr(dB), _ptr(dB2), _ptr(counters), _stream(stream)))
        return dB, dB2
    _check("moe_grouped_gemm_dw_bf16",
           lib().moe_grouped_gemm_dw_bf16(_ptr(A), _ptr(dC), _ptr(dC2), _ptr(offsets), G, R, K, N, _ptr(dB),
                                          _ptr(dB2), _stream(stream)))
    return dB, dB2


def moe_grouped_gemm_dx_swiglu_bwd(dC, B, offsets, h_gate, h_up, dh_gate=None, dh_up=None, stream=None,
                                   workspace=None):
    R, N = dC.shape
    G, K, N2 = B.shape
    if N2 != N:
        raise ValueError("dC and B disagree on N")
    _need(dC, torch.bfloat16, (R, N), "dC")
    _need(B, torch.bfloat16, (G, K, N), "B")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    _need(h_gate, torch.bfloat16, (R, K), "h_gate")
    _need(h_up, torch.bfloat16, (R, K), "h_up")
    dh_gate = torch.empty((R, K), dtype=torch.bfloat16, device=dC.device) if dh_gate is None else dh_gate
    dh_up = torch.empty((R, K), dtype=torch.bfloat16, device=dC.device) if dh_up is None else dh_up
    _need(dh_gate, torch.bfloat16, (R, K), "dh_gate")
    _need(dh_up, torch.bfloat16, (R, K), "dh_up")
    if workspace is None:
        _check("moe_grouped_gemm_dx_swiglu_bwd",
               lib().moe_grouped_gemm_dx_swiglu_bwd(_ptr(dC), _ptr(B), _ptr(offsets), G, R, K, N, _ptr(h_gate),
                                                    _ptr(h_up), _ptr(dh_gate), _ptr(dh_up), _stream(stream)))
    else:
        _check("moe_grouped_gemm_dx_swiglu_bwd_split",
               lib().moe_grouped_gemm_dx_swiglu_bwd_split(_ptr(dC), _ptr(B), _ptr(offsets), G, R, K, N,
                                                          _ptr(h_gate), _ptr(h_up), _ptr(dh_gate), _ptr(dh_up),
                                                          _ptr(workspace), workspace.numel(), _stream(stream)))
    return dh_gate, dh_up


def moe_router_logits(x, wr, bias=None, logits=None, stream=None):
    """logits [T, E] fp32 = x [T, d] bf16 . wr [d, E] fp32 (+ bias [E])."""
    T, d = x.shape
    E = wr.shape[1]
    _need(x, torch.bfloat16, (T, d), "x")
    _need(wr, torch.float32, (d, E), "wr")
    _need(bias, torch.float32, (E,), "bias")
    logits = torch.empty((T, E), dtype=torch.float32, device=x.device) if logits is None else logits
    _need(logits, torch.float32, (T, E), "logits")
    _check("moe_router_logits", lib().moe_router_logits(_ptr(x), _ptr(wr), _ptr(bias), T, d, E, _ptr(logits),
                                                        _stream(stream)))
    return logits


def moe_router_bwd(x, wr, logits, topk_idx, topk_w, d_topk_w, offsets=None, normalize_topk=True,
                   aux_alpha=0.0, dx=None, workspace=None, dlogits=None, dwr=None, stream=None):
    """Router backward: returns (dlogits [T, E], dwr [d, E]); adds the router's share into dx
    [T, d] bf16 in place when dx is given."""
    T, d = x.shape
    E = wr.shape[1]
    k = topk_idx.shape[1]
    _need(x, torch.bfloat16, (T, d), "x")
    _need(wr, torch.float32, (d, E), "wr")
    _need(logits, torch.float32, (T, E), "logits")
    _need(topk_idx, torch.int32, (T, k), "topk_idx")
    _need(topk_w, torch.float32, (T, k), "topk_w")
    _need(d_topk_w, torch.float32, (T, k), "d_topk_w")
    _need(offsets, torch.int32, (E + 1,), "offsets")
    _need(dx, torch.bfloat16, (T, d), "dx")
    dev = x.device
    dlogits = torch.empty((T, E), dtype=torch.float32, device=dev) if dlogits is None else dlogits
    dwr = torch.empty((d, E), dtype=torch.float32, device=dev) if dwr is None else dwr
    _need(dlogits, torch.float32, (T, E), "dlogits")
    _need(dwr, torch.float32, (d, E), "dwr")
    nbytes = lib().moe_router_bwd_workspace_bytes(T, d, E)
    if workspace is None:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    _check("moe_router_bwd",
           lib().moe_router_bwd(_ptr(x), _ptr(wr), _ptr(logits), _ptr(topk_idx), _ptr(topk_w), _ptr(d_topk_w),
                                _ptr(offsets), T, d, E, k, 1 if normalize_topk else 0, float(aux_alpha),
                                _ptr(workspace), workspace.numel(), _ptr(dlogits), _ptr(dwr), _ptr(dx),
                                _stream(stream)))
    return dlogits, dwr


def moe_router_aux_loss(logits, offsets, k, alpha, loss=None, workspace=None, stream=None):
    """Load-balancing loss alpha * E * sum_e f_e * P_e as a one-element fp32 tensor."""
    T, E = logits.shape
    _need(logits, torch.float32, (T, E), "logits")
    _need(offsets, torch.int32, (E + 1,), "offsets")
    dev = logits.device
    loss = torch.empty(1, dtype=torch.float32, device=dev) if loss is None else loss
    nbytes = lib().moe_router_aux_loss_workspace_bytes(T, E)
    if workspace is None:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    _check("moe_router_aux_loss",
           lib().moe_router_aux_loss(_ptr(logits), _ptr(offsets), T, E, k, float(alpha), _ptr(workspace),
                                     workspace.numel(), _ptr(loss), _stream(stream)))
    return loss


def transposed_cols(R, G):
    """Row length (a multiple of 64) of a contraction-major copy of R grouped rows in G groups."""
    b = lib().moe_transposed_cols_bound(R, G)
    return (b + 63) // 64 * 64


def moe_transpose_grouped(src, offsets, dst=None, stream=None):
    """dst [C, ld] bf16: the contraction-major, group-padded copy of src [R, C]."""
    R, C = src.shape
    G = offsets.numel() - 1
    _need(src, torch.bfloat16, (R, C), "src")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    ld = transposed_cols(R, G)
    dst = torch.empty((C, ld), dtype=torch.bfloat16, device=src.device) if dst is None else dst
    _need(dst, torch.bfloat16, (C, ld), "dst")
    _check("moe_transpose_grouped", lib().moe_transpose_grouped(_ptr(src), _ptr(offsets), G, R, C, _ptr(dst), ld,
                                                                _stream(stream)))
    return dst


def moe_grouped_gemm_dw_t(At, dCt, offsets, R, dC2t=None, dB=None, dB2=None, out_bf16=False, stream=None):
    """moe_grouped_gemm_dw from contraction-major copies At [K, ld], dCt (dC2t) [N, ld]."""
    K, ld = At.shape
    N = dCt.shape[0]
    G = offsets.numel() - 1
    _need(At, torch.bfloat16, (K, ld), "At")
    _need(dCt, torch.bfloat16, (N, ld), "dCt")
    _need(dC2t, torch.bfloat16, (N, ld), "dC2t")
    _need(offsets, torch.int32, (G + 1,), "offsets")
    dt = torch.bfloat16 if out_bf16 else torch.float32
    dB = torch.empty((G, K, N), dtype=dt, device=At.device) if dB is None else dB
    if dC2t is not None and dB2 is None:
        dB2 = torch.empty((G, K, N), dtype=dt, device=At.device)
    _need(dB, dt, (G, K, N), "dB")
    _need(dB2, dt, (G, K, N), "dB2")
    _check("moe_grouped_gemm_dw_t",
           lib().moe_grouped_gemm_dw_t(_ptr(At), _ptr(dCt), _ptr(dC2t), _ptr(offsets), G, R, K, N, ld, _ptr(dB),
                                       _ptr(dB2), 1 if out_bf16 else 0, _stream(stream)))
    return dB, dB2
