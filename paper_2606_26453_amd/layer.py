"""The MoE expert-FFN training layer as a fixed sequence of library calls on one stream.

Forward:  [router_logits ->] route_permute [-> router_aux_loss] -> grouped_gemm_fwd (gate/up +
          fused SwiGLU) -> grouped_gemm_fwd (down) [-> shared FFN as one-group calls]
          -> unpermute_combine.
Backward: unpermute_combine_bwd (weighted dY permute + d_topk_w) -> grouped_gemm_dx (down)
          -> grouped_gemm_dw (down) -> swiglu_bwd -> grouped_gemm_dx (gate+up in one contraction)
          -> grouped_gemm_dw (gate+up in one pass) [-> shared FFN backward]
          -> unpermute_combine (unweighted sum of dX_perm + shared dX) [-> router_bwd: dlogits, dWr,
          and the router's share added into dX].  The bracketed router calls run with router=True;
          otherwise the layer starts from the given logits, as the measured hot path does.

All buffers are allocated once (torch owns device memory); a step only enqueues kernels, with no
host synchronization.
"""
from __future__ import annotations

import torch

from . import moe


class _Traced:
    """Optional per-call timing: when `trace` is a list, each library call is bracketed by two
    events recorded on the stream the call is enqueued on, and (name, start, end) is appended."""

    trace = None

    def _run(self, name, fn, *args, stream=None, **kw):
        if self.trace is None:
            return fn(*args, stream=stream, **kw)
        st = torch.cuda.current_stream() if stream is None else stream
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(st)
        out = fn(*args, stream=stream, **kw)
        e1.record(st)
        self.trace.append((name, e0, e1))
        return out

    graph = None

    def capture(self, fn=None):
        """Record one call of `fn` (default: step) into a HIP graph (torch.cuda.CUDAGraph) and keep
        it; replay() then re-issues the whole sequence with one launch.  Every library call of a step
        can be captured: it only enqueues kernels on the current stream (counters and workspaces are
        cleared by kernels, never by a memset), synchronizes nothing and allocates nothing, and the
        layer's buffers are allocated once, so each replay rewrites them exactly as an eager call
        does.  One warm-up call runs on a side stream first, as torch's capture recipe asks."""
        if getattr(self, "concurrent", False):
            raise ValueError("capture the one-stream schedule (concurrent=False)")
        if self.trace is not None:
            raise ValueError("capture without per-call tracing")
        fn = self.step if fn is None else fn
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        self.graph = g
        return g

    def replay(self):
        """Re-issue the captured sequence on the current stream."""
        self.graph.replay()


class MoELayer(_Traced):
    """fuse_swiglu_bwd: the down projection's dX GEMM computes the SwiGLU backward in its epilogue
    (moe_grouped_gemm_dx_swiglu_bwd) instead of storing dA for a separate moe_swiglu_bwd pass;
    dA is then not materialised (buf["d_act"] / buf["d_act_sh"] stay unwritten)."""

    def __init__(self, cfg, inputs: dict, normalize_topk: bool = True, fuse_swiglu_bwd: bool = True,
                 router: bool = False, aux_alpha: float = 0.0, dw_transposed: bool = False,
                 concurrent: bool = False, split_tail: bool = True, gather_fused: bool = False,
                 fp8_forward: bool = False, dw_persistent: bool = True, fp8_requantize: bool = True,
                 fp8_backward: bool = False, mx: bool = False, combine_fused: bool = False,
                 fp8_dw: bool = False):
        self.cfg = cfg
        # fp8_forward: the routed experts' forward products run on E4M3 operands (activations
        # quantized per row each step, weights per output channel once, here): gate and up in one
        # product over their 128-channel-interleaved weights with the SwiGLU in its epilogue, then
        # the down product on the quantized SwiGLU output; everything else (shared FFN, backward)
        # stays bf16
        self.fp8 = fp8_forward
        # fp8_backward: the routed experts' two data-gradient products run on E4M3 operands: dY_perm
        # per row against the down weight per output channel (its stored [f, d] rows), with the
        # SwiGLU backward in the epilogue; then [dH_gate | dH_up] per row against [W_gate | W_up]
        # per output channel (rows of the stored [d, f] weights joined along f), one product over
        # the 2f-long contraction.  The weight gradients stay bf16 (their contraction runs over the
        # tokens, which a per-row or per-channel scale cannot factor out)
        self.fp8_bwd = fp8_backward
        # mx: those E4M3 products take MX block scales instead (a power of two per 32 contraction
        # elements of every row of either operand, applied by the matrix cores): activations are
        # quantized per 32-element block of their rows, and each weight is read once per step for
        # both the forward and the data-gradient orientation (moe_quantize_mx_weight)
        if mx and not (fp8_forward or fp8_backward):
            raise ValueError("mx selects the block scales of the FP8 products: enable fp8_forward and/or fp8_backward")
        self.mx = mx
        # fp8_dw: the weight gradients on MX operands quantized along the tokens (the contraction
        # of dW): X_perm, the SwiGLU output, dY_perm, dH_gate and dH_up are quantized into
        # token-major codes (each expert's rows from a 128-aligned column, so that no 32-token
        # block spans two experts) that moe_grouped_gemm_dw_mx reads
        if fp8_dw and not mx:
            raise ValueError("fp8_dw takes MX block scales (mx=True)")
        if fp8_dw and concurrent:
            raise ValueError("fp8_dw shares its quantizations with the data products: one stream")
        self.fp8_dw = fp8_dw
        # combine_fused: the weighted combine runs in the down product's epilogue
        # (moe_grouped_gemm_fwd_combine: the tile that stores a token's last row of a column tile
        # sums its k rows); bitwise the separate call's Y, measured slower (its coherent stores)
        if combine_fused and fp8_forward:
            raise ValueError("combine_fused is a form of the bf16 down product")
        self.combine_fused = combine_fused
        # gather_fused: the gate/up product reads its rows straight from x through token_of_row
        # (moe_grouped_gemm_fwd_gather); X_perm is then gathered only in the backward, for dW_gate
        # and dW_up (moe_gather_rows), so a forward alone never writes it
        self.gather_fused = gather_fused
        # split_tail: the fwd and dX products on the main stream split their last partial round of
        # tiles along the contraction (a workspace of fp32 partial tiles)
        self.split_ws = moe.split_workspace(inputs["x"].device) if split_tail else None
        self.fuse = fuse_swiglu_bwd
        self.dw_t = dw_transposed
        # dw_persistent: the dW products run as persistent grids that claim their tiles through
        # these counters (every dW call is on one stream, so one set serves them all)
        self.dw_cnt = moe.dw_counters(inputs["x"].device) if dw_persistent else None
        # concurrent: independent products run on a second stream (default priority): the weight
        # gradients beside the data gradients, the shared FFN beside the routed experts, so each
        # kernel's last partial round of tiles fills with the other's tiles
        self.concurrent = concurrent
        self.side = torch.cuda.Stream(device=inputs["x"].device) if concurrent else None
        # the shared experts' products (G = 1) take a split workspace too; on the side stream, one
        # of their own (calls that may overlap need separate workspaces)
        self.split_ws_side = moe.split_workspace(inputs["x"].device) if (split_tail and concurrent) else None
        self.router = router
        # with the router at E <= 16, d <= 4096 its backward (dlogits, dWr) runs as soon as d_topk_w
        # exists, and its share of dX joins the experts' unpermute-sum in one pass over dX
        # (moe_unpermute_router_dx, bitwise the two-pass result)
        self.router_fused_dx = router and cfg.E <= 16 and cfg.d <= 4096
        self.aux_alpha = float(aux_alpha)
        self.inp = inputs
        self.normalize = normalize_topk
        dev = inputs["x"].device
        T, d, f, E, k = cfg.T, cfg.d, cfg.f, cfg.E, cfg.k
        R = T * k
        bf, f32, i32 = torch.bfloat16, torch.float32, torch.int32
        e = lambda shape, dt=bf: torch.empty(shape, dtype=dt, device=dev)
        self.buf = b = {
            "topk_idx": e((T, k), i32), "topk_w": e((T, k), f32), "offsets": e(E + 1, i32),
            "row_of_slot": e(R, i32), "token_of_row": e(R, i32), "x_perm": e((R, d)),
            "h_gate": e((R, f)), "h_up": e((R, f)), "act": e((R, f)), "y_perm": e((R, d)), "y": e((T, d)),
            "dy_perm": e((R, d)), "d_topk_w": e((T, k), f32), "d_act": e((R, f)),
            "dh_gate": e((R, f)), "dh_up": e((R, f)), "dx_perm": e((R, d)), "dx": e((T, d)),
            "dw_gate": e((E, d, f), f32), "dw_up": e((E, d, f), f32), "dw_down": e((E, f, d), f32),
            "workspace": e(max(16, moe.moe_route_permute_workspace_bytes(T, E, k)), torch.uint8),
        }
        if dw_transposed:
            # contraction-major copies of the dW operands (moe_transpose_grouped layout)
            ld = moe.transposed_cols(R, E)
            b.update({"x_perm_t": e((d, ld)), "dy_perm_t": e((d, ld)), "act_t": e((f, ld)),
                      "dh_gate_t": e((f, ld)), "dh_up_t": e((f, ld))})
        if router:
            b.update({
                "logits": e((T, E), f32), "dlogits": e((T, E), f32), "dwr": e((d, E), f32),
                "aux_loss": e(1, f32),
                "router_ws": e(max(16, moe.lib().moe_router_bwd_workspace_bytes(T, d, E)), torch.uint8),
                "aux_ws": e(max(16, moe.lib().moe_router_aux_loss_workspace_bytes(T, E)), torch.uint8),
            })
        P = moe.mx_groups
        if fp8_forward and gather_fused:
            raise ValueError("fp8_forward reads X_perm: it does not combine with gather_fused")
        if fp8_backward and not fuse_swiglu_bwd:
            raise ValueError("fp8_backward fuses the SwiGLU backward into the dX-down product")
        if mx:
            u8 = torch.uint8
            if fp8_forward:
                b.update({"x_q": e((R, d), u8), "x_s": e((P(d), R, 4), u8), "act_q": e((R, f), u8),
                          "act_s": e((P(f), R, 4), u8)})
            if fp8_backward:
                b.update({"dy_q": e((R, d), u8), "dy_s": e((P(d), R, 4), u8), "dh_q": e((R, 2 * f), u8),
                          "dh_s": e((P(2 * f), R, 4), u8)})
            # codes and block scales of the expert weights: "_t" the forward operands [expert, output
            # channel, contraction] (gate/up interleaved by 128 channels), "_r" the data-gradient
            # operands in the stored layouts (W_down's rows; rows of [W_gate | W_up])
            self.wmx = {}
            if fp8_forward:
                self.wmx["gate_up_t"] = (e((E, 2 * f, d), u8), e((P(d), E, 2 * f, 4), u8))
                self.wmx["down_t"] = (e((E, d, f), u8), e((P(f), E, d, 4), u8))
            if fp8_backward:
                self.wmx["gate_up_r"] = (e((E, d, 2 * f), u8), e((P(2 * f), E, d, 4), u8))
                self.wmx["down_r"] = (e((E, f, d), u8), e((P(d), E, f, 4), u8))
            self._quantize_weights_mx()
        elif fp8_forward:
            u8 = torch.uint8
            b.update({"x_q": e((R, d), u8), "x_s": e(R, f32), "act_q": e((R, f), u8), "act_s": e(R, f32)})
            # weights in the layout [expert, output channel, contraction], quantized per channel
            # (moe_quantize_fp8_weight: transposed, gate/up interleaved by 128, one pass each).  A
            # training step re-quantizes them every forward, since the optimizer changes them;
            # fp8_requantize=False keeps this preparation's codes (weights held fixed)
            self.w8 = {
                "gate_up": (e((E, 2 * f, d), u8), e((E, 2 * f), f32)),
                "down": (e((E, d, f), u8), e((E, d), f32)),
            }
            self._quantize_weights()
        self.fp8_requantize = fp8_requantize
        if fp8_backward and not mx:
            u8 = torch.uint8
            b.update({"dy_q": e((R, d), u8), "dy_s": e(R, f32), "dh_q": e((R, 2 * f), u8), "dh_s": e(R, f32)})
            self.w8b = {
                "down": (e((E, f, d), u8), e((E, f), f32)),
                "gate_up": (e((E, d, 2 * f), u8), e((E, d), f32)),
            }
            self._quantize_weights_bwd()
        self.comb_cnt = moe.combine_counters(T, d, dev) if combine_fused else None
        if fp8_dw:
            u8 = torch.uint8
            ldt = moe.mx_tokens_cols(R, E)
            for name, rows in (("x", d), ("act", f), ("dy", d), ("dhg", f), ("dhu", f)):
                b[name + "_qt"] = e((rows, ldt), u8)
                b[name + "_st"] = e((ldt // 128, rows, 4), u8)
        self.shared = cfg.f_shared > 0
        if self.shared:
            fs = cfg.f_shared
            self.offsets_sh = torch.tensor([0, T], dtype=i32, device=dev)
            b.update({
                "h_gate_sh": e((T, fs)), "h_up_sh": e((T, fs)), "act_sh": e((T, fs)), "y_sh": e((T, d)),
                "d_act_sh": e((T, fs)), "dh_gate_sh": e((T, fs)), "dh_up_sh": e((T, fs)), "dx_sh": e((T, d)),
                "dw_gate_sh": e((1, d, fs), f32), "dw_up_sh": e((1, d, fs), f32), "dw_down_sh": e((1, fs, d), f32),
            })
            self.w_sh = (inputs["w_gate_sh"].unsqueeze(0), inputs["w_up_sh"].unsqueeze(0),
                         inputs["w_down_sh"].unsqueeze(0))

    def _quantize_weights(self, stream=None):
        """E4M3 codes and per-channel scales of the expert weights, in the FP8 products' layout."""
        i, w8 = self.inp, self.w8
        moe.moe_quantize_fp8_weight(i["w_gate"], i["w_up"], *w8["gate_up"], stream=stream)
        moe.moe_quantize_fp8_weight(i["w_down"], None, *w8["down"], stream=stream)

    def _quantize_weights_mx(self, stream=None):
        """MX codes and block scales of the expert weights, every orientation the enabled products
        read, from one pass over each weight."""
        i, w = self.inp, self.wmx
        for src, src2, t, r in ((i["w_gate"], i["w_up"], "gate_up_t", "gate_up_r"),
                                (i["w_down"], None, "down_t", "down_r")):
            qt, st = w.get(t, (None, None))
            qr, sr = w.get(r, (None, None))
            moe.moe_quantize_mx_weight(src, src2, want_t=qt is not None, want_r=qr is not None, qt=qt, st=st,
                                       qr=qr, sr=sr, stream=stream)

    def _quantize_weights_bwd(self, stream=None):
        """E4M3 codes and per-row scales of the expert weights in their stored layouts, the
        operands of the FP8 data-gradient products: W_down [E, f, d] per output channel of dA,
        [W_gate | W_up] [E, d, 2f] per output channel of dX."""
        i, w8 = self.inp, self.w8b
        moe.moe_quantize_fp8_rows(i["w_down"], *w8["down"], stream=stream)
        moe.moe_quantize_fp8_rows2(i["w_gate"], i["w_up"], *w8["gate_up"], stream=stream)

    # ------------------------------------------------------------------------------------------
    def _streams(self, stream):
        main = torch.cuda.current_stream() if stream is None else stream
        return main, (self.side if self.concurrent else main)

    @staticmethod
    def _join(waiter, signaller):
        """waiter waits for everything enqueued on signaller so far (no-op on the same stream)."""
        if waiter is not signaller:
            ev = torch.cuda.Event()
            ev.record(signaller)
            waiter.wait_event(ev)

    def forward(self, stream=None):
        b, i, k, run = self.buf, self.inp, self.cfg.k, self._run
        main, side = self._streams(stream)
        stream = main
        self._join(side, main)            # the side stream starts after the main stream's prior work
        add = None
        if self.shared:                   # the shared FFN needs only x: beside the routed experts
            wg, wu, wd = self.w_sh
            sws = self.split_ws if side is main else self.split_ws_side
            run("fwd_gate_up_sh", moe.moe_grouped_gemm_fwd, i["x"], wg, self.offsets_sh, wu, b["h_gate_sh"],
                b["h_up_sh"], b["act_sh"], want_act=True, stream=side, workspace=sws)
            run("fwd_down_sh", moe.moe_grouped_gemm_fwd, b["act_sh"], wd, self.offsets_sh, C=b["y_sh"],
                stream=side, workspace=sws)
            add = b["y_sh"]
        logits = i["logits"]
        if self.router:
            logits = b["logits"]
            run("router_logits", moe.moe_router_logits, i["x"], i["wr"], i.get("router_bias"), logits=logits,
                stream=stream)
        gf = self.gather_fused
        run("route_permute", moe.moe_route_permute, logits, None if gf else i["x"], k, self.normalize,
            b["topk_idx"], b["topk_w"], b["offsets"], b["row_of_slot"], b["token_of_row"],
            None if gf else b["x_perm"], b["workspace"], stream=stream)
        if self.router and self.aux_alpha:
            run("router_aux_loss", moe.moe_router_aux_loss, logits, b["offsets"], k, self.aux_alpha,
                loss=b["aux_loss"], workspace=b["aux_ws"], stream=stream)
        if self.fp8 and self.mx:
            ws = self.split_ws
            if self.fp8_requantize:
                run("quantize_w", self._quantize_weights_mx, stream=stream)
            if self.fp8_dw:   # X_perm's row codes and, from the same read, its token-major codes for dW
                run("quantize_x", self._quantize_mx_both, "x_perm", "x", "x_q", "x_s", stream=stream)
            else:
                run("quantize_x", moe.moe_quantize_mx_rows, b["x_perm"], None, b["x_q"], b["x_s"], stream=stream)
            run("fwd_gate_up", moe.moe_grouped_gemm_fwd_mx_gate_up, b["x_q"], b["x_s"], *self.wmx["gate_up_t"],
                b["offsets"], b["h_gate"], b["h_up"], b["act"], stream=stream, workspace=ws)
            if self.fp8_dw:
                run("quantize_act", self._quantize_mx_both, "act", "act", "act_q", "act_s", stream=stream)
            else:
                run("quantize_act", moe.moe_quantize_mx_rows, b["act"], None, b["act_q"], b["act_s"], stream=stream)
            run("fwd_down", moe.moe_grouped_gemm_fwd_mx, b["act_q"], b["act_s"], *self.wmx["down_t"], b["offsets"],
                C=b["y_perm"], stream=stream, workspace=ws)
        elif self.fp8:
            ws = self.split_ws
            if self.fp8_requantize:
                run("quantize_w", self._quantize_weights, stream=stream)
            run("quantize_x", moe.moe_quantize_fp8_rows, b["x_perm"], b["x_q"], b["x_s"], stream=stream)
            run("fwd_gate_up", moe.moe_grouped_gemm_fwd_fp8_gate_up, b["x_q"], b["x_s"], *self.w8["gate_up"],
                b["offsets"], b["h_gate"], b["h_up"], b["act"], stream=stream, workspace=ws)
            run("quantize_act", moe.moe_quantize_fp8_rows, b["act"], b["act_q"], b["act_s"], stream=stream)
            run("fwd_down", moe.moe_grouped_gemm_fwd_fp8, b["act_q"], b["act_s"], *self.w8["down"], b["offsets"],
                C=b["y_perm"], stream=stream, workspace=ws)
        elif gf:
            run("fwd_gate_up", moe.moe_grouped_gemm_fwd_gather, i["x"], b["token_of_row"], i["w_gate"],
                b["offsets"], i["w_up"], b["h_gate"], b["h_up"], b["act"], want_act=True, stream=stream,
                workspace=self.split_ws)
        else:
            run("fwd_gate_up", moe.moe_grouped_gemm_fwd, b["x_perm"], i["w_gate"], b["offsets"], i["w_up"],
                b["h_gate"], b["h_up"], b["act"], want_act=True, stream=stream, workspace=self.split_ws)
        if self.combine_fused:
            self._join(main, side)        # the shared output is added in the down product
            run("fwd_down_combine", moe.moe_grouped_gemm_fwd_combine, b["act"], i["w_down"], b["offsets"],
                b["topk_w"], b["row_of_slot"], b["token_of_row"], add=add, y_perm=b["y_perm"], y=b["y"],
                counters=self.comb_cnt, workspace=self.split_ws, stream=stream)
            return b["y"]
        if not self.fp8:
            run("fwd_down", moe.moe_grouped_gemm_fwd, b["act"], i["w_down"], b["offsets"], C=b["y_perm"],
                stream=stream, workspace=self.split_ws)
        self._join(main, side)
        run("combine", moe.moe_unpermute_combine, b["y_perm"], b["topk_w"], b["row_of_slot"], k, add=add,
            y=b["y"], stream=stream)
        return b["y"]

    def backward(self, stream=None):
        b, i, k, run = self.buf, self.inp, self.cfg.k, self._run
        main, side = self._streams(stream)
        stream = main
        self._join(side, main)
        if self.gather_fused:             # X_perm for dW_gate/dW_up (the forward read x directly)
            run("gather_x", moe.moe_gather_rows, i["x"], b["row_of_slot"], k, b["x_perm"], stream=side)
        dx_add = None
        if self.shared:                   # needs dY and the shared forward only
            wg, wu, wd = self.w_sh
            sws = self.split_ws if side is main else self.split_ws_side
            dws = sws if self.dw_cnt is not None else None  # the dW split needs the persistent form
            if self.fuse:
                run("dx_down_swiglu_bwd_sh", moe.moe_grouped_gemm_dx_swiglu_bwd, i["dy"], wd, self.offsets_sh,
                    b["h_gate_sh"], b["h_up_sh"], b["dh_gate_sh"], b["dh_up_sh"], stream=side, workspace=sws)
            else:
                run("dx_down_sh", moe.moe_grouped_gemm_dx, i["dy"], wd, self.offsets_sh, dA=b["d_act_sh"],
                    stream=side, workspace=sws)
            run("dw_down_sh", moe.moe_grouped_gemm_dw, b["act_sh"], i["dy"], self.offsets_sh,
                dB=b["dw_down_sh"], stream=side, counters=self.dw_cnt, workspace=dws)
            if not self.fuse:
                run("swiglu_bwd_sh", moe.moe_swiglu_bwd, b["h_gate_sh"], b["h_up_sh"], b["d_act_sh"],
                    b["dh_gate_sh"], b["dh_up_sh"], stream=side)
            run("dx_gate_up_sh", moe.moe_grouped_gemm_dx, b["dh_gate_sh"], wg, self.offsets_sh, b["dh_up_sh"],
                wu, dA=b["dx_sh"], stream=side, workspace=sws)
            run("dw_gate_up_sh", moe.moe_grouped_gemm_dw, i["x"], b["dh_gate_sh"], self.offsets_sh,
                b["dh_up_sh"], dB=b["dw_gate_sh"], dB2=b["dw_up_sh"], stream=side, counters=self.dw_cnt,
                workspace=dws)
            dx_add = b["dx_sh"]
        run("combine_bwd", moe.moe_unpermute_combine_bwd, i["dy"], b["topk_w"], b["row_of_slot"], k,
            y_perm=b["y_perm"], dy_perm=b["dy_perm"], d_topk_w=b["d_topk_w"], stream=stream)
        if self.router_fused_dx:
            run("router_bwd", moe.moe_router_bwd, i["x"], i["wr"], b["logits"], b["topk_idx"], b["topk_w"],
                b["d_topk_w"], b["offsets"], self.normalize, self.aux_alpha, dx=None, workspace=b["router_ws"],
                dlogits=b["dlogits"], dwr=b["dwr"], stream=stream)
        if self.fp8_dw:                   # dY_perm's token-major codes (and its row codes for dX down)
            if self.fp8_bwd:
                run("quantize_dy", self._quantize_mx_both, "dy_perm", "dy", "dy_q", "dy_s", stream=stream)
            else:
                run("quantize_t_dy", self._quantize_mx_both, "dy_perm", "dy", None, None, stream=stream)
        self._join(side, main)            # dW_down needs dY_perm
        if self.fp8_dw:
            if not self.fp8:              # else the forward's quantization wrote them
                run("quantize_t_act", self._quantize_mx_both, "act", "act", None, None, stream=side)
            run("dw_down", moe.moe_grouped_gemm_dw_mx, b["act_qt"], b["act_st"], b["dy_qt"], b["dy_st"],
                b["offsets"], self.R, dB=b["dw_down"], counters=self.dw_cnt, stream=side)
        elif self.dw_t:
            run("transpose_act", moe.moe_transpose_grouped, b["act"], b["offsets"], dst=b["act_t"], stream=side)
            run("transpose_dy_perm", moe.moe_transpose_grouped, b["dy_perm"], b["offsets"], dst=b["dy_perm_t"],
                stream=side)
            run("dw_down", moe.moe_grouped_gemm_dw_t, b["act_t"], b["dy_perm_t"], b["offsets"], self.R,
                dB=b["dw_down"], stream=side)
        else:
            run("dw_down", moe.moe_grouped_gemm_dw, b["act"], b["dy_perm"], b["offsets"], dB=b["dw_down"],
                stream=side, counters=self.dw_cnt)
        if self.fp8_bwd and self.mx:
            if self.fp8_requantize and not self.fp8:   # else the forward's pass wrote both orientations
                run("quantize_w_bwd", self._quantize_weights_mx, stream=stream)
            if not self.fp8_dw:
                run("quantize_dy", moe.moe_quantize_mx_rows, b["dy_perm"], None, b["dy_q"], b["dy_s"], stream=stream)
            run("dx_down_swiglu_bwd", moe.moe_grouped_gemm_dx_swiglu_bwd_mx, b["dy_q"], b["dy_s"],
                *self.wmx["down_r"], b["offsets"], b["h_gate"], b["h_up"], b["dh_gate"], b["dh_up"], stream=stream,
                workspace=self.split_ws)
        elif self.fp8_bwd:
            if self.fp8_requantize:
                run("quantize_w_bwd", self._quantize_weights_bwd, stream=stream)
            run("quantize_dy", moe.moe_quantize_fp8_rows, b["dy_perm"], b["dy_q"], b["dy_s"], stream=stream)
            run("dx_down_swiglu_bwd", moe.moe_grouped_gemm_dx_swiglu_bwd_fp8, b["dy_q"], b["dy_s"],
                *self.w8b["down"], b["offsets"], b["h_gate"], b["h_up"], b["dh_gate"], b["dh_up"], stream=stream,
                workspace=self.split_ws)
        elif self.fuse:
            run("dx_down_swiglu_bwd", moe.moe_grouped_gemm_dx_swiglu_bwd, b["dy_perm"], i["w_down"],
                b["offsets"], b["h_gate"], b["h_up"], b["dh_gate"], b["dh_up"], stream=stream,
                workspace=self.split_ws)
        else:
            run("dx_down", moe.moe_grouped_gemm_dx, b["dy_perm"], i["w_down"], b["offsets"], dA=b["d_act"],
                stream=stream)
            run("swiglu_bwd", moe.moe_swiglu_bwd, b["h_gate"], b["h_up"], b["d_act"], b["dh_gate"],
                b["dh_up"], stream=stream)
        self._join(side, main)            # dW_gate/dW_up need dH
        if self.fp8_bwd and self.mx:
            if self.fp8_dw:               # the joined rows' codes and both token-major codes, one read
                run("quantize_dh", self._quantize_mx_dh, True, stream=stream)
            else:
                run("quantize_dh", moe.moe_quantize_mx_rows, b["dh_gate"], b["dh_up"], b["dh_q"], b["dh_s"],
                    stream=stream)
            run("dx_gate_up", moe.moe_grouped_gemm_fwd_mx, b["dh_q"], b["dh_s"], *self.wmx["gate_up_r"],
                b["offsets"], C=b["dx_perm"], stream=stream, workspace=self.split_ws)
        elif self.fp8_bwd:
            run("quantize_dh", moe.moe_quantize_fp8_rows2, b["dh_gate"], b["dh_up"], b["dh_q"], b["dh_s"],
                stream=stream)
            run("dx_gate_up", moe.moe_grouped_gemm_fwd_fp8, b["dh_q"], b["dh_s"], *self.w8b["gate_up"], b["offsets"],
                C=b["dx_perm"], stream=stream, workspace=self.split_ws)
        else:
            run("dx_gate_up", moe.moe_grouped_gemm_dx, b["dh_gate"], i["w_gate"], b["offsets"], b["dh_up"],
                i["w_up"], dA=b["dx_perm"], stream=stream, workspace=self.split_ws)
        # one stream: the unpermute-sum reads dX_perm right after it was written, while it still sits
        # in the last-level cache (dW gate/up's 3.8 GB of fp32 results would evict it first)
        early = side is main
        if early:
            self._unpermute_dx(dx_add, stream)
        if self.fp8_dw:
            if not self.fp8:
                run("quantize_t_x", self._quantize_mx_both, "x_perm", "x", None, None, stream=side)
            if not self.fp8_bwd:
                run("quantize_t_dh", self._quantize_mx_dh, False, stream=side)
            run("dw_gate_up", moe.moe_grouped_gemm_dw_mx, b["x_qt"], b["x_st"], b["dhg_qt"], b["dhg_st"],
                b["offsets"], self.R, b["dhu_qt"], b["dhu_st"], dB=b["dw_gate"], dB2=b["dw_up"],
                counters=self.dw_cnt, stream=side)
        elif self.dw_t:
            run("transpose_x_perm", moe.moe_transpose_grouped, b["x_perm"], b["offsets"], dst=b["x_perm_t"],
                stream=side)
            run("transpose_dh", self._transpose_dh, stream=side)
            run("dw_gate_up", moe.moe_grouped_gemm_dw_t, b["x_perm_t"], b["dh_gate_t"], b["offsets"], self.R,
                b["dh_up_t"], dB=b["dw_gate"], dB2=b["dw_up"], stream=side)
        else:
            run("dw_gate_up", moe.moe_grouped_gemm_dw, b["x_perm"], b["dh_gate"], b["offsets"], b["dh_up"],
                dB=b["dw_gate"], dB2=b["dw_up"], stream=side, counters=self.dw_cnt)
        self._join(main, side)            # the shared dX, and every weight gradient, are complete
        if not early:
            self._unpermute_dx(dx_add, stream)
        if self.router and not self.router_fused_dx:
            run("router_bwd", moe.moe_router_bwd, i["x"], i["wr"], b["logits"], b["topk_idx"], b["topk_w"],
                b["d_topk_w"], b["offsets"], self.normalize, self.aux_alpha, dx=b["dx"], workspace=b["router_ws"],
                dlogits=b["dlogits"], dwr=b["dwr"], stream=stream)
        return b["dx"]

    def _unpermute_dx(self, dx_add, stream):
        b, i, k = self.buf, self.inp, self.cfg.k
        if self.router_fused_dx:
            self._run("unpermute_dx_router", moe.moe_unpermute_router_dx, b["dx_perm"], b["row_of_slot"], k,
                      b["dlogits"], i["wr"], add=dx_add, dx=b["dx"], stream=stream)
        else:
            self._run("unpermute_dx", moe.moe_unpermute_combine, b["dx_perm"], None, b["row_of_slot"], k,
                      add=dx_add, y=b["dx"], stream=stream)

    @property
    def R(self):
        return self.cfg.T * self.cfg.k

    def _quantize_mx_both(self, src, tok, q, s, stream=None):
        """Token-major MX codes of buffer `src` (into `tok`_qt/_st) and, when q is given, its row codes
        (into q/s), from one read."""
        b = self.buf
        moe.moe_quantize_mx_tokens(b[src], b["offsets"], b[tok + "_qt"], b[tok + "_st"],
                                   qr=None if q is None else b[q], sr=None if s is None else b[s],
                                   want_r=q is not None, stream=stream)

    def _quantize_mx_dh(self, rows, stream=None):
        """Token-major MX codes of dH_gate and dH_up and, with rows, the codes of the joined rows
        [dH_gate | dH_up] (each half written by the call that reads it)."""
        b, f = self.buf, self.cfg.f
        for src, tok, col0 in (("dh_gate", "dhg", 0), ("dh_up", "dhu", f)):
            moe.moe_quantize_mx_tokens(b[src], b["offsets"], b[tok + "_qt"], b[tok + "_st"],
                                       qr=b["dh_q"] if rows else None, sr=b["dh_s"] if rows else None,
                                       col0=col0, want_r=rows, stream=stream)

    def _transpose_dh(self, stream=None):
        b = self.buf
        moe.moe_transpose_grouped(b["dh_gate"], b["offsets"], dst=b["dh_gate_t"], stream=stream)
        moe.moe_transpose_grouped(b["dh_up"], b["offsets"], dst=b["dh_up_t"], stream=stream)

    def step(self, stream=None):
        self.forward(stream)
        self.backward(stream)

    # algorithmic work of each call (FLOPs for GEMMs, unique HBM bytes for the rest)
    def work(self):
        c = self.cfg
        T, d, f, k, E = c.T, c.d, c.f, c.k, c.E
        R = T * k
        # per-row scale bytes: one fp32, or (MX) one byte per 32 elements
        sc = (lambda n: n // 32) if self.mx else (lambda n: 4)
        n_or = (1 if self.fp8 else 0) + (1 if self.fp8_bwd else 0)   # weight orientations written
        w = {
            "route_permute": ("bytes", T * E * 4 + T * k * 8 + R * 8
                              + (0 if self.gather_fused else T * d * 2 + R * d * 2)),
            "gather_x": ("bytes", T * d * 2 + R * d * 2 + R * 4),
            # FP8 forward: E4M3 products (8-bit MFMA work), quantizers and the standalone SwiGLU
            "quantize_x": ("bytes", R * d * (4 if self.fp8_dw else 3) + R * sc(d) * (2 if self.fp8_dw else 1)),
            "quantize_act": ("bytes", R * f * (4 if self.fp8_dw else 3) + R * sc(f) * (2 if self.fp8_dw else 1)),
            # read bf16, write codes (MX: both orientations a step needs, from one read)
            "quantize_w": ("bytes", (3 * E * d * f * (2 + n_or) + n_or * 3 * E * d * f // 32) if self.mx
                           else (3 * E * d * f * 3 + 3 * E * (d + f) * 4)),
            "fwd_gate_up": ("flops8" if self.fp8 else "flops", 4 * R * d * f),
            "fwd_down": ("flops8" if self.fp8 else "flops", 2 * R * f * d),
            "fwd_down_combine": ("flops", 2 * R * f * d),
            "combine": ("bytes", R * d * 2 + T * d * 2 + T * k * 8 + (T * d * 2 if self.shared else 0)),
            "combine_bwd": ("bytes", T * d * 2 + 2 * R * d * 2 + T * k * 12),
            "dx_down": ("flops", 2 * R * d * f), "dw_down": ("flops8" if self.fp8_dw else "flops", 2 * R * f * d),
            "dx_down_swiglu_bwd": ("flops8" if self.fp8_bwd else "flops", 2 * R * d * f),
            # FP8 backward: dY_perm and [dH_gate | dH_up] per row, the weights in their stored layouts
            "quantize_dy": ("bytes", R * d * (4 if self.fp8_dw else 3) + R * sc(d) * (2 if self.fp8_dw else 1)),
            "quantize_dh": ("bytes", 2 * R * f * (4 if self.fp8_dw else 3) + R * sc(2 * f) * (2 if self.fp8_dw else 1)),
            "quantize_w_bwd": ("bytes", (3 * E * d * f * 3 + 3 * E * d * f // 32) if self.mx
                               else (3 * E * d * f * 3 + E * (d + f) * 4)),
            "swiglu_bwd": ("bytes", 5 * R * f * 2),
            "dx_gate_up": ("flops8" if self.fp8_bwd else "flops", 4 * R * d * f),
            "dw_gate_up": ("flops8" if self.fp8_dw else "flops", 4 * R * d * f),
            # MX weight gradient: token-major codes of its operands (read bf16, write codes + scales)
            "quantize_t_x": ("bytes", R * d * 3 + R * d // 32), "quantize_t_act": ("bytes", R * f * 3 + R * f // 32),
            "quantize_t_dy": ("bytes", R * d * 3 + R * d // 32), "quantize_t_dh": ("bytes", 2 * (R * f * 3 + R * f // 32)),
            "unpermute_dx": ("bytes", R * d * 2 + T * d * 2 + R * 4 + (T * d * 2 if self.shared else 0)),
            # router: fp32 vector-ALU work (multiply-adds x2) of the contractions with Wr, with the
            # HBM bytes each call must move (x bf16 read; logits / dlogits fp32; the backward also
            # reads and rewrites dX); at these E the intensity sits below the fp32 VALU / HBM ridge
            "router_logits": ("valu", (2 * T * d * E, T * d * 2 + d * E * 4 + T * E * 4)),
            "router_bwd": (("valu", (2 * T * d * E, T * d * 2 + 2 * T * E * 4 + T * k * 12 + d * E * 4))
                           if self.router_fused_dx else
                           ("valu", (4 * T * d * E, T * d * 2 + 2 * T * d * 2 + 2 * T * E * 4 + T * k * 12))),
            # the unpermute-sum with the router's share of dX (read dlogits and Wr as well)
            "unpermute_dx_router": ("bytes", R * d * 2 + T * d * 2 + R * 4 + T * E * 4 + d * E * 4
                                    + (T * d * 2 if self.shared else 0)),
            "router_aux_loss": ("bytes", T * E * 4),
            # contraction-major copies for the dW products (read + write)
            "transpose_act": ("bytes", 2 * R * f * 2), "transpose_dy_perm": ("bytes", 2 * R * d * 2),
            "transpose_x_perm": ("bytes", 2 * R * d * 2), "transpose_dh": ("bytes", 4 * R * f * 2),
        }
        if self.shared:
            fs = c.f_shared
            w.update({"fwd_gate_up_sh": ("flops", 4 * T * d * fs), "fwd_down_sh": ("flops", 2 * T * fs * d),
                      "dx_down_sh": ("flops", 2 * T * d * fs), "dw_down_sh": ("flops", 2 * T * fs * d),
                      "dx_down_swiglu_bwd_sh": ("flops", 2 * T * d * fs),
                      "swiglu_bwd_sh": ("bytes", 5 * T * fs * 2),
                      "dx_gate_up_sh": ("flops", 4 * T * d * fs), "dw_gate_up_sh": ("flops", 4 * T * d * fs)})
        return w


class DWOnly(_Traced):
    """The weight-gradient-only workload: dW_gate and dW_up in one pass, then dW_down (unless
    cfg.dw1_only: the paper's dW1 alone); fp32 results, or bf16 when cfg.dw_bf16."""

    def __init__(self, cfg, inputs: dict, persistent: bool = True):
        self.cfg = cfg
        self.inp = inputs
        dev = inputs["x_perm"].device
        self.cnt = moe.dw_counters(dev) if persistent else None
        E, d, f = cfg.E, cfg.d, cfg.f
        dt = torch.bfloat16 if cfg.dw_bf16 else torch.float32
        self.buf = {
            "dw_gate": torch.empty((E, d, f), dtype=dt, device=dev),
            "dw_up": torch.empty((E, d, f), dtype=dt, device=dev),
        }
        if not cfg.dw1_only:
            self.buf["dw_down"] = torch.empty((E, f, d), dtype=dt, device=dev)

    def step(self, stream=None):
        i, b = self.inp, self.buf
        dw = moe.moe_grouped_gemm_dw_bf16 if self.cfg.dw_bf16 else moe.moe_grouped_gemm_dw
        self._run("dw_gate_up", dw, i["x_perm"], i["dh_gate"], i["offsets"], i["dh_up"],
                  dB=b["dw_gate"], dB2=b["dw_up"], stream=stream, counters=self.cnt)
        if not self.cfg.dw1_only:
            self._run("dw_down", dw, i["act"], i["dy_perm"], i["offsets"], dB=b["dw_down"], stream=stream,
                      counters=self.cnt)

    def work(self):
        c = self.cfg
        w = {"dw_gate_up": ("flops", 4 * c.R * c.d * c.f)}
        if not c.dw1_only:
            w["dw_down"] = ("flops", 2 * c.R * c.f * c.d)
        return w
