"""Full-size parity of the layer in the launch configuration the benchmark times (MoELayer.step on
the five layer configurations and the paper's own dW1 shape), against the CPU oracle.

Routing indices, expert offsets, the permutation and the gathered rows are compared in full and
bit-exactly.  Floating outputs are compared on samples the oracle computes one by one with the
same definitions: every row of a few sampled tokens (gate/up, SwiGLU, down, dY_perm, dA, dH,
dX_perm, the token's Y and dX and its d_topk_w), whole rows of dW_down and whole columns of
dW_gate/dW_up for the largest and the smallest expert group, and the shared FFN's rows and weight
gradient columns.  Inputs are drawn on the GPU by the seeded generator and copied to the host."""
import sys

import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2606_26453_amd import layer as L
from paper_2606_26453_amd import workloads as W
from tests.gpu_util import check_float, f64, gpu_available, i64

pytestmark = [pytest.mark.gpu, pytest.mark.slow,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

DEV = "cuda:0"


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _rows(t, idx):
    """Rows `idx` of a GPU tensor as float64 numpy."""
    return f64(t[torch.as_tensor(np.asarray(idx), dtype=torch.long, device=t.device)])


@pytest.mark.parametrize("cfg_id,ntok", [(1, 8), (2, 4), (3, 8)])
def test_layer_fullsize_sampled(cfg_id, ntok):
    cfg = W.CONFIGS[cfg_id]
    T, E, k = cfg.T, cfg.E, cfg.k
    _say(f"full-size layer parity: config {cfg_id} {cfg}")
    inp = W.make_inputs(cfg, 0, DEV)
    lay = L.MoELayer(cfg, inp)
    lay.step()
    torch.cuda.synchronize()
    b = lay.buf

    # routing / grouping / permutation / gather: all rows, bit exact
    logits = inp["logits"].cpu().numpy()
    idx, w = O.route_topk(logits, k)
    off, ros, tor = O.permute(idx, E)
    np.testing.assert_array_equal(i64(b["topk_idx"]), idx)
    np.testing.assert_array_equal(i64(b["offsets"]), off)
    np.testing.assert_array_equal(i64(b["row_of_slot"]), ros)
    np.testing.assert_array_equal(i64(b["token_of_row"]), tor)
    assert torch.equal(b["x_perm"].cpu(), inp["x"].cpu()[torch.from_numpy(tor)])
    check_float("topk_w", f64(b["topk_w"]), w, 1e-5)
    counts = np.diff(off)
    _say("groups:", W.group_stats(counts))

    rng = np.random.default_rng(cfg_id)
    toks = np.sort(rng.choice(T, ntok, replace=False))
    x_t = f64(inp["x"][torch.as_tensor(toks, device=DEV)])
    dy_t = f64(inp["dy"][torch.as_tensor(toks, device=DEV)])
    rows_tok = ros.reshape(T, k)[toks]            # [ntok, k]
    exp_tok = idx[toks]
    dwe = sorted({int(np.argmax(counts)), int(np.argmin(np.where(counts > 0, counts, 10 ** 9)))})

    ref = {key: {} for key in ("h_gate", "h_up", "act", "y_perm", "dy_perm", "d_act", "dh_gate", "dh_up",
                               "dx_perm")}
    fused = lay.fuse   # dA is not materialised when the SwiGLU backward is fused into the dX GEMM
    dw_cols = rng.choice(cfg.f, 4, replace=False)
    dw_rows_f = rng.choice(cfg.f, 3, replace=False)
    dy_all = None
    x_all = None
    for e in sorted(set(exp_tok.ravel().tolist()) | set(dwe)):
        wg = f64(inp["w_gate"][e])
        wu = f64(inp["w_up"][e])
        wd = f64(inp["w_down"][e])
        sel = np.argwhere(exp_tok == e)           # (token index in sample, j)
        if len(sel):
            r = rows_tok[sel[:, 0], sel[:, 1]]
            hg, hu, a, yp = O.expert_rows_forward(x_t[sel[:, 0]], wg, wu, wd)
            dyp = O.bf16_round(w[toks[sel[:, 0]], sel[:, 1]][:, None] * dy_t[sel[:, 0]])
            da, dhg, dhu, dxp = O.expert_rows_backward(hg, hu, dyp, wg, wu, wd)
            for key, val in (("h_gate", hg), ("h_up", hu), ("act", a), ("y_perm", yp), ("dy_perm", dyp),
                             ("d_act", da), ("dh_gate", dhg), ("dh_up", dhu), ("dx_perm", dxp)):
                for n, rr in enumerate(r):
                    ref[key][int(rr)] = val[n]
        if e in dwe:
            lo, hi = int(off[e]), int(off[e + 1])
            if x_all is None:
                x_all = f64(inp["x"])
                dy_all = f64(inp["dy"])
            t_e = tor[lo:hi]
            xp_e = x_all[t_e]
            slot_e = np.argsort(ros)[lo:hi]          # slots stored at these rows
            dyp_e = O.bf16_round(w.reshape(-1)[slot_e][:, None] * dy_all[t_e])
            got_dwd = _rows(b["dw_down"][e], dw_rows_f)
            ref_dwd = O.dw_down_rows(xp_e, dyp_e, wg, wu, dw_rows_f)
            check_float(f"dw_down[e={e}] rows", got_dwd, ref_dwd)
            ref_g, ref_u = O.dw_gate_up_cols(xp_e, dyp_e, wg, wu, wd, dw_cols)
            cols_t = torch.as_tensor(dw_cols, dtype=torch.long, device=DEV)
            check_float(f"dw_gate[e={e}] cols", f64(b["dw_gate"][e][:, cols_t]), ref_g)
            check_float(f"dw_up[e={e}] cols", f64(b["dw_up"][e][:, cols_t]), ref_u)
            _say(f"  dW checked for expert {e} ({hi - lo} rows)")
        del wg, wu, wd

    all_rows = sorted(ref["h_gate"])
    for key in ref:
        if key == "d_act" and fused:
            continue
        got = _rows(b[key], all_rows)
        want = np.stack([ref[key][r] for r in all_rows])
        check_float(key, got, want)

    # token-level outputs: combine of the oracle's rows (+ shared FFN)
    y_sh_t = dx_sh_t = None
    if cfg.f_shared:
        wgs, wus, wds = (f64(inp[n_]) for n_ in ("w_gate_sh", "w_up_sh", "w_down_sh"))
        hgs, hus, as_, ys = O.expert_rows_forward(x_t, wgs, wus, wds)
        das, dhgs, dhus, dxs = O.expert_rows_backward(hgs, hus, dy_t, wgs, wus, wds)
        tok_t = torch.as_tensor(toks, dtype=torch.long, device=DEV)
        for key, val in (("h_gate_sh", hgs), ("h_up_sh", hus), ("act_sh", as_), ("y_sh", ys),
                         ("d_act_sh", das), ("dh_gate_sh", dhgs), ("dh_up_sh", dhus), ("dx_sh", dxs)):
            if key == "d_act_sh" and fused:
                continue
            check_float(key, f64(b[key][tok_t]), val)
        y_sh_t, dx_sh_t = ys, dxs
        xs = f64(inp["x"])
        dys = f64(inp["dy"])
        cols = rng.choice(cfg.f_shared, 3, replace=False)
        rg, ru = O.dw_gate_up_cols(xs, dys, wgs, wus, wds, cols)
        cols_t = torch.as_tensor(cols, dtype=torch.long, device=DEV)
        check_float("dw_gate_sh cols", f64(b["dw_gate_sh"][0][:, cols_t]), rg)
        check_float("dw_up_sh cols", f64(b["dw_up_sh"][0][:, cols_t]), ru)
        rws = rng.choice(cfg.f_shared, 3, replace=False)
        check_float("dw_down_sh rows", _rows(b["dw_down_sh"][0], rws), O.dw_down_rows(xs, dys, wgs, wus, rws))

    yp_tok = np.stack([np.stack([ref["y_perm"][int(r)] for r in rr]) for rr in rows_tok])     # [ntok, k, d]
    dxp_tok = np.stack([np.stack([ref["dx_perm"][int(r)] for r in rr]) for rr in rows_tok])
    y_ref = O.bf16_round((w[toks][:, :, None] * yp_tok).sum(1) + (0 if y_sh_t is None else y_sh_t))
    dx_ref = O.bf16_round(dxp_tok.sum(1) + (0 if dx_sh_t is None else dx_sh_t))
    dtw_ref = (dy_t[:, None, :] * yp_tok).sum(2)
    tok_t = torch.as_tensor(toks, dtype=torch.long, device=DEV)
    check_float("y", f64(b["y"][tok_t]), y_ref)
    check_float("dx", f64(b["dx"][tok_t]), dx_ref)
    check_float("d_topk_w", f64(b["d_topk_w"][tok_t]), dtw_ref)


def test_dw_only_fullsize_sampled():
    cfg = W.CONFIGS[4]
    _say(f"full-size dW parity: config 4 {cfg}")
    inp = W.make_dw_inputs(cfg, 0, DEV)
    lay = L.DWOnly(cfg, inp)
    lay.step()
    torch.cuda.synchronize()
    b = lay.buf
    off = i64(inp["offsets"])
    rng = np.random.default_rng(4)
    for e in (0, cfg.E - 1):
        lo, hi = int(off[e]), int(off[e + 1])
        sl = slice(lo, hi)
        cols = rng.choice(cfg.f, 4, replace=False)
        cols_t = torch.as_tensor(cols, dtype=torch.long, device=DEV)
        xp = f64(inp["x_perm"][sl])
        loc = np.array([0, hi - lo])
        check_float(f"dw_gate[{e}] cols", f64(b["dw_gate"][e][:, cols_t]),
                    O.grouped_gemm_dw(xp, f64(inp["dh_gate"][sl][:, cols_t]), loc)[0])
        check_float(f"dw_up[{e}] cols", f64(b["dw_up"][e][:, cols_t]),
                    O.grouped_gemm_dw(xp, f64(inp["dh_up"][sl][:, cols_t]), loc)[0])
        rws = rng.choice(cfg.f, 4, replace=False)
        rws_t = torch.as_tensor(rws, dtype=torch.long, device=DEV)
        check_float(f"dw_down[{e}] rows", f64(b["dw_down"][e][rws_t]),
                    O.grouped_gemm_dw(f64(inp["act"][sl][:, rws_t]), f64(inp["dy_perm"][sl]), loc)[0])


def test_paper_dw1_fullsize_sampled():
    """The paper's GPT-OSS dW1 shape (K = 2880, gate and up 2880 each, 128 experts, 57,768 rows,
    Dirichlet-Multinomial loads with empty experts), bf16 output: sampled columns of the largest,
    a small and the first nonempty expert against the oracle's bf16-rounded sums; every empty
    expert's gradient exactly zero."""
    cfg = W.CONFIGS[5]
    _say(f"full-size dW1 parity: config 5 {cfg}")
    inp = W.make_dw_inputs(cfg, 0, DEV)
    lay = L.DWOnly(cfg, inp)
    lay.step()
    torch.cuda.synchronize()
    b = lay.buf
    assert b["dw_gate"].dtype == torch.bfloat16 and "dw_down" not in b
    off = i64(inp["offsets"])
    counts = np.diff(off)
    _say("groups:", W.group_stats(counts))
    assert (counts == 0).any()
    rng = np.random.default_rng(5)
    nz = np.flatnonzero(counts)
    small = nz[np.argmin(counts[nz])]
    for e in sorted({int(np.argmax(counts)), int(small), int(nz[0])}):
        lo, hi = int(off[e]), int(off[e + 1])
        cols = np.concatenate([rng.choice(cfg.f, 3, replace=False), [cfg.f - 1]])   # incl. the ragged last tile
        cols_t = torch.as_tensor(cols, dtype=torch.long, device=DEV)
        xp = f64(inp["x_perm"][lo:hi])
        loc = np.array([0, hi - lo])
        for name, src in (("dw_gate", "dh_gate"), ("dw_up", "dh_up")):
            want = O.bf16_round(O.grouped_gemm_dw(xp, f64(inp[src][lo:hi][:, cols_t]), loc)[0])
            check_float(f"{name}[{e}] cols", f64(b[name][e][:, cols_t]), want)
    for e in np.flatnonzero(counts == 0):
        assert torch.count_nonzero(b["dw_gate"][int(e)]) == 0 and torch.count_nonzero(b["dw_up"][int(e)]) == 0
