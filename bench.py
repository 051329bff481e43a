"""Benchmark of the MoE expert-FFN training layer (forward + backward) on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 1] [--no-cpu-baseline] [--flush]
python bench.py --all-configs      (an opt-in summary line over configurations 0-5)

--config 0..4 are the layer configurations (1, the Mixtral-shaped layer, is the default and the
headline); --config 5 times the paper's own kernel alone, the gate/up weight gradient dW1 at its
GPT-OSS-120B shape with bf16 output.

A step is one forward and one backward pass of the whole layer (routing, permutation, gather,
gate/up grouped GEMM with fused SwiGLU, down grouped GEMM, combine, and the backward dX/dW grouped
GEMMs, SwiGLU backward, combine backward and dX unpermute) over one batch of synthetic tokens
whose inputs already sit in HBM.  Prints one JSON line.

Besides the whole-region figure (`value`, `ms_per_step`), the line carries the per-step
distribution (median, p10, p90 of the same timed steps, from one event pair per step), the shader
clock sampled while the timed steps run (amdsmi, every XCD) and the fraction of peak at that clock,
and, with --flush, the same steps timed one at a time after a 1 GiB read that replaces the
Infinity Cache contents (a read, so the next step does not pay to write dirty lines back).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
PEAK_FP32_VALU_TFLOPS = 157.3   # MI355X fp32 vector
PEAK_FP8_TFLOPS = 5000.0    # MI355X dense fp8 MFMA
PEAK_CLOCK_MHZ = 2400.0     # the clock the peaks are quoted at
VALU_RIDGE = PEAK_FP32_VALU_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)   # FLOP per byte where fp32 VALU meets HBM
METRIC = "MoE layer fwd+bwd tokens/sec + grouped-GEMM TFLOP/s (% of bf16 MFMA peak), 1 GPU"

# HBM bytes per launch of each layer call on the Mixtral-shaped layer, from rocprofv3 FETCH_SIZE /
# WRITE_SIZE runs scaled by a plain copy of known size (profiles/moe_layer_hbm_traffic_*.md).
# Valid only for the kernel code they were measured on (sha256 prefix of the sources with comments
# and blank lines removed); otherwise reported null.
TRAFFIC_SOURCES = {
    "gemm": (("paper_2606_26453_amd/csrc/grouped_gemm.hip", "paper_2606_26453_amd/csrc/common.h"), "3da9d8a52732f4f6"),
    "route": (("paper_2606_26453_amd/csrc/route_permute.hip", "paper_2606_26453_amd/csrc/common.h"), "72087f561c2c164f"),
    "combine": (("paper_2606_26453_amd/csrc/elementwise.hip", "paper_2606_26453_amd/csrc/common.h"), "5fb5e5e15e3e53f4"),
}
TRAFFIC_CONFIG = 1
FETCH_SCALE, WRITE_SCALE = 2.0 * 1024, 1.0 * 1024
TRAFFIC_KIB = {  # call: (source group, FETCH_SIZE KiB, WRITE_SIZE KiB) per dispatch (routing: both launches)
    "route_permute": ("route", 33112, 131518),
    "fwd_gate_up": ("gemm", 5344905, 1399104), "fwd_down": ("gemm", 1968892, 199688),
    "combine": ("combine", 65813, 65536), "combine_bwd": ("combine", 98585, 131137),
    "dw_down": ("gemm", 1442369, 1835232), "dx_down_swiglu_bwd": ("gemm", 3827159, 917504),
    "dx_gate_up": ("gemm", 4034670, 196616), "unpermute_dx": ("combine", 65692, 65536),
    "dw_gate_up": ("gemm", 2773784, 3670464),
}


def code_hash(text):
    import hashlib
    import re
    lines = [re.sub(r"//.*$", "", ln).rstrip() for ln in text.splitlines()]
    return hashlib.sha256("\n".join(ln for ln in lines if ln.strip()).encode()).hexdigest()[:16]


def source_hash(files):
    return code_hash("".join(open(os.path.join(ROOT, f)).read() for f in files))


def measured_traffic(call, config, variant=False):
    """Counter bytes of `call` from the table above, for the default kernels only (a variant flag
    swaps in other kernels under the same call names)."""
    if variant or config != TRAFFIC_CONFIG or call not in TRAFFIC_KIB:
        return None
    group, f, w = TRAFFIC_KIB[call]
    files, sha = TRAFFIC_SOURCES[group]
    try:
        if source_hash(files) != sha:
            return None
    except OSError:
        return None
    return int(f * FETCH_SCALE + w * WRITE_SCALE)


def _args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=1)
    ap.add_argument("--router", action="store_true",
                    help="also run the router on the GPU (logits, load-balancing loss, router backward); "
                         "the default step starts from given logits")
    ap.add_argument("--aux-alpha", type=float, default=0.01, help="load-balancing loss weight with --router")
    ap.add_argument("--dw-transposed", action="store_true",
                    help="weight gradients from contraction-major copies of their operands")
    ap.add_argument("--fp8-forward", action="store_true",
                    help="the routed experts' forward products on E4M3 operands (a variant; the metric is bf16)")
    ap.add_argument("--fp8-backward", action="store_true",
                    help="the routed experts' data-gradient products on E4M3 operands (a variant; the metric is bf16)")
    ap.add_argument("--mx", action="store_true",
                    help="with --fp8-forward/--fp8-backward: MX block scales (a power of two per 32 contraction "
                         "elements) instead of fp32 per-row/per-channel scales")
    ap.add_argument("--fp8-dw", action="store_true",
                    help="with --mx: the weight gradients on MX operands quantized along the tokens (a variant)")
    ap.add_argument("--fp8-fixed-weights", action="store_true",
                    help="with --fp8-forward/--fp8-backward: quantize the weights once (held fixed), not every step")
    ap.add_argument("--forward-only", action="store_true", help="time the forward alone (a variant)")
    ap.add_argument("--graph", action="store_true",
                    help="capture the step into a HIP graph once and time its replays (no per-call events)")
    ap.add_argument("--combine-fused", action="store_true",
                    help="the weighted combine in the down product's epilogue (a variant)")
    ap.add_argument("--gather-fused", action="store_true",
                    help="gate/up product reads x through token_of_row; X_perm is gathered in the backward")
    ap.add_argument("--no-split-tail", action="store_true",
                    help="persistent dX products do not split their last partial round of tiles")
    ap.add_argument("--dw-one-per-tile", action="store_true",
                    help="variant: the dW products launch one workgroup per tile (no persistent grid)")
    ap.add_argument("--concurrent", action="store_true",
                    help="weight gradients and the shared FFN on a second stream beside the main chain "
                         "(per-call times then include the sharing of the CUs)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-tokens", type=int, default=0)
    ap.add_argument("--no-trace", action="store_true", help="no per-call events inside the timed region")
    ap.add_argument("--gemm-probe", choices=["fwd", "dx", "dw"],
                    help="run one gate/up-shaped grouped GEMM (uniform groups of the chosen config) 3 times and "
                         "exit: the target of hardware-counter runs")
    ap.add_argument("--vendor-loop", action="store_true",
                    help="context only: the paper's dW1 shape (config 5) and the Mixtral-shaped gate/up forward "
                         "through the library and through a per-expert hipBLASLt (torch.matmul) loop; one JSON line")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES bytes 3 times (counter calibration)")
    ap.add_argument("--flush", action="store_true",
                    help="also time each step alone after a 1 GiB read that replaces the Infinity Cache contents")
    ap.add_argument("--no-clock", action="store_true", help="do not sample the shader clock")
    ap.add_argument("--all-configs", action="store_true",
                    help="print one summary line over configurations 0-5 (a few steps each) instead of the headline")
    return ap.parse_args()


class ClockSampler:
    """Samples the current graphics clock of every XCD (amdsmi) from a host thread while the GPU
    works; reads nothing on the GPU, so it does not disturb the kernels.  The driver refreshes this
    table only every ~0.1 s, so the sampler runs over a window of extra steps of its own (after the
    timed ones) and drops the first `delay_s` (values from before the GPU got busy)."""

    def __init__(self, period_s=0.004, delay_s=0.8):
        self.delay = delay_s
        import threading
        self.period = period_s
        self.samples = []
        self.error = None
        self._stop = threading.Event()
        self._thread = None
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            self._smi = amdsmi
            self._h = amdsmi.amdsmi_get_processor_handles()[0]
            self._read()   # fail early if the metric is not readable
        except Exception as e:   # no amdsmi, no permission, no device
            self._smi = None
            self.error = f"{type(e).__name__}: {e}"

    def _read(self):
        m = self._smi.amdsmi_get_gpu_metrics_info(self._h)
        vals = m.get("current_gfxclks")
        if isinstance(vals, (list, tuple)):
            vals = [v for v in vals if isinstance(v, (int, float)) and 0 < v < 10000]
        else:
            vals = []
        if not vals:
            v = m.get("current_gfxclk")
            vals = [v] if isinstance(v, (int, float)) and 0 < v < 10000 else []
        return vals

    def _run(self):
        import time as _t
        if self._stop.wait(self.delay):
            return
        while not self._stop.is_set():
            try:
                self.samples.extend(self._read())
            except Exception as e:
                self.error = f"{type(e).__name__}: {e}"
                return
            _t.sleep(self.period)

    def start(self):
        import threading
        if self._smi is None:
            return
        self._thread = threading.Thread(target=self._run, daemon=True)
        self._thread.start()

    def stop(self):
        if self._thread is not None:
            self._stop.set()
            self._thread.join()
        if self._smi is not None:
            try:
                self._smi.amdsmi_shut_down()
            except Exception:
                pass

    def summary(self):
        if not self.samples:
            return {"gfx_mhz_median": None, "samples": 0, "source": "amdsmi current_gfxclks",
                    "error": self.error or "no samples"}
        v = sorted(self.samples)
        q = lambda f: v[min(len(v) - 1, int(f * (len(v) - 1) + 0.5))]
        return {"gfx_mhz_median": q(0.5), "gfx_mhz_p10": q(0.1), "gfx_mhz_p90": q(0.9), "samples": len(v),
                "source": "amdsmi gpu_metrics current_gfxclks (every XCD), sampled every 4 ms over ~1.2 s of "
                          "extra steps run after the timed ones (the first 0.8 s dropped)"}


def fp8_dtype(a):
    """The arithmetic types of the run: bf16, or which expert products run on E4M3 operands."""
    parts = [n for n, on in (("forward", a.fp8_forward), ("data-gradient", a.fp8_backward),
                              ("weight-gradient", getattr(a, "fp8_dw", False))) if on]
    kind = "mxfp8-e4m3" if getattr(a, "mx", False) else "fp8-e4m3"
    return f"{kind} ({' and '.join(parts)} expert products) + bf16" if parts else "bf16"


def valu_record(flops, nbytes, avg_ms):
    """An fp32 vector-ALU call with its HBM bytes, scored against whichever roof its arithmetic
    intensity reaches first: below the ridge (157.3 TFLOP/s over 8 TB/s, 19.7 FLOP/B) it is HBM-bound."""
    rec = {"tflops_fp32": round(flops / avg_ms / 1e9, 1), "gbs": round(nbytes / avg_ms / 1e6, 1),
           "intensity_flop_per_byte": round(flops / nbytes, 2)}
    if flops / nbytes < VALU_RIDGE:
        rec["bound"] = "hbm"
        rec["frac_peak"] = round(nbytes / avg_ms / 1e6 / PEAK_HBM_GBS, 4)
    else:
        rec["bound"] = "valu"
        rec["frac_peak"] = round(flops / avg_ms / 1e9 / PEAK_FP32_VALU_TFLOPS, 4)
    return rec


def _stats(ts):
    v = sorted(ts)
    q = lambda f: v[min(len(v) - 1, int(f * (len(v) - 1) + 0.5))]
    return {"median": round(q(0.5), 4), "p10": round(q(0.1), 4), "p90": round(q(0.9), 4),
            "min": round(v[0], 4), "max": round(v[-1], 4)}


def copy_probe(nbytes):
    """A plain copy of known size: the reference that scales the HBM byte counters."""
    import torch
    a = torch.ones(nbytes // 2, dtype=torch.bfloat16, device="cuda:0")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes, "copies": 3}), flush=True)


def gemm_probe(kind, cfg):
    """The gate/up-shaped grouped product of one kind on uniform groups (R/E rows each), three
    launches: fwd H_g, H_u (+ SwiGLU) = X·W_{g,u}; dX = dH_g·W_gᵀ + dH_u·W_uᵀ; dW_{g,u} = Xᵀ·dH_{g,u}."""
    import torch

    from paper_2606_26453_amd import moe
    dev = "cuda:0"
    g = torch.Generator(device=dev).manual_seed(0)
    R, d, f, E = cfg.T * cfg.k, cfg.d, cfg.f, cfg.E
    off = torch.tensor([R * e // E for e in range(E + 1)], dtype=torch.int32, device=dev)
    rn = lambda *sh: torch.randn(sh, generator=g, device=dev).to(torch.bfloat16)
    if kind == "fwd":
        A, B, B2 = rn(R, d), rn(E, d, f), rn(E, d, f)
        fn = lambda: moe.moe_grouped_gemm_fwd(A, B, off, B2, want_act=True)
    elif kind == "dx":
        dC, dC2, B, B2 = rn(R, f), rn(R, f), rn(E, d, f), rn(E, d, f)
        fn = lambda: moe.moe_grouped_gemm_dx(dC, B, off, dC2, B2)
    else:
        A, dC, dC2 = rn(R, d), rn(R, f), rn(R, f)
        fn = lambda: moe.moe_grouped_gemm_dw(A, dC, off, dC2)
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    print(json.dumps({"gemm_probe": kind, "R": R, "d": d, "f": f, "E": E, "launches": 3}), flush=True)


def vendor_loop():
    """Context for the grouped kernels: the same products as a loop of per-expert vendor GEMMs
    (hipBLASLt through torch.matmul on contiguous operands; the transposed X_e of the weight gradient
    is copied out before timing).  Medians of 10 timed calls after 3 warm-up calls; each pair's
    results are compared (relative Frobenius distance)."""
    import torch

    from paper_2606_26453_amd import moe
    from paper_2606_26453_amd import workloads as W
    dev = "cuda:0"

    def med_ms(fn, reps=10, warm=3):
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ts = []
        for _ in range(reps):
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        return sorted(ts)[reps // 2]

    rel = lambda x, y: float((x.float() - y.float()).norm() / y.float().norm())
    out = {"metric": "vendor-loop context (not the benchmark metric)"}
    # the paper's dW1 shape: dW_{g,u}[e] = X_e^T dH_{g,u,e}, bf16 results
    cfg = W.CONFIGS[5]
    inp = W.make_dw_inputs(cfg, 0, dev)
    off, x, dg, du = inp["offsets"], inp["x_perm"], inp["dh_gate"], inp["dh_up"]
    o = off.cpu().tolist()
    E, d, f = cfg.E, cfg.d, cfg.f
    cnt = moe.dw_counters(dev)
    lg, lu = (torch.empty((E, d, f), dtype=torch.bfloat16, device=dev) for _ in range(2))
    lib_ms = med_ms(lambda: moe.moe_grouped_gemm_dw_bf16(x, dg, off, du, dB=lg, dB2=lu, counters=cnt))
    xt = [x[o[e]:o[e + 1]].t().contiguous() for e in range(E)]
    vg, vu = torch.empty_like(lg), torch.empty_like(lu)

    def loop_dw():
        for e in range(E):
            if o[e + 1] == o[e]:
                vg[e].zero_()
                vu[e].zero_()
            else:
                torch.matmul(xt[e], dg[o[e]:o[e + 1]], out=vg[e])
                torch.matmul(xt[e], du[o[e]:o[e + 1]], out=vu[e])
    loop_ms = med_ms(loop_dw)
    fl = 4.0 * x.shape[0] * d * f
    out["dw1_paper_shape"] = {"library_ms": round(lib_ms, 4), "vendor_loop_ms": round(loop_ms, 4),
                              "library_tflops": round(fl / lib_ms / 1e9, 1), "vendor_tflops": round(fl / loop_ms / 1e9, 1),
                              "rel_fro": max(rel(lg, vg), rel(lu, vu))}
    del inp, x, dg, du, lg, lu, xt, vg, vu
    torch.cuda.empty_cache()
    # the Mixtral-shaped gate/up forward on uniform groups (the library also computes the SwiGLU)
    cfg = W.CONFIGS[1]
    R, d, f, E = cfg.T * cfg.k, cfg.d, cfg.f, cfg.E
    g = torch.Generator(device=dev).manual_seed(0)
    o = [R * e // E for e in range(E + 1)]
    off = torch.tensor(o, dtype=torch.int32, device=dev)
    x = torch.randn((R, d), generator=g, device=dev).to(torch.bfloat16)
    wg, wu = ((torch.randn((E, d, f), generator=g, device=dev) * 0.02).to(torch.bfloat16) for _ in range(2))
    hg, hu, act = (torch.empty((R, f), dtype=torch.bfloat16, device=dev) for _ in range(3))
    ws = moe.split_workspace(dev)
    lib_ms = med_ms(lambda: moe.moe_grouped_gemm_fwd(x, wg, off, wu, C=hg, C2=hu, act=act, workspace=ws))
    vg, vu = torch.empty_like(hg), torch.empty_like(hu)

    def loop_fwd():
        for e in range(E):
            torch.matmul(x[o[e]:o[e + 1]], wg[e], out=vg[o[e]:o[e + 1]])
            torch.matmul(x[o[e]:o[e + 1]], wu[e], out=vu[o[e]:o[e + 1]])
    loop_ms = med_ms(loop_fwd)
    fl = 4.0 * R * d * f
    out["mixtral_gate_up_forward"] = {"library_ms (with SwiGLU)": round(lib_ms, 4), "vendor_loop_ms": round(loop_ms, 4),
                                      "library_tflops": round(fl / lib_ms / 1e9, 1),
                                      "vendor_tflops": round(fl / loop_ms / 1e9, 1),
                                      "rel_fro": max(rel(hg, vg), rel(hu, vu))}
    print(json.dumps(out), flush=True)


def cpu_baseline(cfg, inp, sample_tokens):
    """The CPU oracle (float64 numpy, as it stands) on a bounded sample of the same workload: the
    full layer forward+backward over the first `sample_tokens` tokens with all experts."""
    import numpy as np

    from oracle import moe_oracle as O
    f = lambda t: t.float().cpu().numpy().astype(np.float64)
    Ts = sample_tokens
    x, dy = f(inp["x"][:Ts]), f(inp["dy"][:Ts])
    logits = inp["logits"][:Ts].cpu().numpy()
    wg, wu, wd = f(inp["w_gate"]), f(inp["w_up"]), f(inp["w_down"])
    shared = None
    if cfg.f_shared:
        shared = (f(inp["w_gate_sh"]), f(inp["w_up_sh"]), f(inp["w_down_sh"]))
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        cores = max((i.get("num_threads", 1) for i in info), default=1)
    except Exception:
        cores = len(os.sched_getaffinity(0))
    t0 = time.perf_counter()
    fwd = O.layer_forward(x, logits, wg, wu, wd, cfg.k, shared=shared)
    O.layer_backward(fwd, x, dy, wg, wu, wd, shared=shared)
    dt = time.perf_counter() - t0
    return {"value": Ts / dt, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"full layer fwd+bwd (float64 numpy oracle) on the first {Ts} of {cfg.T} tokens, "
                      f"all {cfg.E} experts, {dt:.1f} s"}


def workload_name(i, cfg, router=False):
    if not cfg.dw_only:
        return f"config {i}: {cfg.name} MoE FFN layer fwd+bwd" + (" incl. router" if router else "")
    what = "dW1 (gate/up weight gradient) grouped GEMM" if cfg.dw1_only else "dW grouped GEMMs"
    extra = []
    if cfg.dirmult_alpha:
        extra.append(f"Dirichlet-Multinomial loads alpha={cfg.dirmult_alpha}")
    extra.append("bf16 output" if cfg.dw_bf16 else "fp32 output")
    return f"config {i}: {cfg.name} {what}, " + ", ".join(extra)


def all_configs(a):
    """One summary line over configurations 0-5: each layer (or dW-only workload) timed for a few
    steps after a warm-up, with its grouped-GEMM TFLOP/s from per-call events.  Not the headline."""
    import torch

    from paper_2606_26453_amd import layer as L
    from paper_2606_26453_amd import workloads as W
    dev = "cuda:0"
    torch.cuda.set_device(0)
    rows = []
    steps = max(3, min(a.steps, 10))
    for i in sorted(W.CONFIGS):
        cfg = W.CONFIGS[i]
        if cfg.dw_only:
            inp = W.make_dw_inputs(cfg, a.seed, dev)
            lay = L.DWOnly(cfg, inp)
        else:
            inp = W.make_inputs(cfg, a.seed, dev)
            lay = L.MoELayer(cfg, inp)
        for _ in range(2):
            lay.step()
        torch.cuda.synchronize()
        lay.trace = []
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            lay.step()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        work = lay.work()
        gms = gfl = 0.0
        for name, x0, x1 in lay.trace:
            if work[name][0] == "flops":
                gms += x0.elapsed_time(x1) / steps
                gfl += work[name][1]
        gfl /= steps
        rows.append({"config": i, "workload": workload_name(i, cfg), "ms_per_step": round(ms, 4),
                     "tokens_per_s": round(cfg.T / (ms / 1e3), 1),
                     "gemm_tflops": round(gfl / gms / 1e9, 1) if gms else None,
                     "gemm_frac_peak": round(gfl / gms / 1e9 / PEAK_BF16_TFLOPS, 4) if gms else None,
                     "gemm_tflops_step": round(cfg.gemm_flops() / (ms / 1e3) / 1e12, 1)})
        del lay, inp
        torch.cuda.empty_cache()
    print(json.dumps({"summary": "all configurations, 1 GPU, bf16, synthetic inputs", "steps": steps,
                      "configs": rows}), flush=True)


def main():
    a = _args()
    if a.gpus != 1:
        print(f"bench.py measures one GPU only (--gpus {a.gpus} requested): the library has no "
              f"multi-GPU path; run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if a.copy_probe:
        copy_probe(a.copy_probe)
        return
    if a.gemm_probe:
        from paper_2606_26453_amd import workloads as W
        gemm_probe(a.gemm_probe, W.CONFIGS[a.config])
        return
    if a.vendor_loop:
        vendor_loop()
        return
    if a.all_configs:
        all_configs(a)
        return
    import torch

    from paper_2606_26453_amd import layer as L
    from paper_2606_26453_amd import workloads as W

    dev = "cuda:0"
    torch.cuda.set_device(0)
    cfg = W.CONFIGS[a.config]
    t_gen = time.perf_counter()
    if cfg.dw_only:
        inp = W.make_dw_inputs(cfg, a.seed, dev)
        lay = L.DWOnly(cfg, inp, persistent=not a.dw_one_per_tile)
    else:
        inp = W.make_inputs(cfg, a.seed, dev)
        lay = L.MoELayer(cfg, inp, router=a.router, aux_alpha=a.aux_alpha if a.router else 0.0,
                         dw_transposed=a.dw_transposed, concurrent=a.concurrent, split_tail=not a.no_split_tail,
                         gather_fused=a.gather_fused, fp8_forward=a.fp8_forward,
                         fp8_backward=a.fp8_backward, fp8_requantize=not a.fp8_fixed_weights, mx=a.mx,
                         combine_fused=a.combine_fused, fp8_dw=a.fp8_dw,
                         dw_persistent=not a.dw_one_per_tile)
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t_gen

    stream = torch.cuda.current_stream()
    step = lay.forward if (a.forward_only and not cfg.dw_only) else lay.step
    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    if a.graph:   # from here on every step is one replay of the captured sequence
        lay.capture(step)
        torch.cuda.synchronize()
        step = lay.replay

    lay.trace = None if (a.no_trace or a.graph) else []
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    step_ev = [torch.cuda.Event(enable_timing=True) for _ in range(a.steps + 1)]
    torch.cuda.synchronize()
    start.record(stream)
    step_ev[0].record(stream)
    for i in range(a.steps):
        step()
        step_ev[i + 1].record(stream)
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / a.steps
    step_ms = [step_ev[i].elapsed_time(step_ev[i + 1]) for i in range(a.steps)]
    trace = lay.trace
    lay.trace = None

    # the shader clock under this workload: ~2 s of further steps, sampled from the host
    clock = None if a.no_clock else ClockSampler()
    if clock:
        clock.start()
        for _ in range(max(10, int(2000 / max(ms_per_step, 0.01)))):
            step()
        torch.cuda.synchronize()
        clock.stop()

    # per-call averages over the timed region
    per = {}
    for name, e0, e1 in (trace or []):
        per.setdefault(name, []).append(e0.elapsed_time(e1))
    work = lay.work()
    calls = {}
    gemm_ms = gemm_flops = 0.0
    variant = (a.fp8_forward or a.fp8_backward or a.gather_fused or a.dw_transposed or a.no_split_tail
               or a.dw_one_per_tile or a.concurrent or a.combine_fused or a.fp8_dw)
    for name, ts in per.items():
        avg = sum(ts) / len(ts)
        kind, amount = work[name]
        rec = {"ms": round(avg, 4)}
        if kind == "flops":
            rec["tflops"] = round(amount / avg / 1e9, 1)
            rec["frac_peak"] = round(amount / avg / 1e9 / PEAK_BF16_TFLOPS, 4)
            gemm_ms += avg
            gemm_flops += amount
        elif kind == "flops8":
            rec["tflops_fp8"] = round(amount / avg / 1e9, 1)
            rec["frac_peak"] = round(amount / avg / 1e9 / PEAK_FP8_TFLOPS, 4)
        elif kind == "valu":
            rec.update(valu_record(*amount, avg))
        else:
            rec["gbs"] = round(amount / avg / 1e6, 1)
            rec["frac_peak"] = round(amount / avg / 1e6 / PEAK_HBM_GBS, 4)
        hbm = measured_traffic(name, a.config, variant)
        if hbm is not None:   # counter bytes over the algorithmic bytes or operand+output bytes
            rec["hbm_bytes_measured"] = hbm
        calls[name] = rec

    roofline = None
    if per:
        dom = max((n for n in per if work[n][0] != "valu"), key=lambda n: sum(per[n]))
        kind, amount = work[dom]
        avg = sum(per[dom]) / len(per[dom])
        if kind in ("flops", "flops8"):
            ach = amount / avg / 1e9
            peak = PEAK_BF16_TFLOPS if kind == "flops" else PEAK_FP8_TFLOPS
            roofline = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 1), "peak": peak,
                        "unit": "TFLOP/s", "frac": round(ach / peak, 4),
                        "traffic": measured_traffic(dom, a.config, variant) if kind == "flops" else None,
                        "work_per_launch": amount, "avg_launch_ms": round(avg, 4)}
        else:
            ach = amount / avg / 1e6
            roofline = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                        "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
                        "traffic": measured_traffic(dom, a.config, variant),
                        "work_per_launch": amount, "avg_launch_ms": round(avg, 4)}

    clock_info = clock.summary() if clock else None
    mhz = clock_info.get("gfx_mhz_median") if clock_info else None
    if roofline is not None:
        roofline["sustained_clock_mhz"] = mhz
        roofline["frac_at_sustained_clock"] = (round(roofline["frac"] * PEAK_CLOCK_MHZ / mhz, 4) if mhz else None)
        roofline["clock_source"] = (clock_info or {}).get("source")

    flushed = None
    if a.flush:
        # each step alone, after a 1 GiB read (4x the 256 MB Infinity Cache), timed by its own events
        lay.trace = None
        junk = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)
        sink = torch.empty(1, dtype=torch.float32, device=dev)
        ts = []
        for _ in range(a.steps):
            torch.sum(junk, dim=0, keepdim=True, out=sink)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            step()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        flushed = _stats(ts)
        del junk

    tokens = cfg.T
    value = tokens * a.steps / (total_ms / 1e3)
    offs = (inp["offsets"] if cfg.dw_only else lay.buf["offsets"]).cpu().tolist()
    counts = [offs[i + 1] - offs[i] for i in range(len(offs) - 1)]
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": fp8_dtype(a),
        "data": "synthetic (seeded N(0,1) activations, N(0,0.02) weights, router logits X.Wr)",
        "config": {"workload": workload_name(a.config, cfg, a.router and not cfg.dw_only)
                   + (" (forward only)" if a.forward_only and not cfg.dw_only else "")
                   + (", expert forward products in FP8 E4M3" if a.fp8_forward else "")
                   + (", expert data-gradient products in FP8 E4M3" if a.fp8_backward else "")
                   + (", MX block scales (E8M0 per 32 contraction elements)" if a.mx else "")
                   + (", expert weight-gradient products in MX FP8" if a.fp8_dw else "")
                   + (", FP8 weights quantized once (held fixed)" if a.fp8_fixed_weights else "")
                   + (", gather fused into the gate/up product" if a.gather_fused else "")
                   + (", combine fused into the down product" if a.combine_fused else "")
                   + (", HIP graph replay" if a.graph else "")
                   + (", dW from contraction-major copies" if a.dw_transposed else "")
                   + (", no split tail" if a.no_split_tail else "")
                   + (", dW one workgroup per tile" if a.dw_one_per_tile else "")
                   + (", two streams" if a.concurrent else ""),
                   "T": cfg.T, "d": cfg.d, "f": cfg.f, "E": cfg.E, "k": cfg.k, "f_shared": cfg.f_shared,
                   "parallelism": "single GPU"},
        "gemm_tflops": round(gemm_flops / gemm_ms / 1e9, 1) if gemm_ms else None,
        "gemm_frac_peak": round(gemm_flops / gemm_ms / 1e9 / PEAK_BF16_TFLOPS, 4) if gemm_ms else None,
        "gemm_tflops_step": round(cfg.gemm_flops() * (1 / 3 if a.forward_only else 1) / (ms_per_step / 1e3) / 1e12, 1),
        "step_ms": _stats(step_ms),
        "flushed_step_ms": flushed,
        "clock": clock_info,
        "calls": calls,
        "roofline": roofline,
        "groups": W.group_stats(counts),
        "input_gen_s": round(t_gen, 1),
    }
    if not a.no_cpu_baseline and not cfg.dw_only and not (a.fp8_forward or a.fp8_backward or a.forward_only):
        ts = a.cpu_sample_tokens or max(8, min(cfg.T, int(6e12 // (18 * cfg.k * cfg.d * cfg.f))))
        out["cpu_baseline"] = cpu_baseline(cfg, inp, ts)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
