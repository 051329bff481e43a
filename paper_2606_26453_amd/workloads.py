"""Seeded synthetic workloads for the MoE expert-FFN training layer.

This module only draws inputs; it holds none of the layer's arithmetic. Both the GPU path's
tests/bench and the CPU oracle consume the tensors it returns, so they see the same bytes.

Shapes and distributions follow the five layer configurations this library is measured on
(tiny, Mixtral-shaped, fine-grained with shared experts, Zipf-skewed routing, and a
weight-gradient-only long batch).  The paper measures its grouped GEMM on GPT-OSS-120B routing
statistics from a long-context benchmark (Appendix H, "Estimating the token-to-expert
distribution"); neither that model nor that dataset is used here: seeded Gaussian activations and
weights and router logits X.Wr stand in for them.

Draw order (one torch.Generator per call, seeded): X, Wr, W_gate, W_up, W_down,
[shared W_gate, W_up, W_down], dY, [Zipf expert permutation].  Normal draws are float32,
multiplied by their standard deviation, then rounded to bfloat16 (round-to-nearest-even).
"""
from __future__ import annotations

import dataclasses
import math

import torch


@dataclasses.dataclass(frozen=True)
class MoEConfig:
    name: str
    T: int            # tokens
    d: int            # hidden size
    f: int            # expert FFN width
    E: int            # experts
    k: int            # experts per token (top-k)
    f_shared: int = 0  # width of the always-on shared FFN (0 = none)
    zipf_s: float = 0.0      # Zipf exponent of the per-expert logit bias profile (0 = no bias)
    zipf_beta: float = 0.0   # bias scale: bias_e = beta * ln(z_rank(e))
    dw_only: bool = False    # weight-gradient path only, exactly uniform groups
    dirmult_alpha: float = 0.0   # dw_only: group sizes ~ Dirichlet(alpha)-Multinomial(R) instead
    dw1_only: bool = False   # dw_only: only the gate/up weight gradient (the paper's dW1)
    dw_bf16: bool = False    # dw_only: weight gradients stored in bf16 (the paper's output dtype)

    @property
    def R(self) -> int:
        return self.T * self.k

    def gemm_flops(self) -> int:
        """Algorithmic FLOPs of all grouped GEMMs of one step (only real rows, no padding)."""
        if self.dw_only:
            return (4 if self.dw1_only else 6) * self.R * self.d * self.f
        fl = 18 * self.R * self.d * self.f
        if self.f_shared:
            fl += 18 * self.T * self.d * self.f_shared
        return fl


CONFIGS = {
    0: MoEConfig("tiny", T=256, d=256, f=512, E=4, k=2),
    1: MoEConfig("mixtral", T=8192, d=4096, f=14336, E=8, k=2),
    2: MoEConfig("fine_grained_shared", T=16384, d=2048, f=1408, E=64, k=6, f_shared=2 * 1408),
    3: MoEConfig("zipf_skew", T=16384, d=4096, f=2048, E=32, k=4, zipf_s=1.2, zipf_beta=1.5),
    4: MoEConfig("dw_long_batch", T=65536, d=4096, f=4096, E=16, k=2, dw_only=True),
    # The paper's own measurement shape (section 5.4, Appendix H): GPT-OSS-120B's gate_up_proj
    # weight gradient dW1 (hidden 2880, gate and up 2880 each), 128 experts, top-4, 57,768 routed
    # rows, expert loads from the paper's Dirichlet-Multinomial fit (alpha = 0.24, empty experts
    # possible), bf16 output.  Synthetic operands stand in for the model's activations.
    5: MoEConfig("paper_dw1_gptoss", T=14442, d=2880, f=2880, E=128, k=4, dw_only=True,
                 dirmult_alpha=0.24, dw1_only=True, dw_bf16=True),
}

ACT_STD = 1.0
W_STD = 0.02
ROUTER_STD = 0.02


def custom(name="custom", **kw) -> MoEConfig:
    return MoEConfig(name=name, **kw)


def _normal(shape, std, gen, device, dtype=torch.bfloat16):
    x = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(dtype)


def zipf_bias(cfg: MoEConfig, gen: torch.Generator, device="cpu") -> torch.Tensor:
    """Per-expert logit bias bias_e = beta * ln(z_rank(e)), z = normalised Zipf(s) over E ranks,
    expert<->rank assignment drawn by a seeded permutation."""
    ranks = torch.arange(1, cfg.E + 1, dtype=torch.float64)
    z = ranks.pow(-cfg.zipf_s)
    z = z / z.sum()
    perm = torch.randperm(cfg.E, generator=gen, device=device).cpu()
    bias = torch.empty(cfg.E, dtype=torch.float64)
    bias[perm] = cfg.zipf_beta * torch.log(z)
    return bias.to(torch.float32)


def make_inputs(cfg: MoEConfig, seed: int = 0, device="cpu", expert_bias=None,
                want_dy: bool = True) -> dict:
    """Draw one seeded input set for `cfg` on `device`.

    Returns bf16 tensors x [T,d], w_gate/w_up [E,d,f], w_down [E,f,d], dy [T,d], the float32
    router weight wr [d,E] and logits [T,E] (= x.float() @ wr, plus the Zipf bias / `expert_bias`,
    which is also returned as router_bias [E] when present), and for a shared-FFN config
    w_gate_sh/w_up_sh [d,f_sh], w_down_sh [f_sh,d].  The logits are computed once here and
    handed bit-identically to the oracle and to the GPU path.
    """
    if cfg.dw_only:
        return make_dw_inputs(cfg, seed, device)
    gen = torch.Generator(device=device).manual_seed(seed)
    T, d, f, E = cfg.T, cfg.d, cfg.f, cfg.E
    out = {}
    out["x"] = _normal((T, d), ACT_STD, gen, device)
    wr = _normal((d, E), ROUTER_STD, gen, device, dtype=torch.float32)
    out["wr"] = wr
    out["w_gate"] = _normal((E, d, f), W_STD, gen, device)
    out["w_up"] = _normal((E, d, f), W_STD, gen, device)
    out["w_down"] = _normal((E, f, d), W_STD, gen, device)
    if cfg.f_shared:
        fs = cfg.f_shared
        out["w_gate_sh"] = _normal((d, fs), W_STD, gen, device)
        out["w_up_sh"] = _normal((d, fs), W_STD, gen, device)
        out["w_down_sh"] = _normal((fs, d), W_STD, gen, device)
    if want_dy:
        out["dy"] = _normal((T, d), ACT_STD, gen, device)
    logits = out["x"].float() @ wr
    bias = None
    if cfg.zipf_s:
        bias = zipf_bias(cfg, gen, device).to(device)
    if expert_bias is not None:
        eb = torch.as_tensor(expert_bias, dtype=torch.float32, device=device)
        bias = eb if bias is None else bias + eb
    if bias is not None:
        logits += bias
        out["router_bias"] = bias        # [E] fp32: the per-expert logit bias (absent: none)
    out["logits"] = logits.contiguous()
    return out


def dirmult_counts(E: int, R: int, alpha: float, seed: int = 0):
    """Rows per expert drawn as p ~ Dirichlet(alpha, ..., alpha) over E experts, then
    counts ~ Multinomial(R, p) (the load model fitted in Appendix H, "Estimating the token-to-expert
    distribution").  numpy's seeded generator; small alpha leaves some experts empty."""
    import numpy as np
    rng = np.random.default_rng(seed)
    p = rng.dirichlet([alpha] * E)
    return [int(v) for v in rng.multinomial(R, p)]


def make_dw_inputs(cfg: MoEConfig, seed: int = 0, device="cpu", counts=None) -> dict:
    """Operands of the weight-gradient-only workload: exactly uniform groups (R/E rows each), or
    Dirichlet-Multinomial group sizes when cfg.dirmult_alpha > 0, unless `counts` is given;
    x_perm [R,d], dh_gate/dh_up [R,f] and (unless cfg.dw1_only) act [R,f], dy_perm [R,d] ~ N(0,1)
    bf16."""
    gen = torch.Generator(device=device).manual_seed(seed)
    R, d, f, E = cfg.R, cfg.d, cfg.f, cfg.E
    if counts is None and cfg.dirmult_alpha > 0:
        counts = dirmult_counts(E, R, cfg.dirmult_alpha, seed)
    if counts is None:
        assert R % E == 0
        counts = [R // E] * E
    counts = torch.as_tensor(counts, dtype=torch.int64)
    assert int(counts.sum()) == R and counts.numel() == E
    offsets = torch.zeros(E + 1, dtype=torch.int32)
    offsets[1:] = torch.cumsum(counts, 0).to(torch.int32)
    out = {"offsets": offsets.to(device), "x_perm": _normal((R, d), ACT_STD, gen, device)}
    if not cfg.dw1_only:
        out["act"] = _normal((R, f), ACT_STD, gen, device)
    out["dh_gate"] = _normal((R, f), ACT_STD, gen, device)
    out["dh_up"] = _normal((R, f), ACT_STD, gen, device)
    if not cfg.dw1_only:
        out["dy_perm"] = _normal((R, d), ACT_STD, gen, device)
    return out


def small_int_(t: torch.Tensor, gen: torch.Generator, lo=-1, hi=1, density=1.0) -> torch.Tensor:
    """Overwrite `t` with integers in [lo, hi] (optionally sparse); used to make GEMM results exact."""
    v = torch.randint(lo, hi + 1, t.shape, generator=gen, device=t.device).to(t.dtype)
    if density < 1.0:
        keep = torch.rand(t.shape, generator=gen, device=t.device) < density
        v = v * keep.to(t.dtype)
    t.copy_(v)
    return t


def group_stats(counts) -> dict:
    c = [int(v) for v in counts]
    n = len(c)
    mean = sum(c) / n
    var = sum((v - mean) ** 2 for v in c) / n
    return {"min": min(c), "max": max(c), "mean": mean,
            "cv": (math.sqrt(var) / mean) if mean else 0.0,
            "empty": sum(1 for v in c if v == 0), "under64": sum(1 for v in c if v < 64)}
