"""Input generators (no GPU): the Dirichlet-Multinomial expert loads of the paper's dW1 shape."""
import numpy as np

from paper_2606_26453_amd import workloads as W


def test_dirmult_counts_basic():
    c = W.CONFIGS[5]
    a = np.array(W.dirmult_counts(c.E, c.R, c.dirmult_alpha, 0))
    assert a.sum() == c.R == 57768 and len(a) == 128 and (a >= 0).all()
    assert (a == 0).any()                              # alpha = 0.24 leaves experts empty
    assert a.tolist() == W.dirmult_counts(c.E, c.R, c.dirmult_alpha, 0)   # seeded


def test_dirmult_counts_moments():
    """Mean and variance of one expert's count over many draws match the Dirichlet-Multinomial
    closed forms: E = R/E_n, Var = R (1/E_n)(1 - 1/E_n)(R + E_n a) / (1 + E_n a)."""
    En, R, al = 16, 400, 0.5
    x = np.array([W.dirmult_counts(En, R, al, s)[3] for s in range(3000)], dtype=np.float64)
    p = 1.0 / En
    var = R * p * (1 - p) * (R + En * al) / (1 + En * al)
    assert abs(x.mean() - R * p) < 4 * np.sqrt(var / len(x))
    assert abs(x.var() / var - 1) < 0.15


def test_paper_dw1_config():
    c = W.CONFIGS[5]
    assert (c.d, c.f, c.E, c.k, c.R) == (2880, 2880, 128, 4, 57768)
    assert c.dw_only and c.dw1_only and c.dw_bf16
    assert c.gemm_flops() == 4 * 57768 * 2880 * 2880        # dW1: X^T [dH_g | dH_u], N = 5760
