"""Helpers for the GPU parity tests (tensor <-> float64 numpy, tolerance checks)."""
import numpy as np
import torch

from oracle import moe_oracle as O

FRO_TOL = 2e-2   # Frobenius-relative error bar for floating outputs (bf16 in, fp32 accumulate)


def gpu_available():
    try:
        return torch.cuda.is_available()
    except Exception:
        return False


def f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def i64(t):
    return t.detach().cpu().numpy().astype(np.int64)


def check_float(name, got, ref, tol=FRO_TOL, log=None):
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    err = O.rel_fro(got, ref)
    if log is not None:
        log[name] = err
    assert err <= tol, f"{name}: Frobenius-relative error {err:.3e} > {tol}"
    return err


def poison_(t):
    """Fill an output buffer with NaN (float) or a sentinel (int) so unwritten elements show."""
    if t.dtype.is_floating_point:
        t.fill_(float("nan"))
    else:
        t.fill_(-7)
    return t
