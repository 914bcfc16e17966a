"""Shared helpers of the GPU parity tests (tolerances, error metrics, input staging)."""
import sys

import numpy as np
import torch

# Parity bar: normwise max relative error ||x - ref||_inf / ||ref||_inf per output
# tensor (and per layer), 1e-4 for fp32 runs and 2e-2 for bf16 runs.
TOL = {"f32": 1e-4, "bf16": 2e-2}


def say(*args):
    print(*args, flush=True)
    sys.stdout.flush()


def rel_err(x, ref) -> float:
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = float(np.max(np.abs(ref)))
    num = float(np.max(np.abs(x - ref)))
    if den == 0.0:
        return num
    return num / den


def assert_close(x, ref, dtype: str, what: str):
    e = rel_err(x, ref)
    assert np.all(np.isfinite(np.asarray(x, dtype=np.float64))), f"{what}: non-finite output"
    assert e <= TOL[dtype], f"{what}: normwise relative error {e:.3e} > {TOL[dtype]:.0e}"
    return e


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu").to(torch.float64).numpy()


def cuda(t: torch.Tensor) -> torch.Tensor:
    return t.to("cuda:0").contiguous()
