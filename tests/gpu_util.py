"""Helpers for the GPU parity tests: device transfer and the comparison metric."""
from __future__ import annotations

import os
import sys

import numpy as np
import torch

from paper_2607_02945_amd import synth

# Tolerances: fp32 members 1e-5, bf16 storage with fp32 accumulation 2e-2,
# both as an inf-normwise relative error per member (or per piece): elementwise
# relative error is unbounded where LayerNorm or tanh outputs pass near zero.
TOL = {"fp32": 1e-5, "bf16": 2e-2}


def say(*a):
    """Name the case before a GPU step (flushed, so a fault still shows it)."""
    print(*a, flush=True)
    sys.stdout.flush()


def dev(t):
    return None if t is None else t.to("cuda", non_blocking=False)


def host64(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return synth.exact64(t)


def normwise(gpu: np.ndarray, ref: np.ndarray) -> float:
    ref = np.asarray(ref, np.float64)
    return float(np.max(np.abs(np.asarray(gpu, np.float64) - ref)) / max(float(np.max(np.abs(ref))), 1e-30))


def elementwise(gpu: np.ndarray, ref: np.ndarray) -> float:
    """Diagnostic only (not a pass criterion): max_i |g_i - r_i| / (|r_i| + rms(r)).
    The rms term keeps it bounded where LayerNorm or tanh outputs pass near 0."""
    ref = np.asarray(ref, np.float64)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    den = np.abs(ref) + max(rms, 1e-30)
    return float(np.max(np.abs(np.asarray(gpu, np.float64) - ref) / den)) if ref.size else 0.0


# worst elementwise diagnostic per (test, dtype), printed in the run's summary
DIAG = {}


def assert_close(gpu, ref, dtype: str, what: str = ""):
    e = normwise(gpu, ref)
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite output"
    assert e <= TOL[dtype], f"{what}: normwise rel err {e:.3e} > {TOL[dtype]:.0e}"
    test = os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0]
    key = (test, dtype)
    d = elementwise(gpu, ref)
    if d > DIAG.get(key, (-1.0, ""))[0]:
        DIAG[key] = (d, what)
    return e


def empty_like_rows(rows, cols, dtype, fill=float("nan")):
    return torch.full((rows, cols), fill, dtype=synth.DTYPES[dtype], device="cuda")
