"""Shared helpers for the GPU parity tests (device setup, comparisons)."""

import numpy as np
import pytest

TOL = {"f32": 1e-4, "bf16": 2e-2}


def gpu_lib():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2402_15106_amd as dm
    return dm, dm.Dsmp(0), torch


def rel_err(got, ref) -> float:
    """max |got - ref| / max |ref| (the parity measure for floating outputs)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.abs(ref).max() if ref.size else 0.0
    if den == 0.0:
        return float(np.abs(got).max()) if got.size else 0.0
    return float(np.abs(got - ref).max() / den)


def announce(*parts):
    print("CASE", *parts, flush=True)
