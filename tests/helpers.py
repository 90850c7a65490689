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


def rel_err(got, ref, allow=None) -> float:
    """max |got - ref| / max |ref| (the parity measure for floating outputs).

    ``allow`` (same shape, optional) is an elementwise bound on how far
    decisions the oracle marks as ambiguous may move the result; only the
    excess beyond it counts."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    diff = np.abs(got - ref)
    if allow is not None:
        diff = np.maximum(diff - np.asarray(allow, dtype=np.float64), 0.0)
    den = np.abs(ref).max() if ref.size else 0.0
    if den == 0.0:
        return float(diff.max()) if got.size else 0.0
    return float(diff.max() / den)


def announce(*parts):
    print("CASE", *parts, flush=True)
