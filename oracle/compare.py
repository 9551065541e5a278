"""Comparison rules between a result under test and the fp64 oracle.

TEST INFRASTRUCTURE ONLY (imported by tests, the smoke check and the benchmark).

Tolerances:
  * fp32 partial sums of squares: relative error <= 1e-5.
  * bf16 outputs: relative error <= 8e-3 (about two bf16 ulps) per element;
    where the oracle is exactly 0 the result must be exactly 0; NaN must match
    NaN and infinities must match in sign.
Error metrics reported next to them are the three the paper uses against its
fp64 gold output (Sec. IV-C): maximum, mean and RMS absolute error.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

PARTIAL_RTOL = 1e-5
OUTPUT_RTOL = 8e-3


def rel_error(test: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """|test - ref| / |ref| elementwise; 0 where both are 0, inf where only ref is 0."""
    test = np.asarray(test, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    diff = np.abs(test - ref)
    mag = np.abs(ref)
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(mag > 0, diff / np.where(mag > 0, mag, 1.0),
                     np.where(diff == 0, 0.0, np.inf))
    return r


def check_close(test: np.ndarray, ref: np.ndarray, rtol: float, what: str) -> float:
    """Assert elementwise relative agreement with special values matched.

    Returns the largest relative error over finite elements.
    """
    test = np.asarray(test, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if test.shape != ref.shape:
        raise AssertionError(f"{what}: shape {test.shape} != {ref.shape}")
    nan_t, nan_r = np.isnan(test), np.isnan(ref)
    if not np.array_equal(nan_t, nan_r):
        bad = np.argwhere(nan_t != nan_r)[:5]
        raise AssertionError(f"{what}: NaN mismatch at {bad.tolist()}")
    inf_r = np.isinf(ref)
    if not np.array_equal(np.isinf(test), inf_r) or \
            not np.array_equal(test[inf_r], ref[inf_r]):
        raise AssertionError(f"{what}: infinity mismatch")
    fin = ~(nan_r | inf_r)
    if not fin.any():
        return 0.0
    r = rel_error(test[fin], ref[fin])
    worst = float(r.max())
    if not worst <= rtol:
        idx = np.argwhere(fin)[int(np.argmax(r))]
        raise AssertionError(
            f"{what}: max rel err {worst:.3e} > {rtol:.1e} at {idx.tolist()} "
            f"(test {test[tuple(idx)]!r}, oracle {ref[tuple(idx)]!r})")
    return worst


def paper_error_metrics(test: np.ndarray, ref: np.ndarray) -> Dict[str, float]:
    """Max, mean and RMS absolute error against the fp64 reference (Sec. IV-C)."""
    test = np.asarray(test, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    fin = np.isfinite(ref) & np.isfinite(test)
    d = np.abs(test[fin] - ref[fin])
    if d.size == 0:
        return {"max_abs": 0.0, "mean_abs": 0.0, "rms_abs": 0.0}
    return {"max_abs": float(d.max()), "mean_abs": float(d.mean()),
            "rms_abs": float(np.sqrt(np.mean(d * d)))}
