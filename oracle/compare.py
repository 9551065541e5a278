"""Comparison rules between a result under test and the fp64 oracle.

TEST INFRASTRUCTURE ONLY (imported by tests, the smoke check and the benchmark).

Tolerances:
  * fp32 partial sums of squares: relative error <= 1e-5.
  * bf16 outputs: relative error <= 8e-3 (about two bf16 ulps) per element;
    where the oracle is exactly 0 the result must be exactly 0; NaN must match
    NaN and infinities must match in sign.
  * FP8-E4M3 outputs (``check_fp8``): the result must be what rounding to
    nearest gives for some value within a relative FP8_NOISE of the fp64
    oracle (the fp32 arithmetic before the final rounding is that close), i.e.
    |y - ref| <= half an FP8 step at |ref| (1 + noise) + noise |ref|; values
    that round past 448 must be NaN (the format has no infinity).
Error metrics reported next to them are the three the paper uses against its
fp64 gold output (Sec. IV-C): maximum, mean and RMS absolute error.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

PARTIAL_RTOL = 1e-5
OUTPUT_RTOL = 8e-3
FP8_NOISE = 1e-5
E4M3_MAX = 448.0
E4M3_OVERFLOW = 464.0  # halfway between 448 and the next step, 480, which has no code


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


def e4m3_half_step(mag: np.ndarray) -> np.ndarray:
    """Half the FP8-E4M3 grid step at magnitude `mag` (>= 0).

    Step 2^(k-3) in the binade [2^k, 2^(k+1)) for k >= -6, and 2^-9 below 2^-6
    (subnormals, same step as the first normal binade).
    """
    mag = np.asarray(mag, dtype=np.float64)
    k = np.frexp(np.where(mag > 0, mag, 1.0))[1] - 1
    k = np.where(mag > 0, np.maximum(k, -6), -6)
    return np.exp2(k - 4.0)


def check_fp8(test: np.ndarray, ref: np.ndarray, what: str, noise: float = FP8_NOISE) -> float:
    """Assert that decoded FP8-E4M3 results are ref rounded to nearest, up to `noise`.

    test: the results decoded to fp64; ref: the fp64 oracle. Returns the largest
    error in units of half an FP8 step (<= 1 + a little when the check passes).
    """
    test = np.asarray(test, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if test.shape != ref.shape:
        raise AssertionError(f"{what}: shape {test.shape} != {ref.shape}")
    if np.isinf(test).any():
        raise AssertionError(f"{what}: FP8 results cannot be infinite")
    mag = np.abs(ref)
    with np.errstate(invalid="ignore"):
        must_nan = np.isnan(ref) | (mag * (1 - noise) > E4M3_OVERFLOW)
        may_nan = must_nan | (mag * (1 + noise) > E4M3_OVERFLOW)
    nan_t = np.isnan(test)
    if (must_nan & ~nan_t).any() or (nan_t & ~may_nan).any():
        bad = np.argwhere((must_nan & ~nan_t) | (nan_t & ~may_nan))[:5]
        raise AssertionError(f"{what}: NaN mismatch at {bad.tolist()}")
    fin = ~nan_t & ~must_nan
    if not fin.any():
        return 0.0
    r, t = ref[fin], test[fin]
    zero = r == 0
    if (t[zero] != 0).any():
        raise AssertionError(f"{what}: nonzero result where the oracle is exactly 0")
    half = e4m3_half_step(np.abs(r) * (1 + noise))
    err = np.abs(t - r)
    bound = half + noise * np.abs(r)
    if not np.all(err <= bound):
        i = int(np.argmax(err - bound))
        idx = np.argwhere(fin)[i]
        raise AssertionError(
            f"{what}: FP8 result {t[i]!r} is not the rounding of oracle {r[i]!r} "
            f"at {idx.tolist()} (error {err[i]:.3e} > {bound[i]:.3e})")
    return float(np.max(err / half))


# ---------------------------------------------------------------- projection

FP32_UNIT = 2.0 ** -24  # unit roundoff of fp32


def bf16_step(mag: np.ndarray) -> np.ndarray:
    """bf16 grid step at magnitude `mag` (>= 0): 2^(e-7) in the binade
    [2^e, 2^(e+1)), e >= -126; the subnormal step 2^-133 below."""
    mag = np.asarray(mag, dtype=np.float64)
    k = np.frexp(np.where(mag > 0, mag, 1.0))[1] - 1
    k = np.where(mag > 0, np.maximum(k, -126), -126)
    return np.exp2(k - 7.0)


def projection_error_bound(q_exact: np.ndarray, dot_abs: np.ndarray, hidden: int) -> np.ndarray:
    """Largest |q_stored - q_exact| for q accumulated in fp32 (any order) over
    `hidden` exact bf16 products, then rounded once to bf16:
    eps = (hidden - 1) u sum|x w| for the sum (to first order, padded by 1 %),
    plus half a bf16 step at |q| + eps for the rounding."""
    eps = 1.01 * max(hidden - 1, 0) * FP32_UNIT * np.asarray(dot_abs, dtype=np.float64)
    return 0.5 * bf16_step(np.abs(q_exact) + eps) + eps


def check_projection(q_test: np.ndarray, q_exact: np.ndarray, dot_abs: np.ndarray,
                     hidden: int, what: str) -> float:
    """Assert |q_test - q_exact| <= projection_error_bound elementwise; returns
    the largest error as a fraction of its bound."""
    q_test = np.asarray(q_test, dtype=np.float64)
    q_exact = np.asarray(q_exact, dtype=np.float64)
    if q_test.shape != q_exact.shape:
        raise AssertionError(f"{what}: shape {q_test.shape} != {q_exact.shape}")
    if not np.isfinite(q_test).all():
        raise AssertionError(f"{what}: non-finite results")
    bound = projection_error_bound(q_exact, dot_abs, hidden)
    err = np.abs(q_test - q_exact)
    frac = np.where(bound > 0, err / np.where(bound > 0, bound, 1.0), np.where(err > 0, np.inf, 0.0))
    worst = float(frac.max()) if frac.size else 0.0
    if not worst <= 1.0:
        idx = np.unravel_index(int(np.argmax(frac)), frac.shape)
        raise AssertionError(f"{what}: |q - exact| = {err[idx]:.3e} > bound {bound[idx]:.3e} at "
                             f"{list(idx)} (q {q_test[idx]!r}, exact {q_exact[idx]!r})")
    return worst


def projection_partial_bound(q_exact: np.ndarray, dot_abs: np.ndarray, hidden: int) -> np.ndarray:
    """Largest |P_test - sum_j round_bf16(q_exact)^2| per token, where P_test is
    an fp32 sum of the squares of the stored values: each stored value differs
    from the correctly rounded one by at most delta = one bf16 step at |q| + eps
    plus eps; squares then differ by at most delta (2 |q| + 2 delta); the fp32
    sum of d squares adds at most d u of the total (padded by 1 %)."""
    q = np.abs(np.asarray(q_exact, dtype=np.float64))
    eps = 1.01 * max(hidden - 1, 0) * FP32_UNIT * np.asarray(dot_abs, dtype=np.float64)
    delta = bf16_step(q + eps) + eps
    d = q.shape[1]
    top = q + delta
    return np.sum(delta * (2 * q + 2 * delta), axis=1) + 1.01 * d * FP32_UNIT * np.sum(top * top, axis=1)
