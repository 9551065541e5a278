"""fp64 CPU oracle for the Q/K projection that feeds layerwise QK-Norm.

TEST INFRASTRUCTURE ONLY, like ``oracle.qknorm``: imported by the tests, the
smoke check and the benchmark's CPU-baseline leg, never by the product path.
It shares no code with the HIP library.

What it computes, and from which passage:

* Column-parallel projection (Sec. II-B, Fig. 1(b)): the first linear
  projection of attention is split along its output dimension, so rank r
  holds rows [r*d_local, (r+1)*d_local) of the weight W (out x in, the layout
  of a linear layer) and computes its slice of the projected activations,
  q[t, j] = sum_k x[t, k] * W[j, k], from the full input x.
* The projected activations are stored in the activation format (bf16): the
  stored value is q rounded once to bf16, to nearest even (``round_bf16``).
* Phase A (Sec. III-A, Alg. 1) on that slice: the rank's statistic of token t
  is the sum of squares of its stored projected values,
  P[t] = sum_j round_bf16(q[t, j])^2 (``stored_partials``).

Everything is fp64: bf16 inputs decode exactly, each product x*W of two bf16
values is exact, and the fp64 sum of up to 16384 such terms is within
16384 * 2^-53 of the exact dot product relative to sum |x*W| -- far below any
tolerance used against fp32 hardware.

Parity status: pinned in ``tests/test_oracle_projection.py`` (a hand-worked
case, correctly rounded dot products by ``math.fsum``, torch's fp32 -> bf16
cast for ``round_bf16``, planted mistakes).
"""
from __future__ import annotations

import numpy as np

from oracle.qknorm import decode_bf16


def project(x_bits: np.ndarray, w_bits: np.ndarray) -> np.ndarray:
    """q = x @ W^T in fp64 for bf16 x [T, hidden] and W [d_local, hidden]."""
    x = decode_bf16(x_bits)
    w = decode_bf16(w_bits)
    if x.shape[1] != w.shape[1]:
        raise ValueError(f"hidden sizes differ: {x.shape} vs {w.shape}")
    return x @ w.T


def round_bf16(v: np.ndarray) -> np.ndarray:
    """fp64 values rounded to the nearest bf16 value, ties to even (as fp64).

    bf16 has fp32's exponent range and 8 significant bits: in the binade
    [2^e, 2^(e+1)), e >= -126, the grid step is 2^(e-7); below 2^-126 the
    subnormal step is 2^-133. Magnitudes that round past the largest finite
    bf16, (2 - 2^-7) * 2^127, become infinite. NaN stays NaN.
    """
    v = np.asarray(v, dtype=np.float64)
    mag = np.abs(v)
    fin = np.isfinite(mag)
    with np.errstate(invalid="ignore", over="ignore"):
        e = np.frexp(np.where(fin & (mag > 0), mag, 1.0))[1] - 1
        e = np.maximum(e, -126)
        step = np.exp2(e - 7.0)
        q = np.round(mag / step) * step  # halfway cases to the even multiple
    q = np.where(fin, q, mag)
    q = np.where(q > (2.0 - 2.0 ** -7) * 2.0 ** 127, np.inf, q)
    return np.copysign(q, v)


def stored_partials(x_bits: np.ndarray, w_bits: np.ndarray) -> np.ndarray:
    """Phase A on the rank's stored projected slice: sum_j round_bf16(q[t, j])^2."""
    q = round_bf16(project(x_bits, w_bits))
    return np.sum(q * q, axis=1)


def dot_abs(x_bits: np.ndarray, w_bits: np.ndarray) -> np.ndarray:
    """sum_k |x[t, k] * W[j, k]| in fp64: the scale of the rounding error of
    any fp32 evaluation of q[t, j] (used for error bounds)."""
    return np.abs(decode_bf16(x_bits)) @ np.abs(decode_bf16(w_bits)).T
