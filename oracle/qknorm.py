"""fp64 CPU oracle for sharded layerwise QK-Norm (SwiftQK, arXiv 2608.09160).

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this module; the product path never does. It shares
no code with the HIP library: its inputs come from ``workloads`` (seeded data,
no normalisation arithmetic) and everything below is written from the paper.

What it computes, and from which passage:

* Eq. 1 (Sec. II-A), RMSNorm of a full projected vector x of width H:
  y = x / sqrt(mean_j x_j^2 + eps) * gamma.
* Layerwise QK-Norm (Sec. II-A): one factor per token over the whole projected
  Q, and a separate one over the whole projected K (not one per head).
* Tensor-parallel layout (Sec. II-B, Fig. 1(b)): the column-parallel projection
  leaves rank r with a contiguous slice of the hidden dimension.
* Phase A (Sec. III-A, Alg. 1): rank r's statistic is the sum of squares of its
  slice. Adding the statistics of all ranks gives the full sum of squares, so
  the result equals Eq. 1 on the unsharded vector (the method keeps the global
  normalisation semantics, Sec. III-A and Sec. V). The oracle therefore computes
  the output as the plain definition -- Eq. 1 on the full row -- and slices it;
  the per-rank partial sums are computed separately, as defined.
* Phases B and C (Sec. III-B/C, Alg. 1): the global factor is
  1 / sqrt(S_global / H_total + eps), and the output is x * gamma * factor.

Everything is fp64. bf16 and FP8-E4M3 inputs (the two activation formats of
Sec. IV-C) are decoded exactly; fp32 gamma is widened exactly. IEEE semantics
are kept on purpose: NaN propagates, and with eps = 0 an all-zero row gives
0 * inf = NaN. The output is the exact (fp64) value; rounding it to the
activation format is left to the comparison (``encode_e4m3`` gives the
round-to-nearest-even FP8 code of a value when a test needs exact bits).

Parity status: every function here is pinned by the tests in
``tests/test_oracle_pins.py`` (hand-worked 2x4 cases, a library RMSNorm, a
correctly rounded sum, closed forms and invariants; the FP8 decoder against
every code of torch's float8_e4m3fn and the format's closed forms, the encoder
against torch's cast on a dense sweep with every halfway case). The paper's own kernel
outputs are not printed anywhere, so no pin uses them.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

# Rows per block when a workload is processed in pieces to bound host memory.
ROW_BLOCK = 1024


def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """Exact bf16 -> fp64: a bf16 value is the top half of an IEEE fp32 word."""
    bits = np.asarray(bits, dtype=np.uint16)
    with np.errstate(invalid="ignore"):  # signalling-NaN patterns widen to NaN
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def decode_e4m3(bits: np.ndarray) -> np.ndarray:
    """Exact FP8-E4M3 (OCP e4m3fn) -> fp64, from the format's definition.

    Bit 7 is the sign, bits 6..3 the exponent field E (bias 7), bits 2..0 the
    mantissa field M. E = 0: subnormal, M * 2^-9. Otherwise (1 + M/8) * 2^(E-7),
    except that E = 15 with M = 7 is NaN. There are no infinities; the largest
    finite magnitude is 1.75 * 2^8 = 448.
    """
    b = np.asarray(bits, dtype=np.uint8).astype(np.int64)
    sign = np.where(b >> 7, -1.0, 1.0)
    E = (b >> 3) & 0xF
    M = b & 0x7
    mag = np.where(E == 0, M * 2.0 ** -9, (8 + M) * np.exp2(E - 10.0))
    out = sign * mag
    out[(E == 15) & (M == 7)] = np.nan
    return out


def encode_e4m3(v: np.ndarray) -> np.ndarray:
    """fp64 -> FP8-E4M3 code, rounding to nearest with ties to even.

    A magnitude that rounds above 448 has no code (the format has no infinity)
    and becomes NaN (0x7f with the value's sign), as does a NaN. Zeros keep
    their sign. Steps: the grid spacing at |v| is 2^(e-3) for 2^e <= |v| (e >=
    -6) and 2^-9 below 2^-6; |v| is rounded to that grid (halfway cases to the
    even multiple), then the code is read off the rounded magnitude.
    """
    v = np.asarray(v, dtype=np.float64)
    out = np.empty(v.shape, dtype=np.uint8)
    sign = np.signbit(v).astype(np.uint8) << 7
    mag = np.abs(v)
    nan = np.isnan(v)
    with np.errstate(invalid="ignore", over="ignore"):
        _, e2 = np.frexp(np.where(nan | np.isinf(mag), 1.0, mag))  # mag = f * 2^e2, f in [0.5, 1)
        e = np.maximum(e2 - 1, -6)  # binade exponent, floored at the subnormal range
        step = np.exp2(e - 3.0)
        q = np.round(mag / step) * step  # numpy rounds halfway cases to even
    q = np.where(np.isinf(mag), np.inf, q)
    over = nan | (q > 448.0)
    qs = np.where(over, 1.0, q)
    _, qe2 = np.frexp(np.where(qs == 0, 1.0, qs))
    qe = qe2 - 1
    sub = qs < 2.0 ** -6
    code = np.where(sub, np.round(qs / 2.0 ** -9),
                    ((qe + 7) << 3) + np.round(qs / np.exp2(qe - 3.0)) - 8)
    out[...] = code.astype(np.uint8) | sign
    out[over] = 0x7F | sign[over]
    return out


def decode(bits: np.ndarray, fmt: str = "bf16") -> np.ndarray:
    """Exact decoding of activation bits in format `fmt` ("bf16" or "fp8")."""
    if fmt == "bf16":
        return decode_bf16(bits)
    if fmt == "fp8":
        return decode_e4m3(bits)
    raise ValueError(f"unknown activation format {fmt!r}")


def shard_slice(d_full: int, tp: int, rank: int) -> slice:
    """Hidden columns owned by `rank` under column-parallel TP (Sec. II-B).

    Rank r owns the contiguous range [r * d_full/tp, (r+1) * d_full/tp).
    """
    if tp < 1 or not 0 <= rank < tp or d_full % tp:
        raise ValueError(f"bad shard: d_full={d_full} tp={tp} rank={rank}")
    d_local = d_full // tp
    return slice(rank * d_local, (rank + 1) * d_local)


def sum_of_squares(x: np.ndarray) -> np.ndarray:
    """Per-row sum of x_j^2 in fp64 (the quantity under the root of Eq. 1)."""
    x = np.asarray(x, dtype=np.float64)
    return np.sum(x * x, axis=-1)


def shard_partials(x_full: np.ndarray, tp: int) -> np.ndarray:
    """Phase A for every rank: P[k, t] = sum of squares of rank k's slice of row t.

    (Sec. III-A; Alg. 1, Phase A.) Returns fp64 [tp, T].
    """
    x_full = np.asarray(x_full, dtype=np.float64)
    d_full = x_full.shape[-1]
    return np.stack([sum_of_squares(x_full[:, shard_slice(d_full, tp, k)])
                     for k in range(tp)])


def rms_factor(sum_sq: np.ndarray, d_full: int, eps: float) -> np.ndarray:
    """Phase B factor: 1 / sqrt(S / H_total + eps) (Eq. 1 denominator; Alg. 1 Phase B).

    H_total is the full (unsharded) width of the vector.
    """
    mean_sq = np.asarray(sum_sq, dtype=np.float64) / float(d_full)
    with np.errstate(divide="ignore", invalid="ignore"):
        return 1.0 / np.sqrt(mean_sq + float(eps))


def rmsnorm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """Eq. 1 on full rows: x / sqrt(mean(x^2) + eps) * gamma, in fp64."""
    x = np.asarray(x, dtype=np.float64)
    gamma = np.asarray(gamma, dtype=np.float64)
    inv = rms_factor(sum_of_squares(x), x.shape[-1], eps)
    with np.errstate(invalid="ignore", over="ignore"):
        return x * inv[:, None] * gamma[None, :]


def qknorm_shard(x_bits: np.ndarray, gamma: np.ndarray, tp: int, rank: int,
                 eps: float, row_block: int = ROW_BLOCK, fmt: str = "bf16") -> Dict[str, np.ndarray]:
    """Rank `rank`'s share of layerwise QK-Norm for one tensor (Q or K).

    x_bits: full unsharded activations as bits of format `fmt` (bf16 uint16 or
            FP8-E4M3 uint8), [T, d_full].
    gamma:  full gamma, [d_full] (fp32 or fp64).
    Returns fp64 arrays:
      ``partials`` [tp, T]   Phase A statistic of every rank,
      ``inv``      [T]       the global factor 1/sqrt(S/d_full + eps),
      ``y``        [T, d_local] rank `rank`'s slice of Eq. 1 on the full row.
    Rows are processed in blocks of `row_block` to bound memory; blocks are
    independent because every token is normalised on its own.
    """
    x_bits = np.asarray(x_bits)
    T, d_full = x_bits.shape
    cols = shard_slice(d_full, tp, rank)
    g = np.asarray(gamma, dtype=np.float64)
    partials = np.empty((tp, T), dtype=np.float64)
    inv = np.empty(T, dtype=np.float64)
    y = np.empty((T, cols.stop - cols.start), dtype=np.float64)
    for t0 in range(0, T, row_block):
        t1 = min(T, t0 + row_block)
        x = decode(x_bits[t0:t1], fmt)
        partials[:, t0:t1] = shard_partials(x, tp)
        inv[t0:t1] = rms_factor(sum_of_squares(x), d_full, eps)
        y[t0:t1] = rmsnorm(x, g, eps)[:, cols]
    return {"partials": partials, "inv": inv, "y": y}


def qknorm_layerwise(xq_bits: np.ndarray, xk_bits: np.ndarray, gq: np.ndarray,
                     gk: np.ndarray, tp: int, rank: int, eps: float,
                     row_block: int = ROW_BLOCK,
                     fmt: str = "bf16") -> Dict[str, Dict[str, np.ndarray]]:
    """Layerwise QK-Norm: Q and K are normalised separately, each over its full width.

    (Sec. II-A: one factor over the whole projected Q, another over the whole
    projected K.) Returns {"q": qknorm_shard(...), "k": qknorm_shard(...)}.
    """
    return {"q": qknorm_shard(xq_bits, gq, tp, rank, eps, row_block, fmt=fmt),
            "k": qknorm_shard(xk_bits, gk, tp, rank, eps, row_block, fmt=fmt)}
