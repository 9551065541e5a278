"""Seeded synthetic workloads for sharded layerwise QK-Norm.

This module only draws inputs: projected Q and K activations (as bf16 or
FP8-E4M3 bit patterns), the fp32 gamma vectors, and the shard layout. It holds none of the
normalisation arithmetic, so both the fp64 oracle and the HIP path can take
their inputs from here without sharing any of the method's code.

Shapes follow the tensor-parallel layout of the paper (Sec. II-B, Fig. 1(b)):
the column-parallel Q/K projection leaves rank r with a contiguous slice of
the hidden dimension of Q and of K. The paper's own workloads (OLMoE, OLMo 2,
OLMo 3 serving ShareGPT prompts, Sec. IV-A) need weights and a dataset that
are not available; the named workloads below stand in for them with GQA-style
Q/K widths and decode/prefill token counts.

Recipe (shared by every workload):
  * one ``numpy.random.Generator`` per stream, seeded with
    ``SeedSequence([seed, stream_id])``; stream ids: 0 = X_Q, 1 = X_K,
    2 = per-token scales, 3 = outlier channels, 4 = gamma_Q, 5 = gamma_K;
    the activations X_Q and X_K are drawn in blocks of 1024 tokens, block b
    from ``SeedSequence([seed, stream_id, b])``, so blocks can be drawn in
    parallel and the bits do not depend on the number of threads;
  * activations are drawn in fp32, shaped by the workload's distribution,
    then rounded to the workload's format with round-to-nearest-even: bf16,
    or FP8-E4M3 (OCP e4m3fn) after clamping to its finite range [-448, 448]
    (a saturating quantiser, as FP8 activations are produced in practice);
    everyone consumes the same bits;
  * lognormal(mu, sigma) = exp(N(mu, sigma)), one draw per token per tensor,
    multiplying that token's whole (unsharded) row;
  * outlier channels: n = max(1, round(0.001 * d_full)) channels per tensor,
    picked without replacement, fixed across tokens, scaled x50 before the
    bf16 rounding;
  * Student-t uses ``Generator.standard_t(df)``;
  * gamma ~ U[0.5, 1.5), stored as fp32.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace
from typing import Dict, Tuple

import numpy as np

BLOCK_TOKENS = 1024

STREAM_XQ, STREAM_XK, STREAM_SCALE, STREAM_OUTLIER, STREAM_GQ, STREAM_GK = range(6)
STREAM_PROJ_X, STREAM_PROJ_WQ, STREAM_PROJ_WK = 6, 7, 8


@dataclass(frozen=True)
class Workload:
    """One QK-Norm workload: T tokens, full Q/K widths, TP degree, distribution."""

    name: str
    T: int
    q_full: int
    k_full: int
    tp: int
    dist: str  # "normal" | "normal_lognormal" | "normal_outliers" | "student_t"
    seed: int
    sigma: float = 0.0  # lognormal sigma for "normal_lognormal"
    df: float = 3.0  # degrees of freedom for "student_t"
    eps: float = 1e-6
    dtype: str = "bf16"  # activation format: "bf16" | "fp8" (FP8-E4M3)

    @property
    def q_local(self) -> int:
        return self.q_full // self.tp

    @property
    def k_local(self) -> int:
        return self.k_full // self.tp

    def with_tp(self, tp: int) -> "Workload":
        """Same tokens and data, another TP degree (the data do not depend on tp)."""
        if self.q_full % tp or self.k_full % tp:
            raise ValueError(f"tp={tp} does not divide {self.q_full}/{self.k_full}")
        return replace(self, tp=tp, name=f"{self.name}@tp{tp}")

    def with_tokens(self, T: int) -> "Workload":
        return replace(self, T=T, name=f"{self.name}@T{T}")

    def with_dtype(self, dtype: str) -> "Workload":
        """Same draws, quantised to another activation format."""
        if dtype not in ("bf16", "fp8"):
            raise ValueError(dtype)
        return replace(self, dtype=dtype, name=f"{self.name}@{dtype}")


# The five workloads. Seeds: the tiny case uses seed 0; the others 1..4.
TINY_FULL = Workload("tiny_full_T16_q512_k128_tp1", 16, 512, 128, 1, "normal", 0)
DECODE_TP4 = Workload("decode_T64_q4096_k1024_tp4", 64, 4096, 1024, 4,
                      "normal_lognormal", 1, sigma=1.0)
DECODE_TP8 = Workload("decode_T256_q5120_k1024_tp8", 256, 5120, 1024, 8,
                      "normal_outliers", 2)
PREFILL_TP2 = Workload("prefill_T8192_q4096_k1024_tp2", 8192, 4096, 1024, 2,
                       "normal_lognormal", 3, sigma=0.5)
LONG_PREFILL_TP4 = Workload("long_prefill_T32768_q8192_k1024_tp4", 32768, 8192, 1024, 4,
                            "student_t", 4, df=3.0)

WORKLOADS: Dict[str, Workload] = {w.name: w for w in
                                  (TINY_FULL, DECODE_TP4, DECODE_TP8, PREFILL_TP2, LONG_PREFILL_TP4)}


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even); return uint16 bits.

    Input conversion only (the data format), not part of the normalisation.
    NaN inputs map to a quiet NaN of the same sign.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        rounded[nan] = ((u[nan] >> 16).astype(np.uint16) & 0x8000) | 0x7FC0
    return rounded


E4M3_MAX = 448.0


def f32_to_e4m3_bits(a: np.ndarray) -> np.ndarray:
    """Quantise fp32 values to FP8-E4M3 (OCP e4m3fn) bits, saturating.

    Input conversion only (the data format), not part of the normalisation.
    Values are clamped to [-448, 448], then rounded to the nearest code (ties
    to the even code); magnitudes below 2^-6 use the subnormal grid 2^-9.
    NaN maps to 0x7f (0xff if negative).
    """
    a = np.asarray(a, dtype=np.float32).astype(np.float64)
    nan = np.isnan(a)
    neg = np.signbit(a)
    m = np.minimum(np.abs(np.where(nan, 0.0, a)), E4M3_MAX)
    # binade exponent of m (m = f * 2^k, 0.5 <= f < 1), at least -6
    k = np.frexp(np.where(m > 0, m, 1.0))[1] - 1
    k = np.where(m > 0, np.maximum(k, -6), -6)
    units = np.round(m * np.exp2(3.0 - k))  # multiples of the grid step 2^(k-3); half to even
    # units is in [0, 16]; 16 means the next binade's 1.000
    normal = (k > -6) | (units >= 8)
    exp_field = np.where(normal, k + 7 + (units >= 16), 0)
    mant = np.where(units >= 16, 0, np.where(normal, units - 8, units))
    bits = (exp_field.astype(np.int64) << 3) | mant.astype(np.int64)
    bits = bits | (neg.astype(np.int64) << 7)
    bits = np.where(nan, np.where(neg, 0xFF, 0x7F), bits)
    return bits.astype(np.uint8)


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, stream]))


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _activations(wl: Workload, d_full: int, stream: int, scale_col: int) -> np.ndarray:
    """Activation bits [T, d_full] of one tensor, drawn block by block."""
    if wl.dist not in ("normal", "student_t", "normal_lognormal", "normal_outliers"):
        raise ValueError(f"unknown distribution {wl.dist!r}")
    T = wl.T
    scale = None
    if wl.dist == "normal_lognormal":
        # one scale per token per tensor; column 0 = Q, column 1 = K
        s = np.exp(_rng(wl.seed, STREAM_SCALE).normal(0.0, wl.sigma, size=(T, 2)))
        scale = s[:, scale_col:scale_col + 1].astype(np.float32)
    idx = outlier_channels(wl)[scale_col] if wl.dist == "normal_outliers" else None
    fp8 = wl.dtype == "fp8"
    if wl.dtype not in ("bf16", "fp8"):
        raise ValueError(f"unknown activation format {wl.dtype!r}")
    out = np.empty((T, d_full), dtype=np.uint8 if fp8 else np.uint16)

    def block(b: int) -> None:
        t0, t1 = b * BLOCK_TOKENS, min(T, (b + 1) * BLOCK_TOKENS)
        rng = np.random.default_rng(np.random.SeedSequence([wl.seed, stream, b]))
        if wl.dist == "student_t":
            x = rng.standard_t(wl.df, size=(t1 - t0, d_full)).astype(np.float32)
        else:
            x = rng.standard_normal(size=(t1 - t0, d_full), dtype=np.float32)
        if scale is not None:
            x *= scale[t0:t1]
        if idx is not None:
            x[:, idx] *= np.float32(50.0)
        out[t0:t1] = f32_to_e4m3_bits(x) if fp8 else f32_to_bf16_bits(x)

    nblocks = (T + BLOCK_TOKENS - 1) // BLOCK_TOKENS
    if nblocks <= 1:
        for b in range(nblocks):
            block(b)
    else:
        with ThreadPoolExecutor(min(_threads(), nblocks)) as ex:
            list(ex.map(block, range(nblocks)))
    return out


def outlier_channels(wl: Workload) -> Tuple[np.ndarray, np.ndarray]:
    """The outlier channel indices of a "normal_outliers" workload (Q, K).

    Q's channels are drawn first, then K's, from one stream.
    """
    orng = _rng(wl.seed, STREAM_OUTLIER)
    nq = max(1, round(0.001 * wl.q_full))
    nk = max(1, round(0.001 * wl.k_full))
    return (orng.choice(wl.q_full, size=nq, replace=False),
            orng.choice(wl.k_full, size=nk, replace=False))


def generate(wl: Workload) -> Dict[str, np.ndarray]:
    """Full (unsharded) inputs of a workload.

    Returns ``xq`` [T, q_full], ``xk`` [T, k_full] (bf16 bits as uint16, or
    FP8-E4M3 bits as uint8 when ``wl.dtype == "fp8"``), ``gq`` float32
    [q_full], ``gk`` float32 [k_full].
    """
    xq = _activations(wl, wl.q_full, STREAM_XQ, 0)
    xk = _activations(wl, wl.k_full, STREAM_XK, 1)
    gq = _rng(wl.seed, STREAM_GQ).uniform(0.5, 1.5, size=wl.q_full).astype(np.float32)
    gk = _rng(wl.seed, STREAM_GK).uniform(0.5, 1.5, size=wl.k_full).astype(np.float32)
    return {"xq": xq, "xk": xk, "gq": gq, "gk": gk}


def shard_cols(d_full: int, tp: int, rank: int) -> slice:
    """Columns held by `rank`: a contiguous slice, as column-parallel projections leave them."""
    if d_full % tp:
        raise ValueError(f"tp={tp} does not divide d_full={d_full}")
    d_local = d_full // tp
    return slice(rank * d_local, (rank + 1) * d_local)


def random_rows(seed: int, T: int, d: int, dist: str = "normal", scale: float = 1.0,
                dtype: str = "bf16") -> np.ndarray:
    """Small ad-hoc inputs for edge-case tests ([T, d] bits: uint16 bf16 or uint8 FP8)."""
    rng = _rng(seed, 100)
    if dist == "normal":
        x = rng.standard_normal(size=(T, d), dtype=np.float32)
    elif dist == "student_t":
        x = rng.standard_t(3.0, size=(T, d)).astype(np.float32)
    elif dist == "uniform":
        x = rng.uniform(-1.0, 1.0, size=(T, d)).astype(np.float32)
    else:
        raise ValueError(dist)
    x = x * np.float32(scale)
    return f32_to_e4m3_bits(x) if dtype == "fp8" else f32_to_bf16_bits(x)


def random_gamma(seed: int, d: int) -> np.ndarray:
    return _rng(seed, 101).uniform(0.5, 1.5, size=d).astype(np.float32)


# ------------------------------------------------------------------ projection inputs
#
# Inputs of the column-parallel Q/K projection that produces the activations
# (Sec. II-B): the layer input x [T, hidden] and the full projection weights
# W_Q [q_full, hidden], W_K [k_full, hidden] (a linear layer's out x in
# layout; rank r's slice is rows shard_cols(...) of each). Recipe: x ~ N(0, 1)
# drawn in 1024-token blocks from SeedSequence([seed, 6, block]); W_Q and W_K ~
# N(0, 1/hidden) from streams 7 and 8 (so each projected value has unit
# variance); all rounded to bf16 (RNE). The model width `hidden` is the Q
# width of the workload unless given.

def projection_inputs(wl: Workload, hidden: int = 0) -> Dict[str, np.ndarray]:
    """``x`` uint16 [T, hidden], ``wq`` uint16 [q_full, hidden], ``wk`` uint16
    [k_full, hidden] (bf16 bits)."""
    hidden = hidden or wl.q_full
    T = wl.T
    x = np.empty((T, hidden), dtype=np.uint16)

    def block(b: int) -> None:
        t0, t1 = b * BLOCK_TOKENS, min(T, (b + 1) * BLOCK_TOKENS)
        rng = np.random.default_rng(np.random.SeedSequence([wl.seed, STREAM_PROJ_X, b]))
        x[t0:t1] = f32_to_bf16_bits(rng.standard_normal(size=(t1 - t0, hidden), dtype=np.float32))

    nblocks = (T + BLOCK_TOKENS - 1) // BLOCK_TOKENS
    if nblocks <= 1:
        for b in range(nblocks):
            block(b)
    else:
        with ThreadPoolExecutor(min(_threads(), nblocks)) as ex:
            list(ex.map(block, range(nblocks)))
    scale = np.float32(1.0 / np.sqrt(hidden))
    wq = _rng(wl.seed, STREAM_PROJ_WQ).standard_normal(size=(wl.q_full, hidden), dtype=np.float32)
    wk = _rng(wl.seed, STREAM_PROJ_WK).standard_normal(size=(wl.k_full, hidden), dtype=np.float32)
    return {"x": x, "wq": f32_to_bf16_bits(wq * scale), "wk": f32_to_bf16_bits(wk * scale)}
