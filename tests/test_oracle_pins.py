"""Pins for the fp64 oracle: checks against things other than the oracle itself.

* hand-worked 2x4-style cases of Eq. 1 under the TP shard layout (tests/golden);
* exhaustive bf16 decoding against torch's bf16 -> fp64 conversion;
* torch.nn.functional.rms_norm in fp64 (a library RMSNorm) at TP = 1;
* correctly rounded sums (math.fsum) for the Phase A partials and their total;
* closed forms and invariants that Eq. 1 fixes: gamma = 1 gives an output RMS
  of sqrt(ms / (ms + eps)); power-of-two scaling with eps = 0 leaves the output
  unchanged bit for bit; concatenating the TP shards gives the unsharded
  output for every TP degree; Q and K are normalised independently;
* FP8-E4M3: hand-worked codes, encodings and a QK-Norm case (tests/golden),
  every one of the 256 codes against torch's float8_e4m3fn, the encoder
  against torch's cast on a dense fp32 sweep holding every halfway case, and
  the FP8 path against torch's RMSNorm on decoded inputs;
* mutation tests: plausible mistakes planted in the oracle must each fail at
  least one of the pins above.
"""
from __future__ import annotations

import contextlib
import json
import math
import os

import numpy as np
import pytest
import torch

import workloads
from oracle import compare
from oracle import qknorm as Q

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_checks.json")
GOLDEN_FP8 = os.path.join(os.path.dirname(__file__), "golden", "fp8_hand_checks.json")


def _golden_cases():
    with open(GOLDEN) as f:
        return json.load(f)["cases"]


def _num(v):
    return float(v)  # also parses "inf" and "nan"


def _as_array(rows):
    return np.array([[_num(v) for v in r] for r in rows], dtype=np.float64)


def _bits(x):
    return workloads.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def _torch_rmsnorm(x_bits, gamma, eps):
    """Library RMSNorm (PyTorch, fp64) on exactly decoded inputs."""
    x = torch.from_numpy(np.ascontiguousarray(x_bits).astype(np.int16)).view(torch.bfloat16).double()
    g = torch.from_numpy(np.asarray(gamma, dtype=np.float64))
    return torch.nn.functional.rms_norm(x, (x.shape[-1],), g, eps).numpy()


# ---------------------------------------------------------------- pin checks
# Each check raises AssertionError on a mismatch. They look the oracle up as
# module attributes so that the mutation tests below can plant mistakes in it.

def check_golden():
    for case in _golden_cases():
        x = np.array(case["x"], dtype=np.float32)
        bits = _bits(x)
        assert np.array_equal(Q.decode_bf16(bits), x.astype(np.float64)), case["name"]
        tp, eps = case["tp"], case["eps"]
        y_full = _as_array(case["y_full"])
        inv = np.array([_num(v) for v in case["inv"]])
        partials = np.array(case["partials"], dtype=np.float64)
        d_full = x.shape[1]
        d_local = d_full // tp
        for r in range(tp):
            out = Q.qknorm_shard(bits, np.array(case["gamma"], dtype=np.float32), tp, r, eps)
            assert np.array_equal(out["partials"], partials), (case["name"], out["partials"])
            compare.check_close(out["inv"], inv, 1e-15, f"{case['name']} inv")
            compare.check_close(out["y"], y_full[:, r * d_local:(r + 1) * d_local], 1e-15,
                                f"{case['name']} y rank {r}")


def check_bf16_decode_exhaustive():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ours = Q.decode_bf16(bits)
    ref = torch.from_numpy(bits.astype(np.int16)).view(torch.bfloat16).double().numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])
    # signed zeros keep their sign
    assert np.array_equal(np.signbit(ours[~nan]), np.signbit(ref[~nan]))


def _fp8_golden():
    with open(GOLDEN_FP8) as f:
        return json.load(f)


def _codes(rows):
    return np.array([[int(v, 16) for v in r] for r in rows], dtype=np.uint8)


def check_fp8_golden():
    g = _fp8_golden()
    for c in g["decode"]:
        v = Q.decode_e4m3(np.array([int(c["code"], 16)], np.uint8))[0]
        want = _num(c["value"])
        if math.isnan(want):
            assert math.isnan(v), c
        else:
            assert v == want and math.copysign(1, v) == math.copysign(1, want), c
    for c in g["encode"]:
        got = int(Q.encode_e4m3(np.array([c["value"]], np.float64))[0])
        assert got == int(c["code"], 16), (c, hex(got))
    for case in g["cases"]:
        x = _codes(case["x_codes"])
        tp, eps = case["tp"], case["eps"]
        d_local = x.shape[1] // tp
        y_full = _as_array(case["y_full"])
        for r in range(tp):
            out = Q.qknorm_shard(x, np.array(case["gamma"], np.float32), tp, r, eps, fmt="fp8")
            assert np.array_equal(out["partials"], np.array(case["partials"], np.float64))
            compare.check_close(out["inv"], np.array(case["inv"]), 1e-15, case["name"])
            ys = y_full[:, r * d_local:(r + 1) * d_local]
            compare.check_close(out["y"], ys, 1e-15, case["name"])
            codes = _codes(case["y_codes"])[:, r * d_local:(r + 1) * d_local]
            assert np.array_equal(Q.encode_e4m3(out["y"]), codes), case["name"]


def _torch_e4m3(codes):
    return torch.from_numpy(np.asarray(codes, np.uint8)).view(torch.float8_e4m3fn).double().numpy()


def check_e4m3_decode_exhaustive():
    codes = np.arange(256, dtype=np.uint8)
    ours, ref = Q.decode_e4m3(codes), _torch_e4m3(codes)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan) and nan.sum() == 2
    assert np.array_equal(ours[~nan], ref[~nan])
    assert np.array_equal(np.signbit(ours[~nan]), np.signbit(ref[~nan]))


def _fp32_sweep():
    """fp32 values: every finite code value, every halfway point between
    neighbours and the fp32 numbers on either side of it, the overflow edge,
    and scaled normal draws."""
    vals = np.unique(_torch_e4m3(np.arange(256, dtype=np.uint8)))
    vals = vals[np.isfinite(vals)]
    mids = ((vals[1:] + vals[:-1]) / 2).astype(np.float32)
    edge = np.array([448, 456, 464, 472, 480, 1e6, np.inf], np.float32)
    mids = np.concatenate([mids, edge, -edge])
    rng = np.random.default_rng(7)
    draws = (rng.standard_normal(50000) * rng.choice([1e-3, 0.1, 1, 30, 400], 50000)).astype(np.float32)
    return np.concatenate([vals.astype(np.float32), mids, np.nextafter(mids, np.float32(np.inf)),
                           np.nextafter(mids, np.float32(-np.inf)), draws,
                           np.array([0.0, -0.0, np.nan], np.float32)])


def check_e4m3_encode_against_torch():
    x = _fp32_sweep()
    ours = Q.encode_e4m3(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    bad = np.nonzero(ours != ref)[0]
    assert bad.size == 0, [(float(x[i]), hex(ours[i]), hex(ref[i])) for i in bad[:5]]
    codes = np.arange(256, dtype=np.uint8)
    finite = ~np.isnan(Q.decode_e4m3(codes))
    assert np.array_equal(Q.encode_e4m3(Q.decode_e4m3(codes[finite])), codes[finite])


def check_fp8_library_rmsnorm():
    for T, d, eps, scale, tp in [(16, 512, 1e-6, 1.0, 2), (5, 96, 1e-3, 20.0, 3),
                                 (3, 64, 0.0, 0.01, 4)]:
        codes = workloads.random_rows(d, T, d, "student_t", scale, dtype="fp8")
        g = workloads.random_gamma(d, d)
        x = torch.from_numpy(_torch_e4m3(codes))
        ref = torch.nn.functional.rms_norm(x, (d,), torch.from_numpy(g.astype(np.float64)), eps).numpy()
        parts = [Q.qknorm_shard(codes, g, tp, r, eps, fmt="fp8")["y"] for r in range(tp)]
        compare.check_close(np.concatenate(parts, axis=1), ref, 1e-12, f"fp8 rms_norm d={d}")


def check_library_rmsnorm(seed=0):
    for T, d, eps, dist in [(16, 512, 1e-6, "normal"), (5, 96, 1e-3, "student_t"),
                            (3, 8, 0.0, "uniform"), (7, 1000, 1e-6, "normal")]:
        bits = workloads.random_rows(seed + d, T, d, dist)
        g = workloads.random_gamma(seed + d, d)
        ref = _torch_rmsnorm(bits, g, eps)
        out = Q.qknorm_shard(bits, g, 1, 0, eps)["y"]
        compare.check_close(out, ref, 1e-12, f"rms_norm T={T} d={d}")


def check_fsum_partials():
    for wl in (workloads.TINY_FULL, workloads.DECODE_TP4.with_tokens(8),
               workloads.DECODE_TP8.with_tokens(8)):
        data = workloads.generate(wl)
        for key, d_full in (("xq", wl.q_full), ("xk", wl.k_full)):
            x = Q.decode_bf16(data[key])
            P = Q.shard_partials(x, wl.tp)
            assert P.shape == (wl.tp, wl.T)
            for t in range(wl.T):
                full = math.fsum(v * v for v in x[t].tolist())
                for k in range(wl.tp):
                    lo, hi = k * (d_full // wl.tp), (k + 1) * (d_full // wl.tp)
                    exact = math.fsum(v * v for v in x[t, lo:hi].tolist())
                    assert abs(P[k, t] - exact) <= 1e-13 * exact, (wl.name, key, k, t)
                assert abs(math.fsum(P[:, t].tolist()) - full) <= 1e-13 * full


def check_concat_equals_unsharded():
    wl = workloads.PREFILL_TP2.with_tokens(6)
    data = workloads.generate(wl)
    for key, gkey in (("xq", "gq"), ("xk", "gk")):
        ref = _torch_rmsnorm(data[key], data[gkey], wl.eps)
        for tp in (1, 2, 4, 8):
            parts = [Q.qknorm_shard(data[key], data[gkey], tp, r, wl.eps)["y"] for r in range(tp)]
            compare.check_close(np.concatenate(parts, axis=1), ref, 1e-12,
                                f"{key} concat tp={tp}")


def check_gamma_one_closed_form():
    for eps in (1e-6, 0.5):
        bits = workloads.random_rows(3, 9, 256, "student_t")
        y = Q.qknorm_shard(bits, np.ones(256, np.float32), 1, 0, eps)["y"]
        x = Q.decode_bf16(bits)
        ms = np.array([math.fsum(v * v for v in row.tolist()) / 256 for row in x])
        rms_y = np.sqrt(np.mean(y * y, axis=1))
        compare.check_close(rms_y, np.sqrt(ms / (ms + eps)), 1e-12, "gamma=1 RMS")


def check_scale_invariance():
    bits = workloads.random_rows(4, 5, 128, "normal")
    g = workloads.random_gamma(4, 128)
    base = Q.qknorm_shard(bits, g, 2, 1, 0.0)["y"]
    x = Q.decode_bf16(bits)
    for k in (-3, 2, 7):
        scaled = _bits(x * 2.0 ** k)
        assert np.array_equal(Q.decode_bf16(scaled), x * 2.0 ** k)
        out = Q.qknorm_shard(scaled, g, 2, 1, 0.0)["y"]
        assert np.array_equal(out, base), k
    # with eps > 0 the factor changes by at most eps / (2 ms) relative
    eps = 1e-2
    ms = np.mean(x * x, axis=1)
    y1 = Q.qknorm_shard(bits, g, 1, 0, eps)["y"]
    y2 = Q.qknorm_shard(_bits(x * 8.0), g, 1, 0, eps)["y"]
    rel = np.abs(y2 - y1) / np.abs(y1).clip(1e-300)
    bound = (eps / (2 * ms))[:, None] + 1e-14
    assert np.all(rel[np.abs(y1) > 0] <= np.broadcast_to(bound, rel.shape)[np.abs(y1) > 0])


def check_layerwise_independent():
    wl = workloads.DECODE_TP4.with_tokens(4)
    data = workloads.generate(wl)
    out = Q.qknorm_layerwise(data["xq"], data["xk"], data["gq"], data["gk"], wl.tp, 2, wl.eps)
    refq = _torch_rmsnorm(data["xq"], data["gq"], wl.eps)[:, workloads.shard_cols(wl.q_full, wl.tp, 2)]
    refk = _torch_rmsnorm(data["xk"], data["gk"], wl.eps)[:, workloads.shard_cols(wl.k_full, wl.tp, 2)]
    compare.check_close(out["q"]["y"], refq, 1e-12, "layerwise q")
    compare.check_close(out["k"]["y"], refk, 1e-12, "layerwise k")


ALL_PINS = [check_golden, check_bf16_decode_exhaustive, check_library_rmsnorm,
            check_fsum_partials, check_concat_equals_unsharded, check_gamma_one_closed_form,
            check_scale_invariance, check_layerwise_independent, check_fp8_golden,
            check_e4m3_decode_exhaustive, check_e4m3_encode_against_torch,
            check_fp8_library_rmsnorm]


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin()


def test_row_blocks_do_not_change_result():
    wl = workloads.DECODE_TP8.with_tokens(37)
    data = workloads.generate(wl)
    a = Q.qknorm_shard(data["xq"], data["gq"], wl.tp, 5, wl.eps, row_block=1024)
    b = Q.qknorm_shard(data["xq"], data["gq"], wl.tp, 5, wl.eps, row_block=5)
    for key in a:
        assert np.array_equal(a[key], b[key])


def test_nan_and_inf_propagate():
    x = np.array([[1.0, np.nan, 2.0, 3.0], [1.0, np.inf, 0.0, 1.0], [1, 2, 3, 4]], np.float32)
    out = Q.qknorm_shard(_bits(x), np.ones(4, np.float32), 2, 0, 1e-6)
    assert np.isnan(out["y"][0]).all()          # NaN in the row poisons its factor
    assert np.isnan(out["partials"][0, 0])       # rank 0's slice holds the NaN
    assert out["partials"][1, 0] == 13.0
    assert out["inv"][1] == 0.0 and out["y"][1, 0] == 0.0  # inf sum -> factor 0
    assert np.isfinite(out["y"][2]).all()


def test_compare_fp8_rule():
    ref = np.array([1.03, 1.0625, 1.0625 * (1 + 1e-7), 0.0, 470.0, 464.0, np.nan, 1.5e-3, -2.6])
    ok = np.array([1.0, 1.0, 1.125, 0.0, np.nan, 448.0, np.nan, 2 ** -9, -2.5])
    assert compare.check_fp8(ok, ref, "ok") <= 1.0 + 1e-3
    for i, bad in [(0, 1.125), (3, 2 ** -9), (4, 448.0), (5, 416.0), (6, 1.0), (7, 0.0), (8, -2.75)]:
        t = ok.copy()
        t[i] = bad
        with pytest.raises(AssertionError):
            compare.check_fp8(t, ref, f"bad {i}")
    assert np.array_equal(compare.e4m3_half_step(np.array([0.0, 2 ** -8, 1.0, 1.99, 300.0])),
                          np.array([2 ** -10, 2 ** -10, 2 ** -4, 2 ** -4, 16.0]))


def test_compare_rules():
    ref = np.array([1.0, 0.0, np.nan, np.inf, -2.0])
    compare.check_close(ref * (1 + 1e-3), ref, 8e-3, "ok")
    with pytest.raises(AssertionError):
        compare.check_close(np.array([1.0, 1e-30, np.nan, np.inf, -2.0]), ref, 8e-3, "zero")
    with pytest.raises(AssertionError):
        compare.check_close(np.array([1.0, 0.0, 1.0, np.inf, -2.0]), ref, 8e-3, "nan")
    with pytest.raises(AssertionError):
        compare.check_close(ref * 1.01, ref, 8e-3, "tol")
    m = compare.paper_error_metrics(np.array([1.0, 2.0]), np.array([1.0, 2.5]))
    assert m["max_abs"] == 0.5 and m["mean_abs"] == 0.25


# ---------------------------------------------------------------- mutation tests

def _mut_eps_outside(S, d_full, eps):
    return 1.0 / (np.sqrt(np.asarray(S, np.float64) / d_full) + eps)


def _mut_divisor_off_by_one(S, d_full, eps):
    return 1.0 / np.sqrt(np.asarray(S, np.float64) / (d_full - 1) + eps)


def _mut_no_reciprocal(S, d_full, eps):
    return np.sqrt(np.asarray(S, np.float64) / d_full + eps)


def _mut_abs_sum(x):
    return np.sum(np.abs(np.asarray(x, np.float64)), axis=-1)


def _mut_drop_last(x):
    x = np.asarray(x, np.float64)[..., :-1]
    return np.sum(x * x, axis=-1)


def _mut_next_rank(d_full, tp, rank):
    d_local = d_full // tp
    r = (rank + 1) % tp
    return slice(r * d_local, (r + 1) * d_local)


def _mut_interleaved(d_full, tp, rank):
    return slice(rank, None, tp)


def _mut_gamma_reversed(x, gamma, eps):
    x = np.asarray(x, np.float64)
    inv = Q.rms_factor(Q.sum_of_squares(x), x.shape[-1], eps)
    return x * inv[:, None] * np.asarray(gamma, np.float64)[::-1][None, :]


def _mut_no_gamma(x, gamma, eps):
    x = np.asarray(x, np.float64)
    return x * Q.rms_factor(Q.sum_of_squares(x), x.shape[-1], eps)[:, None]


def _mut_decode_truncated(bits):
    bits = np.asarray(bits, np.uint16) & np.uint16(0xFFFE)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _mut_local_stat(x_bits, gamma, tp, rank, eps, row_block=1024, fmt="bf16"):
    # the classic TP mistake: normalise the shard with its own statistic
    x = Q.decode(x_bits, fmt)
    cols = Q.shard_slice(x.shape[1], tp, rank)
    P = Q.shard_partials(x, tp)
    xs = x[:, cols]
    inv = Q.rms_factor(Q.sum_of_squares(xs), xs.shape[1], eps)
    return {"partials": P, "inv": inv,
            "y": xs * inv[:, None] * np.asarray(gamma, np.float64)[cols][None, :]}


def _mut_joint_qk(xq_bits, xk_bits, gq, gk, tp, rank, eps, row_block=1024, fmt="bf16"):
    # one factor over Q and K together instead of one per tensor
    xq, xk = Q.decode(xq_bits, fmt), Q.decode(xk_bits, fmt)
    S = Q.sum_of_squares(xq) + Q.sum_of_squares(xk)
    inv = Q.rms_factor(S, xq.shape[1] + xk.shape[1], eps)
    out = {}
    for name, x, g in (("q", xq, gq), ("k", xk, gk)):
        cols = Q.shard_slice(x.shape[1], tp, rank)
        out[name] = {"partials": Q.shard_partials(x, tp), "inv": inv,
                     "y": (x * inv[:, None] * np.asarray(g, np.float64)[None, :])[:, cols]}
    return out


def _mut_partials_reversed(x_full, tp):
    x_full = np.asarray(x_full, np.float64)
    d = x_full.shape[-1]
    return np.stack([Q.sum_of_squares(x_full[:, Q.shard_slice(d, tp, k)])
                     for k in reversed(range(tp))])


def _mut_e4m3_bias8(bits):
    b = np.asarray(bits, np.uint8).astype(np.int64)
    E, M = (b >> 3) & 0xF, b & 7
    mag = np.where(E == 0, M * 2.0 ** -10, (8 + M) * np.exp2(E - 11.0))
    out = np.where(b >> 7, -mag, mag)
    out[(E == 15) & (M == 7)] = np.nan
    return out


def _mut_e4m3_no_subnormals(bits):
    b = np.asarray(bits, np.uint8).astype(np.int64)
    E, M = (b >> 3) & 0xF, b & 7
    mag = (8 + M) * np.exp2(E - 10.0)  # E = 0 read as a normal binade
    out = np.where(b >> 7, -mag, mag)
    out[(E == 15) & (M == 7)] = np.nan
    return out


def _mut_e4m3_inf_code(bits):
    out = Q_ORIG["decode_e4m3"](bits)
    b = np.asarray(bits, np.uint8)
    out[(b & 0x7F) == 0x7F] = np.where(b[(b & 0x7F) == 0x7F] >> 7, -np.inf, np.inf)
    return out


def _mut_encode_ties_away(v):
    v = np.asarray(v, np.float64)
    step = np.exp2(np.maximum(np.frexp(np.where(v != 0, np.abs(v), 1.0))[1] - 1, -6) - 3.0)
    nudged = np.abs(v) + step * 1e-9  # halfway cases now round up in magnitude
    return Q_ORIG["encode_e4m3"](np.copysign(nudged, v))


def _mut_encode_saturates(v):
    return Q_ORIG["encode_e4m3"](np.clip(np.asarray(v, np.float64), -448.0, 448.0))


def _mut_decode_ignores_format(bits, fmt="bf16"):
    return Q_ORIG["decode_bf16"](np.asarray(bits).astype(np.uint16))


Q_ORIG = {name: getattr(Q, name) for name in ("decode_e4m3", "encode_e4m3", "decode_bf16")}

MUTANTS = {
    "eps_outside_sqrt": ("rms_factor", _mut_eps_outside),
    "divisor_off_by_one": ("rms_factor", _mut_divisor_off_by_one),
    "no_reciprocal": ("rms_factor", _mut_no_reciprocal),
    "abs_instead_of_square": ("sum_of_squares", _mut_abs_sum),
    "drops_last_column": ("sum_of_squares", _mut_drop_last),
    "wrong_rank_slice": ("shard_slice", _mut_next_rank),
    "interleaved_shards": ("shard_slice", _mut_interleaved),
    "gamma_reversed": ("rmsnorm", _mut_gamma_reversed),
    "gamma_dropped": ("rmsnorm", _mut_no_gamma),
    "bf16_decode_truncates": ("decode_bf16", _mut_decode_truncated),
    "local_statistic": ("qknorm_shard", _mut_local_stat),
    "joint_qk_factor": ("qknorm_layerwise", _mut_joint_qk),
    "partials_rank_reversed": ("shard_partials", _mut_partials_reversed),
    "e4m3_bias_8": ("decode_e4m3", _mut_e4m3_bias8),
    "e4m3_no_subnormals": ("decode_e4m3", _mut_e4m3_no_subnormals),
    "e4m3_has_infinity": ("decode_e4m3", _mut_e4m3_inf_code),
    "e4m3_ties_away": ("encode_e4m3", _mut_encode_ties_away),
    "e4m3_saturating_encode": ("encode_e4m3", _mut_encode_saturates),
    "fp8_read_as_bf16": ("decode", _mut_decode_ignores_format),
}


@contextlib.contextmanager
def _planted(name, fn):
    orig = getattr(Q, name)
    setattr(Q, name, fn)
    try:
        yield
    finally:
        setattr(Q, name, orig)


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_pins_catch_planted_mistake(mutant):
    name, fn = MUTANTS[mutant]
    caught = []
    with _planted(name, fn):
        for pin in ALL_PINS:
            try:
                pin()
            except Exception as e:  # an error is as good as a mismatch here
                caught.append((pin.__name__, type(e).__name__))
    assert caught, f"no pin caught the planted mistake {mutant!r}"
