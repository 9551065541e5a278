"""Pins for the projection oracle (oracle/projection.py) and its error bounds.

* a hand-worked projection and its Phase A statistic;
* every dot product against math.fsum (correctly rounded) on small inputs;
* round_bf16 against torch's fp32 -> bf16 cast on every halfway point between
  neighbouring bf16 values of several binades, their fp32 neighbours, random
  values and the overflow edge;
* the fp32 error bound: an fp32 evaluation (torch, CPU) of the same products,
  rounded to bf16, stays inside it, and a one-step perturbation does not;
* planted mistakes (transposed weight, truncating rounding, squares of the
  unrounded values, a dropped column) each fail a pin.
"""
from __future__ import annotations

import contextlib
import math

import numpy as np
import pytest
import torch

import workloads
from oracle import compare
from oracle import projection as P
from oracle.qknorm import decode_bf16


def _bits(a):
    return workloads.f32_to_bf16_bits(np.asarray(a, np.float32))


def check_hand_worked():
    # x = [[1, 2], [3, 4]], W = [[1, 0], [1, 1], [0, -1]] (3 outputs of 2 inputs)
    x = _bits([[1, 2], [3, 4]])
    w = _bits([[1, 0], [1, 1], [0, -1]])
    q = P.project(x, w)
    assert np.array_equal(q, np.array([[1, 3, -2], [3, 7, -4]], np.float64))
    assert np.array_equal(P.stored_partials(x, w), np.array([14.0, 74.0]))
    # 257 and 259 are not bf16 values (step 2 in [256, 512)): 257 is halfway
    # between 256 and 258 and goes to the even significand (256), 259 to 260
    assert np.array_equal(P.round_bf16(np.array([257.0, 259.0, -257.0])), [256.0, 260.0, -256.0])
    # stored values are rounded before squaring: q = [1 + 2^-8, 1 + 3 * 2^-8] are both
    # halfway cases of the step 2^-7 and round to even: 1 and 1 + 2^-6
    x = _bits([[1.0, 1.0]])
    w = _bits([[1.0, 2.0 ** -8], [1.0, 3 * 2.0 ** -8]])
    assert np.array_equal(P.project(x, w), [[1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8]])
    assert np.array_equal(P.stored_partials(x, w), [1.0 + (1 + 2.0 ** -6) ** 2])


def check_fsum_dot_products():
    rng = np.random.default_rng(5)
    for T, d, h in ((3, 5, 7), (4, 8, 96), (2, 3, 1000)):
        x = _bits(rng.standard_normal((T, h)))
        w = _bits(rng.standard_normal((d, h)) * 0.1)
        q = P.project(x, w)
        xf, wf = decode_bf16(x), decode_bf16(w)
        for t in range(T):
            for j in range(d):
                exact = math.fsum((xf[t] * wf[j]).tolist())  # products of bf16 are exact in fp64
                scale = math.fsum(np.abs(xf[t] * wf[j]).tolist())
                assert abs(q[t, j] - exact) <= 1e-15 * scale + 1e-300, (T, d, h, t, j)


def check_round_bf16_against_torch():
    vals = []
    for e in (-130, -126, -10, -1, 0, 5, 120, 127):
        base = 2.0 ** e
        m = np.arange(128, 256, dtype=np.float64)  # 8 significant bits
        grid = m / 128.0 * base
        mids = (grid[:-1] + grid[1:]) / 2
        vals += [grid, mids, np.nextafter(mids.astype(np.float32), np.float32(np.inf)),
                 np.nextafter(mids.astype(np.float32), np.float32(-np.inf))]
    rng = np.random.default_rng(9)
    vals.append(rng.standard_normal(20000) * rng.choice([1e-30, 1e-3, 1.0, 1e5, 1e30], 20000))
    vals.append(np.array([3.3895e38, 3.4e38, 0.0, -0.0, 1e-45]))
    x = np.concatenate(vals).astype(np.float32)
    x = x[np.isfinite(x)]
    ours = P.round_bf16(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).double().numpy()
    bad = np.nonzero(~((ours == ref) | (np.isnan(ours) & np.isnan(ref))))[0]
    assert bad.size == 0, [(float(x[i]), ours[i], ref[i]) for i in bad[:5]]


def check_error_bound_holds_for_fp32():
    rng = np.random.default_rng(11)
    T, d, h = 16, 24, 4096
    x = _bits(rng.standard_normal((T, h)))
    w = _bits(rng.standard_normal((d, h)) / np.sqrt(h))
    q = P.project(x, w)
    da = P.dot_abs(x, w)
    # an fp32 evaluation (torch on the CPU, its own summation order), rounded to bf16
    xt = torch.from_numpy(decode_bf16(x).astype(np.float32))
    wt = torch.from_numpy(decode_bf16(w).astype(np.float32))
    q32 = (xt @ wt.T).to(torch.bfloat16).double().numpy()
    assert compare.check_projection(q32, q, da, h, "fp32 evaluation") <= 1.0
    # one bf16 step off is outside the bound (for values away from zero)
    off = q32 + np.sign(q32) * compare.bf16_step(np.abs(q32))
    with pytest.raises(AssertionError):
        compare.check_projection(off, q, da, h, "perturbed")
    # the partial bound holds for the fp32 evaluation's stored values
    P32 = np.sum(q32 * q32, axis=1)
    assert np.all(np.abs(P32 - P.stored_partials(x, w)) <= compare.projection_partial_bound(q, da, h))


PINS = [check_hand_worked, check_fsum_dot_products, check_round_bf16_against_torch,
        check_error_bound_holds_for_fp32]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin()


def _mut_transposed(x_bits, w_bits):
    return decode_bf16(x_bits) @ decode_bf16(w_bits)  # W read as in x out


def _mut_truncating_round(v):
    v = np.asarray(v, np.float64)
    mag = np.abs(v)
    e = np.maximum(np.frexp(np.where(mag > 0, mag, 1.0))[1] - 1, -126)
    step = np.exp2(e - 7.0)
    return np.copysign(np.floor(mag / step) * step, v)


def _mut_unrounded_squares(x_bits, w_bits):
    q = P.project(x_bits, w_bits)
    return np.sum(q * q, axis=1)


def _mut_drop_column(x_bits, w_bits):
    q = P.round_bf16(P.project(x_bits, w_bits))[:, :-1]
    return np.sum(q * q, axis=1)


MUTANTS = {
    "transposed_weight": ("project", _mut_transposed),
    "truncating_round": ("round_bf16", _mut_truncating_round),
    "partials_of_unrounded": ("stored_partials", _mut_unrounded_squares),
    "partials_drop_column": ("stored_partials", _mut_drop_column),
}


@contextlib.contextmanager
def _planted(name, fn):
    orig = getattr(P, name)
    setattr(P, name, fn)
    try:
        yield
    finally:
        setattr(P, name, orig)


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_pins_catch_planted_mistake(mutant):
    name, fn = MUTANTS[mutant]
    caught = []
    with _planted(name, fn):
        for pin in PINS:
            try:
                pin()
            except Exception as e:  # an error is as good as a mismatch here
                caught.append((pin.__name__, type(e).__name__))
    assert caught, f"no pin caught the planted mistake {mutant!r}"


def test_projection_inputs_are_deterministic():
    wl = workloads.DECODE_TP4
    a, b = workloads.projection_inputs(wl), workloads.projection_inputs(wl)
    for k in a:
        assert np.array_equal(a[k], b[k])
    assert a["x"].shape == (wl.T, wl.q_full) and a["wq"].shape == (wl.q_full, wl.q_full)
    assert a["wk"].shape == (wl.k_full, wl.q_full)
    q = P.project(a["x"][:4], a["wq"][:64])
    assert 0.5 < float(np.std(q)) < 2.0  # unit-variance projections
