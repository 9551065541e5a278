"""The seeded input generator: rounding, determinism and the distributions' shape."""
import numpy as np
import torch

import workloads


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(7)
    a = np.concatenate([
        rng.standard_normal(200000).astype(np.float32) * np.float32(10.0) ** rng.integers(-30, 30, 200000).astype(np.float32),
        np.array([0.0, -0.0, np.inf, -np.inf, 3.4e38, -3.4e38, 1e-40, 1.00390625, 1.01171875], np.float32),
    ]).astype(np.float32)
    ours = workloads.f32_to_bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    assert np.array_equal(ours, ref)
    nan = workloads.f32_to_bf16_bits(np.array([np.nan, -np.nan], np.float32))
    assert (nan & 0x7FC0 == 0x7FC0).all()


def test_generate_is_deterministic_and_shaped():
    wl = workloads.DECODE_TP4
    a, b = workloads.generate(wl), workloads.generate(wl)
    for k in a:
        assert np.array_equal(a[k], b[k])
    assert a["xq"].shape == (64, 4096) and a["xq"].dtype == np.uint16
    assert a["xk"].shape == (64, 1024)
    assert a["gq"].dtype == np.float32 and a["gq"].min() >= 0.5 and a["gq"].max() < 1.5
    assert wl.q_local == 1024 and wl.k_local == 256


def _f(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def test_distributions():
    # per-token lognormal(0, 1): row RMS spreads over orders of magnitude
    d = workloads.generate(workloads.DECODE_TP4)
    rms = np.sqrt(np.mean(_f(d["xq"]) ** 2, axis=1))
    assert rms.max() / rms.min() > 20
    # outlier channels carry ~50x the typical magnitude
    wl = workloads.DECODE_TP8
    d = workloads.generate(wl)
    qi, ki = workloads.outlier_channels(wl)
    assert len(qi) == 5 and len(ki) == 1
    x = np.abs(_f(d["xq"]))
    assert x[:, qi].mean() > 30 * np.delete(x, qi, axis=1).mean()
    # Student-t(3): heavy tails (kurtosis far above a Gaussian's 3)
    small = workloads.LONG_PREFILL_TP4.with_tokens(64)
    d = workloads.generate(small)
    v = _f(d["xk"]).ravel()
    assert np.mean(v ** 4) / np.mean(v ** 2) ** 2 > 6


def test_shard_cols_and_with_tp():
    assert workloads.shard_cols(4096, 4, 3) == slice(3072, 4096)
    wl = workloads.PREFILL_TP2.with_tp(1)
    assert wl.q_local == 4096 and wl.tp == 1


def test_fp8_quantiser_matches_torch_after_clamp():
    """The saturating FP8-E4M3 quantiser equals torch's e4m3fn cast of the
    value clamped to [-448, 448], on every halfway point and its neighbours."""
    vals = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).float().numpy()
    vals = np.unique(vals[np.isfinite(vals)])
    mids = ((vals[1:] + vals[:-1]) / 2).astype(np.float32)
    rng = np.random.default_rng(3)
    x = np.concatenate([vals, mids, np.nextafter(mids, np.float32(1e9)),
                        np.nextafter(mids, np.float32(-1e9)),
                        (rng.standard_normal(20000) * rng.choice([1e-3, 1, 100, 1e4], 20000)),
                        [0.0, -0.0, 449.0, 464.0, 1e30, -1e30, np.inf, -np.inf]]).astype(np.float32)
    ours = workloads.f32_to_e4m3_bits(x)
    ref = torch.from_numpy(np.clip(x, -448, 448)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(ours, ref)
    assert workloads.f32_to_e4m3_bits(np.array([np.nan, -np.nan], np.float32)).tolist() == [0x7F, 0xFF]


def test_fp8_workload_is_deterministic_and_saturated():
    wl = workloads.LONG_PREFILL_TP4.with_tokens(1100).with_dtype("fp8")
    a, b = workloads.generate(wl), workloads.generate(wl)
    assert a["xq"].dtype == np.uint8 and a["xq"].shape == (1100, wl.q_full)
    assert np.array_equal(a["xq"], b["xq"]) and np.array_equal(a["xk"], b["xk"])
    # the same draws as the bf16 workload, quantised once more
    bf = workloads.generate(workloads.LONG_PREFILL_TP4.with_tokens(1100))
    f32 = (bf["xq"].astype(np.uint32) << 16).view(np.float32)
    near = np.abs(f32) < 400  # away from the clamp, FP8(x) is within one FP8 step of bf16(x)
    v = torch.from_numpy(a["xq"]).view(torch.float8_e4m3fn).float().numpy()
    assert np.all(np.abs(v[near] - f32[near]) <= np.maximum(np.abs(f32[near]) / 8, 2.0 ** -9))
    assert not np.isnan(v).any() and np.abs(v).max() <= 448  # heavy tails saturate, never NaN
    assert np.array_equal(a["gq"], bf["gq"])
