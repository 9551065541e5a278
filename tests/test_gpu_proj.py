"""GPU parity: the Q/K projection with Phase A in its epilogue (qkn_proj_partial).

Against the fp64 projection oracle (oracle/projection.py) with the bounds of
oracle/compare.py: every stored value within half a bf16 step (at |q| + eps)
plus eps of the exact dot product, eps = (hidden - 1) 2^-24 sum|x w| (fp32
accumulation of exact bf16 products, any order); the statistic within the
bound those errors imply for sum round_bf16(q)^2. Properties on the kernel's
own outputs: the statistic equals the sum of squares of the stored row within
fp32 summation error (1e-5 relative), results are deterministic, and Q and K
in one launch equal Q and K in two. End to end: the projection's statistics
of every rank, combined by qkn_apply, normalise the rank's slice to Eq. 1 of
the exact full projection.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workloads
from oracle import compare
from oracle import projection as P
from oracle import qknorm as Q
from paper_2608_09160_amd import _lib as L

from gpu_util import DEV, bits_of, to_dev_bf16, to_dev_f32

pytestmark = pytest.mark.gpu


def _run(x_bits, w_list, x_dev=None, w_devs=None, y_devs=None):
    x = to_dev_bf16(x_bits) if x_dev is None else x_dev
    segs = [L.ProjSeg(w=to_dev_bf16(w) if w_devs is None else w_devs[i],
                      y=None if y_devs is None else y_devs[i])
            for i, w in enumerate(w_list)]
    L.qkn_proj_partial(x, segs)
    info = L.qkn_last_launch()
    torch.cuda.synchronize()
    return [(bits_of(s.y), s.partials.cpu().numpy()) for s in segs], info


def _check(x_bits, w_bits, y_bits, part, what):
    hidden = x_bits.shape[1]
    q = P.project(x_bits, w_bits)
    da = P.dot_abs(x_bits, w_bits)
    yv = Q.decode_bf16(y_bits)
    compare.check_projection(yv, q, da, hidden, f"{what} y")
    ref = P.stored_partials(x_bits, w_bits)
    bound = compare.projection_partial_bound(q, da, hidden)
    err = np.abs(part.astype(np.float64) - ref)
    assert np.all(err <= bound), f"{what} partial: {err.max():.3e} > bound"
    # the statistic is the fp32 sum of the stored row's squares
    own = np.sum(yv * yv, axis=1)
    compare.check_close(part, own, compare.PARTIAL_RTOL, f"{what} partial vs stored row")


@pytest.mark.parametrize("T,hidden,dq,dk", [(300, 4096, 2048, 512), (1, 64, 8, 0), (129, 136, 200, 72),
                                             (77, 1000, 128, 8), (256, 2048, 1024, 256),
                                             (5, 8, 16, 0), (130, 4104, 136, 0), (37, 520, 264, 40),
                                             (64, 8192, 8, 2040)])
def test_projection_matches_oracle(T, hidden, dq, dk):
    rng = np.random.default_rng(T * 31 + hidden)
    x = workloads.f32_to_bf16_bits(rng.standard_normal((T, hidden), dtype=np.float32))
    ws = [workloads.f32_to_bf16_bits(rng.standard_normal((d, hidden), dtype=np.float32) / np.sqrt(hidden))
          for d in (dq, dk) if d]
    print(f"[proj] T={T} hidden={hidden} d={dq}/{dk}", flush=True)
    outs, info = _run(x, ws)
    assert info["kernel"].startswith("proj<"), info
    for (y, part), w, t in zip(outs, ws, "qk"):
        _check(x, w, y, part, f"{t} T={T} h={hidden}")


def test_q_and_k_in_one_launch_equal_separate_launches():
    wl = workloads.DECODE_TP4
    data = workloads.projection_inputs(wl)
    x = data["x"]
    wq = data["wq"][workloads.shard_cols(wl.q_full, wl.tp, 1)]
    wk = data["wk"][workloads.shard_cols(wl.k_full, wl.tp, 1)]
    both, _ = _run(x, [wq, wk])
    q_alone, _ = _run(x, [wq])
    k_alone, _ = _run(x, [wk])
    assert np.array_equal(both[0][0], q_alone[0][0]) and np.array_equal(both[0][1], q_alone[0][1])
    assert np.array_equal(both[1][0], k_alone[0][0]) and np.array_equal(both[1][1], k_alone[0][1])
    again, _ = _run(x, [wq, wk])
    for a, b in zip(again, both):
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_strided_operands_and_column_slices():
    """x and W as column slices of wider buffers, Q and K written into disjoint
    column ranges of one [T, dq + dk + 64] buffer."""
    rng = np.random.default_rng(3)
    T, h, dq, dk = 200, 512, 256, 64
    x = workloads.f32_to_bf16_bits(rng.standard_normal((T, h), dtype=np.float32))
    wq = workloads.f32_to_bf16_bits(rng.standard_normal((dq, h), dtype=np.float32) / 20)
    wk = workloads.f32_to_bf16_bits(rng.standard_normal((dk, h), dtype=np.float32) / 20)
    base, _ = _run(x, [wq, wk])
    xbig = torch.zeros((T, h + 24), dtype=torch.bfloat16, device=DEV)
    xbig[:, 16:16 + h] = to_dev_bf16(x)
    wbig = torch.zeros((dq + dk, h + 8), dtype=torch.bfloat16, device=DEV)
    wbig[:dq, 8:] = to_dev_bf16(wq)
    wbig[dq:, 8:] = to_dev_bf16(wk)
    out = torch.zeros((T, dq + dk + 64), dtype=torch.bfloat16, device=DEV)
    outs, _ = _run(x, [wq, wk], x_dev=xbig[:, 16:16 + h], w_devs=[wbig[:dq, 8:], wbig[dq:, 8:]],
                   y_devs=[out[:, 8:8 + dq], out[:, 8 + dq:8 + dq + dk]])
    for a, b in zip(outs, base):
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert not out[:, :8].float().abs().sum() and not out[:, 8 + dq + dk:].float().abs().sum()


def test_end_to_end_with_apply_matches_full_norm():
    """Every rank projects its slices (statistic in the epilogue); rank r's
    qkn_apply with all ranks' statistics gives Eq. 1 of the exact projection."""
    wl = workloads.DECODE_TP4
    data = workloads.projection_inputs(wl)
    gamma = workloads.generate(wl)
    x = data["x"]
    hidden = x.shape[1]
    for key, wkey, gkey, d_full in (("q", "wq", "gq", wl.q_full), ("k", "wk", "gk", wl.k_full)):
        print(f"[proj] end to end {key}", flush=True)
        stats = torch.empty((wl.tp, wl.T), dtype=torch.float32, device=DEV)
        ys = []
        for r in range(wl.tp):
            outs, _ = _run(x, [data[wkey][workloads.shard_cols(d_full, wl.tp, r)]])
            y, part = outs[0]
            stats[r] = torch.from_numpy(part).to(DEV)
            ys.append(y)
        q_exact = P.project(x, data[wkey])
        da = P.dot_abs(x, data[wkey])
        g = gamma[gkey]
        ref = Q.rmsnorm(q_exact, g, wl.eps)
        inv = Q.rms_factor(Q.sum_of_squares(q_exact), d_full, wl.eps)
        for r in (0, wl.tp - 1):
            cols = workloads.shard_cols(d_full, wl.tp, r)
            out = L.qkn_apply(to_dev_bf16(ys[r]), to_dev_f32(g[cols]), stats, d_full, wl.eps)
            torch.cuda.synchronize()
            got = Q.decode_bf16(bits_of(out))
            # relative 8e-3 (the output's rounding, the stored projection's
            # rounding and the factor's change) plus the projection's absolute
            # error carried through gamma and the factor
            eps_abs = compare.projection_error_bound(q_exact[:, cols], da[:, cols], hidden)
            scale = inv[:, None] * np.abs(g[cols].astype(np.float64))[None, :]
            bound = compare.OUTPUT_RTOL * np.abs(ref[:, cols]) + 1.01 * scale * eps_abs
            excess = np.abs(got - ref[:, cols]) - bound
            assert np.all(excess <= 0), (key, r, float(excess.max()))


def test_full_size_prefill_sampled():
    """The prefill shapes (8192 tokens, hidden 4096, Q/K slices 2048/512 of rank
    0 of tp 2) in one launch; the oracle checks 128 sampled tokens."""
    wl = workloads.PREFILL_TP2
    data = workloads.projection_inputs(wl)
    x = data["x"]
    wq = data["wq"][workloads.shard_cols(wl.q_full, wl.tp, 0)]
    wk = data["wk"][workloads.shard_cols(wl.k_full, wl.tp, 0)]
    print("[proj] full-size prefill", flush=True)
    outs, info = _run(x, [wq, wk])
    rng = np.random.default_rng(4)
    rows = np.unique(np.concatenate([[0, wl.T - 1], rng.choice(wl.T, 126, replace=False)]))
    for (y, part), w, t in zip(outs, (wq, wk), "qk"):
        _check(x[rows], w, y[rows], part[rows], f"{t} sampled")
        yv = Q.decode_bf16(y)
        compare.check_close(part, np.sum(yv * yv, axis=1), compare.PARTIAL_RTOL, f"{t} all rows")


def test_errors_raise():
    x = torch.zeros((4, 64), dtype=torch.bfloat16, device=DEV)
    w = torch.zeros((16, 64), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(L.QknError) as e:
        L.qkn_proj_partial(x[:, 1:57], [L.ProjSeg(w=w[:, :56])])
    assert e.value.status == L.QKN_ENOTSUP  # x misaligned by one element
    y = torch.zeros((4, 16), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(L.QknError) as e:
        L.qkn_proj_partial(x, [L.ProjSeg(w=w, y=y, partials=y.view(torch.float32)[0, :4])])
    assert e.value.status == L.QKN_EOVERLAP


def test_all_kernels_give_the_same_bits():
    """The direct-to-LDS kernels (16 x 16 x 32 and 32 x 32 x 16 MFMAs) and the
    register-staged one accumulate every output over the same k-blocks in the
    same order: identical y and statistics."""
    rng = np.random.default_rng(8)
    T, h, dq, dk = 333, 1096, 264, 136
    x = workloads.f32_to_bf16_bits(rng.standard_normal((T, h), dtype=np.float32))
    ws = [workloads.f32_to_bf16_bits(rng.standard_normal((d, h), dtype=np.float32) / 30) for d in (dq, dk)]
    outs = []
    for choice, suffix in ((1, "dl2,mi16>"), (2, "reg>"), (3, "dl2>")):
        L.qkn_set_option("proj_tile", choice)
        try:
            o, info = _run(x, ws)
        finally:
            L.qkn_set_option("proj_tile", 0)
        assert info["kernel"].endswith(suffix), info
        outs.append(o)
    for other in outs[1:]:
        for a, b in zip(outs[0], other):
            assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    for (y, part), w, t in zip(outs[0], ws, "qk"):
        _check(x, w, y, part, t)


@pytest.mark.parametrize("T,hidden", [(64, 4096), (1, 1096), (1024, 512)])
def test_split_k_against_one_slice(T, hidden):
    """Decode-sized launches split k into slices added in ascending order; the
    forced single-slice kernel sums the same products in another order. Both
    pass the oracle, so they differ by at most twice the error bound; and as
    the same fp32 sums in two orders, most stored values are identical."""
    rng = np.random.default_rng(T + hidden)
    dq, dk = 1024, 264
    x = workloads.f32_to_bf16_bits(rng.standard_normal((T, hidden), dtype=np.float32))
    ws = [workloads.f32_to_bf16_bits(rng.standard_normal((d, hidden), dtype=np.float32) / np.sqrt(hidden))
          for d in (dq, dk)]
    print(f"[proj] split k T={T} hidden={hidden}", flush=True)
    split, info = _run(x, ws)
    assert info["kernel"].endswith("splitk>"), info
    L.qkn_set_option("proj_tile", 1)
    try:
        whole, info1 = _run(x, ws)
    finally:
        L.qkn_set_option("proj_tile", 0)
    assert not info1["kernel"].endswith("splitk>"), info1
    for (ys, ps), (yw, pw), w, t in zip(split, whole, ws, "qk"):
        _check(x, w, ys, ps, f"{t} split")
        _check(x, w, yw, pw, f"{t} one slice")
        a, b = Q.decode_bf16(ys), Q.decode_bf16(yw)
        assert np.mean(a == b) > 0.9, (t, float(np.mean(a == b)))
    again, _ = _run(x, ws)
    for a, b in zip(again, split):
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])

