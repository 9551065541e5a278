"""GPU parity for FP8-E4M3 activations: the *_fp8 entry points against the oracle.

Sec. IV-C evaluates the method on FP8-E4M3 as well as bf16, with fp32
accumulation of the local and cross-rank sums. Inputs are the same seeded
draws as the bf16 workloads, quantised to e4m3fn (saturating at 448).

Tolerances (oracle/compare.py): fp32 partial sums within 1e-5 relative; FP8
outputs must be the round-to-nearest-even FP8 code of a value within 1e-5
relative of the fp64 oracle (``check_fp8``), NaN where the value rounds past
448. Internal invariants are bit-exact, as for bf16. Device buffers that are
sliced or filled here are uint8 tensors (the binding takes uint8 or
float8_e4m3fn), so no test depends on torch's own FP8 device kernels.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workloads
from oracle import compare
from oracle import qknorm as Q
from paper_2608_09160_amd import _lib as L

from gpu_util import (DEV, bits_of, check_ranks_every_token, inputs, peer_partials, run_fused_rank,
                      shard, to_dev_f32, to_dev_fp8)

pytestmark = pytest.mark.gpu

SMALL8 = [w.with_dtype("fp8") for w in
          (workloads.TINY_FULL, workloads.DECODE_TP4, workloads.DECODE_TP8,
           workloads.PREFILL_TP2.with_tokens(1000), workloads.LONG_PREFILL_TP4.with_tokens(777))]


def _ref(wl, data, tp, rank):
    return Q.qknorm_layerwise(data["xq"], data["xk"], data["gq"], data["gk"], tp, rank, wl.eps,
                              fmt="fp8")


@pytest.mark.parametrize("wl", SMALL8, ids=lambda w: w.name)
def test_fp8_every_rank_matches_oracle(wl):
    data = inputs(wl)
    invs, ys = [], {"q": [], "k": []}
    for rank in range(wl.tp):
        print(f"[fp8] {wl.name} rank {rank}", flush=True)
        out = run_fused_rank(wl, data, rank)
        assert out["launch"]["kernel"].startswith("rows_fp8<"), out["launch"]
        ref = _ref(wl, data, wl.tp, rank)
        for t, key, d_full in (("q", "xq", wl.q_full), ("k", "xk", wl.k_full)):
            compare.check_fp8(Q.decode_e4m3(out[t]["y"]), ref[t]["y"], f"{wl.name} r{rank} {t} y")
            compare.check_close(out[t]["partials"][rank], ref[t]["partials"][rank],
                                compare.PARTIAL_RTOL, f"{t} partial")
            compare.check_close(out[t]["inv"], ref[t]["inv"], 1e-5, f"{t} inv")
            alone = L.qkn_partial_sumsq_fp8(to_dev_fp8(shard(data, key, d_full, wl.tp, rank)))
            assert np.array_equal(out[t]["partials"][rank], alone.cpu().numpy())
            ys[t].append(out[t]["y"])
        invs.append((out["q"]["inv"], out["k"]["inv"]))
    for q_inv, k_inv in invs[1:]:
        assert np.array_equal(q_inv, invs[0][0]) and np.array_equal(k_inv, invs[0][1])
    full = _ref(wl, data, 1, 0)
    for t in "qk":
        got = Q.decode_e4m3(np.concatenate(ys[t], axis=1))
        compare.check_fp8(got, full[t]["y"], f"{wl.name} {t} concat")
        # the three error metrics of Sec. IV-C against the fp64 output
        m = compare.paper_error_metrics(got, full[t]["y"])
        print(f"[fp8] {wl.name} {t} max/mean/rms abs error "
              f"{m['max_abs']:.3e} {m['mean_abs']:.3e} {m['rms_abs']:.3e}", flush=True)


@pytest.mark.parametrize("wl,kernel", [
    (workloads.PREFILL_TP2.with_tp(1).with_tokens(513).with_dtype("fp8"), "rows_fp8<4,1>/fused"),
    (workloads.LONG_PREFILL_TP4.with_tp(1).with_tokens(300).with_dtype("fp8"), "wide_fp8<8,1>/fused"),
    (workloads.DECODE_TP8.with_tp(1).with_dtype("fp8"), "wide_fp8<8,1>/fused")],
    ids=lambda v: getattr(v, "name", v))
def test_fp8_full_vector_matches_oracle(wl, kernel):
    data = inputs(wl)
    print(f"[fp8] full {wl.name}", flush=True)
    segs = [L.Seg(x=to_dev_fp8(data["xq"]), w=to_dev_f32(data["gq"]), d_full=wl.q_full,
                  partials=torch.empty((1, wl.T), dtype=torch.float32, device=DEV),
                  inv_rms=torch.empty(wl.T, dtype=torch.float32, device=DEV)),
            L.Seg(x=to_dev_fp8(data["xk"]), w=to_dev_f32(data["gk"]), d_full=wl.k_full)]
    L.qkn_full_fp8(segs, wl.eps)
    assert L.qkn_last_launch()["kernel"] == kernel
    torch.cuda.synchronize()
    ref = _ref(wl, data, 1, 0)
    y = [bits_of(s.y) for s in segs]
    compare.check_fp8(Q.decode_e4m3(y[0]), ref["q"]["y"], "q")
    compare.check_fp8(Q.decode_e4m3(y[1]), ref["k"]["y"], "k")
    compare.check_close(segs[0].partials.cpu().numpy()[0], ref["q"]["partials"][0],
                        compare.PARTIAL_RTOL, "q full sum")
    # the general kernel gives the same bits
    L.qkn_set_option("force_generic", 1)
    try:
        for s in segs:
            s.y = None
        L.qkn_full_fp8(segs, wl.eps)
        assert L.qkn_last_launch()["kernel"] == "generic_fp8/fused"
        torch.cuda.synchronize()
    finally:
        L.qkn_set_option("force_generic", 0)
    assert np.array_equal(bits_of(segs[0].y), y[0]) and np.array_equal(bits_of(segs[1].y), y[1])


def test_fp8_two_step_equals_fused_bitwise():
    wl = workloads.DECODE_TP4.with_dtype("fp8")
    data = inputs(wl)
    rank = 2
    fused = run_fused_rank(wl, data, rank)
    for t, key, gkey, d_full in (("q", "xq", "gq", wl.q_full), ("k", "xk", "gk", wl.k_full)):
        x = to_dev_fp8(shard(data, key, d_full, wl.tp, rank))
        P = peer_partials(data, key, d_full, wl.tp, wl.T, rank)
        L.qkn_partial_sumsq_fp8(x, out=P[rank])
        inv = torch.empty(wl.T, dtype=torch.float32, device=DEV)
        y = L.qkn_apply_fp8(x, to_dev_f32(data[gkey][workloads.shard_cols(d_full, wl.tp, rank)]),
                            P, d_full, wl.eps, inv_rms=inv)
        assert L.qkn_last_launch()["kernel"] == "rows_fp8<1,0>/apply"
        assert np.array_equal(bits_of(y), fused[t]["y"])
        assert np.array_equal(inv.cpu().numpy(), fused[t]["inv"])


def test_fp8_phase_c_is_rne_of_fp32_product():
    """y == e4m3fn_rne((x * w) * inv) in fp32 with the kernel's own factor (CPU torch cast)."""
    wl = workloads.DECODE_TP8.with_dtype("fp8")
    data = inputs(wl)
    out = run_fused_rank(wl, data, 3)
    for t, key, gkey, d_full in (("q", "xq", "gq", wl.q_full), ("k", "xk", "gk", wl.k_full)):
        cols = workloads.shard_cols(d_full, wl.tp, 3)
        x = torch.from_numpy(np.ascontiguousarray(data[key][:, cols])).view(torch.float8_e4m3fn).float()
        w = torch.from_numpy(data[gkey][cols])
        inv = torch.from_numpy(out[t]["inv"])[:, None]
        expect = ((x * w) * inv).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        assert np.array_equal(out[t]["y"], expect)


def _single8(x_bits, gamma, d_full, tp, rank, eps, peers, x_dev=None, y_dev=None):
    T = x_bits.shape[0]
    x = to_dev_fp8(x_bits) if x_dev is None else x_dev
    P = torch.from_numpy(np.asarray(peers, np.float32)).to(DEV)
    inv = torch.empty(T, dtype=torch.float32, device=DEV)
    seg = L.Seg(x=x, w=to_dev_f32(gamma), d_full=d_full, partials=P, inv_rms=inv, y=y_dev)
    L.qkn_fused_shard_fp8([seg], tp, rank, eps)
    info = L.qkn_last_launch()
    torch.cuda.synchronize()
    return bits_of(seg.y), P.cpu().numpy(), inv.cpu().numpy(), info


@pytest.mark.parametrize("T,d_local,tp", [(1, 1, 1), (3, 7, 2), (33, 100, 3), (70, 4112, 2),
                                          (130, 16, 4), (67, 4096, 2), (64, 1040, 4),
                                          (5, 32, 65), (37, 5120, 1), (300, 8192, 2),
                                          (21, 16384, 1), (13, 8208, 3), (9, 20000, 1)])
def test_fp8_shapes_fast_and_general(T, d_local, tp):
    d_full = d_local * tp
    x_full = workloads.random_rows(T * 7 + d_local, T, d_full, "student_t", dtype="fp8")
    g_full = workloads.random_gamma(d_local, d_full)
    rank = tp // 2
    ref = Q.qknorm_shard(x_full, g_full, tp, rank, 1e-6, fmt="fp8")
    cols = workloads.shard_cols(d_full, tp, rank)
    peers = ref["partials"].astype(np.float32)
    peers[rank] = np.nan  # must not be read
    print(f"[fp8] shape T={T} d={d_local} tp={tp}", flush=True)
    y, P, inv, info = _single8(x_full[:, cols], g_full[cols], d_full, tp, rank, 1e-6, peers)
    compare.check_fp8(Q.decode_e4m3(y), ref["y"], "y")
    compare.check_close(P[rank], ref["partials"][rank], compare.PARTIAL_RTOL, "own partial")
    L.qkn_set_option("force_generic", 1)
    try:
        y2, P2, inv2, info2 = _single8(x_full[:, cols], g_full[cols], d_full, tp, rank, 1e-6,
                                       peers.copy())
    finally:
        L.qkn_set_option("force_generic", 0)
    assert info2["kernel"] == "generic_fp8/fused"
    assert np.array_equal(y2, y) and np.array_equal(P2[rank], P[rank]) and np.array_equal(inv2, inv)


def test_fp8_strided_misaligned_and_in_place():
    T, d, tp, rank = 45, 512, 2, 1
    x_full = workloads.random_rows(5, T, d * tp, dtype="fp8")
    g_full = workloads.random_gamma(5, d * tp)
    ref = Q.qknorm_shard(x_full, g_full, tp, rank, 1e-6, fmt="fp8")
    peers = ref["partials"].astype(np.float32)
    shard_bits = x_full[:, d:]
    base, _, _, info = _single8(shard_bits, g_full[d:], d * tp, tp, rank, 1e-6, peers)
    assert info["kernel"].startswith("rows_fp8")
    compare.check_fp8(Q.decode_e4m3(base), ref["y"], "contiguous")
    src = torch.from_numpy(np.ascontiguousarray(shard_bits)).to(DEV)  # uint8 on the device
    # column slice of a wider uint8 buffer (16-byte aligned stride) -> fast path
    wide = torch.zeros((T, 1536), dtype=torch.uint8, device=DEV)
    wide[:, 512:1024] = src
    ystore = torch.zeros((T, 1536), dtype=torch.uint8, device=DEV)
    y, _, _, info = _single8(shard_bits, g_full[d:], d * tp, tp, rank, 1e-6, peers,
                             x_dev=wide[:, 512:1024], y_dev=ystore[:, 16:528])
    assert info["kernel"].startswith("rows_fp8")
    assert np.array_equal(y, base)
    assert not ystore[:, :16].any() and not ystore[:, 528:].any()
    # 8 bytes off a 16-byte boundary -> general path, same bits
    odd = torch.zeros((T, 1536), dtype=torch.uint8, device=DEV)
    odd[:, 8:520] = src
    y, _, _, info = _single8(shard_bits, g_full[d:], d * tp, tp, rank, 1e-6, peers,
                             x_dev=odd[:, 8:520])
    assert info["kernel"] == "generic_fp8/fused"
    assert np.array_equal(y, base)
    # in place
    xin = src.clone()
    y, _, _, _ = _single8(shard_bits, g_full[d:], d * tp, tp, rank, 1e-6, peers, x_dev=xin, y_dev=xin)
    assert np.array_equal(y, base)


def test_fp8_special_values():
    """NaN codes, overflow past 448 (no infinity: NaN), zero rows, negative zero."""
    T, d = 6, 64
    x = np.full((T, 2 * d), 0x38, np.uint8)   # 1.0
    x[0, 3] = 0x7F                            # NaN in rank 0's slice: the row's factor is NaN
    x[1, :] = 0x00
    x[1, 0] = 0x7E                            # one 448 in a zero row: y = sqrt(128) * gamma there
    x[2] = 0x00                               # zero row (NaN with eps = 0)
    x[3, d:] = 0x80                           # rank 1 holds -0.0
    x[4, :d] = 0xFE                           # rank 0 holds -448
    g = np.full(2 * d, 1.0, np.float32)
    g[0] = 64.0                               # row 1: y = sqrt(128) * 64 = 724, past 448: NaN
    for eps in (0.0, 1e-3):
        for rank in (0, 1):
            ref = Q.qknorm_shard(x, g, 2, rank, eps, fmt="fp8")
            peers = ref["partials"].astype(np.float32)
            y, P, inv, _ = _single8(x[:, rank * d:(rank + 1) * d], g[rank * d:(rank + 1) * d],
                                    2 * d, 2, rank, eps, peers)
            compare.check_fp8(Q.decode_e4m3(y), ref["y"], f"eps={eps} rank={rank}")
            compare.check_close(inv, ref["inv"], 1e-6, "inv")
            if rank == 0:
                assert y[1, 0] == 0x7F           # no infinity in e4m3fn: overflow is NaN
            if rank == 1:
                assert np.all(y[3] == 0x80)      # -0.0 * w * inv keeps its sign


def test_fp8_zero_tokens_and_dtype_errors():
    x = torch.zeros((0, 64), dtype=torch.uint8, device=DEV)
    seg = L.Seg(x=x, w=torch.ones(64, device=DEV), d_full=128,
                partials=torch.zeros((2, 0), device=DEV))
    L.qkn_fused_shard_fp8([seg], 2, 0, 1e-6)
    assert seg.y.shape == (0, 64)
    xb = torch.zeros((4, 64), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(TypeError):
        L.qkn_partial_sumsq_fp8(xb)
    with pytest.raises(TypeError):
        L.qkn_partial_sumsq(torch.zeros((4, 64), dtype=torch.uint8, device=DEV))
    buf = torch.zeros(4 * 64 + 16, dtype=torch.uint8, device=DEV)
    seg = L.Seg(x=buf[:256].view(4, 64), w=torch.ones(64, device=DEV), d_full=128,
                partials=torch.zeros((2, 4), device=DEV), y=buf[1:257].view(4, 64))
    with pytest.raises(L.QknError) as e:
        L.qkn_fused_shard_fp8([seg], 2, 0, 1e-6)
    assert e.value.status == L.QKN_EOVERLAP


@pytest.mark.parametrize("wl,kernel", [
    (workloads.PREFILL_TP2.with_dtype("fp8"), "rows_fp8<2,1>/fused"),
    (workloads.LONG_PREFILL_TP4.with_dtype("fp8"), "rows_fp8<2,1>/fused")],
    ids=lambda v: getattr(v, "name", v))
def test_fp8_full_size_every_token(wl, kernel):
    """The FP8 prefill shards at their full token counts in the benchmark's
    launch shape (several tokens per wavefront): every rank and every token
    against the oracle; own statistic == Phase A alone; a second launch gives
    the same bits."""
    data = inputs(wl)
    outs = {}
    for rank in range(wl.tp):
        print(f"[fp8] full size {wl.name} rank {rank}", flush=True)
        out = run_fused_rank(wl, data, rank)
        assert out["launch"]["kernel"] == kernel and out["launch"]["waves"] < wl.T
        for t, key, d_full in (("q", "xq", wl.q_full), ("k", "xk", wl.k_full)):
            assert not np.isnan(Q.decode_e4m3(out[t]["y"])).any()
            alone = L.qkn_partial_sumsq_fp8(to_dev_fp8(shard(data, key, d_full, wl.tp, rank)))
            assert np.array_equal(out[t]["partials"][rank], alone.cpu().numpy())
        outs[rank] = out
    print(f"[fp8] oracle on every token: {wl.name}", flush=True)
    check_ranks_every_token(wl, data, outs, wl.name)
    again = run_fused_rank(wl, data, 0)
    for t in "qk":
        assert np.array_equal(again[t]["y"], outs[0][t]["y"])
