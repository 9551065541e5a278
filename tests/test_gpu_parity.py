"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Tolerances (stated in oracle/compare.py): fp32 partial sums within 1e-5
relative, bf16 outputs within 8e-3 relative (about 2 bf16 ulps), specials
matched. Internal invariants are bit-exact: a rank's own statistic equals
qkn_partial_sumsq of its slice, every rank gets the same factor, repeated and
re-shaped launches and the general kernel give the same bits.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workloads
from oracle import compare
from oracle import qknorm as Q
from paper_2608_09160_amd import _lib as L

from gpu_util import (DEV, bits_of, check_rank_every_token, check_ranks_every_token, inputs,
                      peer_partials, run_fused_rank, shard, to_dev_bf16, to_dev_f32)

pytestmark = pytest.mark.gpu

# Workloads at sizes the oracle finishes in seconds: the three small ones in
# full, the two prefill ones with fewer tokens and a ragged token count.
SMALL = [workloads.TINY_FULL, workloads.DECODE_TP4, workloads.DECODE_TP8,
         workloads.PREFILL_TP2.with_tokens(1000), workloads.LONG_PREFILL_TP4.with_tokens(777)]


def _check_rank(wl, data, rank, out):
    ref = Q.qknorm_layerwise(data["xq"], data["xk"], data["gq"], data["gk"], wl.tp, rank, wl.eps)
    ey, ep = [], []
    for t in "qk":
        r = ref[t]
        got = out[t]
        ey.append(compare.check_close(Q.decode_bf16(got["y"]), r["y"], compare.OUTPUT_RTOL,
                                      f"{wl.name} rank {rank} {t} y"))
        ep.append(compare.check_close(got["partials"][rank], r["partials"][rank],
                                      compare.PARTIAL_RTOL, f"{wl.name} rank {rank} {t} partial"))
        compare.check_close(got["inv"], r["inv"], 1e-5, f"{wl.name} rank {rank} {t} inv")
    print(f"[errors] {wl.name} rank {rank}: max y rel error {max(ey):.3e}, max statistic rel "
          f"error {max(ep):.3e}", flush=True)


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_fused_every_rank_matches_oracle(wl):
    data = inputs(wl)
    invs = []
    ys = {"q": [], "k": []}
    for rank in range(wl.tp):
        print(f"[parity] {wl.name} rank {rank}", flush=True)
        out = run_fused_rank(wl, data, rank)
        assert out["launch"]["kernel"].startswith("rows"), out["launch"]
        _check_rank(wl, data, rank, out)
        invs.append((out["q"]["inv"], out["k"]["inv"]))
        for t in "qk":
            ys[t].append(out[t]["y"])
        # the own statistic is bit-identical to Phase A alone on the same slice
        for t, key, d_full in (("q", "xq", wl.q_full), ("k", "xk", wl.k_full)):
            alone = L.qkn_partial_sumsq(to_dev_bf16(shard(data, key, d_full, wl.tp, rank)))
            assert np.array_equal(out[t]["partials"][rank], alone.cpu().numpy())
    # every rank combines the same statistics in the same order: equal factors
    for q_inv, k_inv in invs[1:]:
        assert np.array_equal(q_inv, invs[0][0]) and np.array_equal(k_inv, invs[0][1])
    # concatenated shards == unsharded Eq. 1
    full = Q.qknorm_layerwise(data["xq"], data["xk"], data["gq"], data["gk"], 1, 0, wl.eps)
    for t in "qk":
        got = Q.decode_bf16(np.concatenate(ys[t], axis=1))
        compare.check_close(got, full[t]["y"], compare.OUTPUT_RTOL, f"{wl.name} {t} concat")
        # the three error metrics of Sec. IV-C against the fp64 output
        m = compare.paper_error_metrics(got, full[t]["y"])
        print(f"[parity] {wl.name} {t} max/mean/rms abs error "
              f"{m['max_abs']:.3e} {m['mean_abs']:.3e} {m['rms_abs']:.3e}", flush=True)


@pytest.mark.parametrize("wl", [workloads.TINY_FULL, workloads.PREFILL_TP2.with_tp(1).with_tokens(513)],
                         ids=lambda w: w.name)
def test_full_vector_matches_oracle(wl):
    data = inputs(wl)
    print(f"[parity] full {wl.name}", flush=True)
    segs = [L.Seg(x=to_dev_bf16(data["xq"]), w=to_dev_f32(data["gq"]), d_full=wl.q_full,
                  partials=torch.empty((1, wl.T), dtype=torch.float32, device=DEV)),
            L.Seg(x=to_dev_bf16(data["xk"]), w=to_dev_f32(data["gk"]), d_full=wl.k_full)]
    L.qkn_full(segs, wl.eps)
    torch.cuda.synchronize()
    ref = Q.qknorm_layerwise(data["xq"], data["xk"], data["gq"], data["gk"], 1, 0, wl.eps)
    compare.check_close(Q.decode_bf16(bits_of(segs[0].y)), ref["q"]["y"], compare.OUTPUT_RTOL, "q")
    compare.check_close(Q.decode_bf16(bits_of(segs[1].y)), ref["k"]["y"], compare.OUTPUT_RTOL, "k")
    compare.check_close(segs[0].partials.cpu().numpy()[0], ref["q"]["partials"][0],
                        compare.PARTIAL_RTOL, "q full sum")


@pytest.mark.parametrize("wl", [workloads.LONG_PREFILL_TP4.with_tp(1).with_tokens(777),
                                workloads.DECODE_TP8.with_tp(1)], ids=lambda w: w.name)
def test_wide_full_vector_matches_oracle(wl):
    """tp = 1 with Q wider than the register path (8192 and 5120 columns)."""
    data = inputs(wl)
    print(f"[parity] wide full {wl.name}", flush=True)
    out = run_fused_rank(wl, data, 0)
    assert out["launch"]["kernel"].startswith("wide<16,2>"), out["launch"]
    ref = Q.qknorm_layerwise(data["xq"], data["xk"], data["gq"], data["gk"], 1, 0, wl.eps)
    for t in "qk":
        compare.check_close(Q.decode_bf16(out[t]["y"]), ref[t]["y"], compare.OUTPUT_RTOL, t)
        compare.check_close(out[t]["partials"][0], ref[t]["partials"][0], compare.PARTIAL_RTOL, t)
    # the general kernel gives the same bits
    L.qkn_set_option("force_generic", 1)
    try:
        gen = run_fused_rank(wl, data, 0)
    finally:
        L.qkn_set_option("force_generic", 0)
    assert gen["launch"]["kernel"] == "generic/fused"
    for t in "qk":
        assert np.array_equal(gen[t]["y"], out[t]["y"]) and np.array_equal(gen[t]["inv"], out[t]["inv"])


def test_tp_invariance():
    """One oracle, every TP degree: shards at tp 1, 2, 4, 8 all agree with it."""
    base = workloads.PREFILL_TP2.with_tokens(300)
    data = inputs(base)
    full = Q.qknorm_layerwise(data["xq"], data["xk"], data["gq"], data["gk"], 1, 0, base.eps)
    for tp in (1, 2, 4, 8):
        wl = base.with_tp(tp)
        parts = {"q": [], "k": []}
        for rank in range(tp):
            out = run_fused_rank(wl, data, rank)
            for t in "qk":
                parts[t].append(out[t]["y"])
        for t in "qk":
            compare.check_close(Q.decode_bf16(np.concatenate(parts[t], axis=1)), full[t]["y"],
                                compare.OUTPUT_RTOL, f"tp={tp} {t}")


def test_two_step_equals_fused_bitwise():
    """Phase A then Phases B+C as two launches (x read twice) gives the same bits."""
    wl = workloads.DECODE_TP4
    data = inputs(wl)
    rank = 2
    fused = run_fused_rank(wl, data, rank)
    for t, key, gkey, d_full in (("q", "xq", "gq", wl.q_full), ("k", "xk", "gk", wl.k_full)):
        x = to_dev_bf16(shard(data, key, d_full, wl.tp, rank))
        P = peer_partials(data, key, d_full, wl.tp, wl.T, rank)
        L.qkn_partial_sumsq(x, out=P[rank])
        inv = torch.empty(wl.T, dtype=torch.float32, device=DEV)
        y = L.qkn_apply(x, to_dev_f32(data[gkey][workloads.shard_cols(d_full, wl.tp, rank)]), P,
                        d_full, wl.eps, inv_rms=inv)
        assert L.qkn_last_launch()["kernel"].endswith("/apply")
        assert np.array_equal(bits_of(y), fused[t]["y"])
        assert np.array_equal(inv.cpu().numpy(), fused[t]["inv"])


def test_oracle_partials_as_peers():
    """Peers' statistics from the fp64 oracle (rounded to fp32) instead of the GPU."""
    wl = workloads.DECODE_TP8
    data = inputs(wl)
    rank = 5
    ref = Q.qknorm_layerwise(data["xq"], data["xk"], data["gq"], data["gk"], wl.tp, rank, wl.eps)
    segs = []
    for t, key, gkey, d_full in (("q", "xq", "gq", wl.q_full), ("k", "xk", "gk", wl.k_full)):
        cols = workloads.shard_cols(d_full, wl.tp, rank)
        P = to_dev_f32(ref[t]["partials"].astype(np.float32))
        segs.append(L.Seg(x=to_dev_bf16(data[key][:, cols]), w=to_dev_f32(data[gkey][cols]),
                          d_full=d_full, partials=P))
    L.qkn_fused_shard(segs, wl.tp, rank, wl.eps)
    torch.cuda.synchronize()
    for s, t in zip(segs, "qk"):
        compare.check_close(Q.decode_bf16(bits_of(s.y)), ref[t]["y"], compare.OUTPUT_RTOL, t)


def test_phase_c_rounding_is_rne_of_fp32_product():
    """y == bf16_rne((x * w) * inv) in fp32, with the kernel's own factor (CPU torch)."""
    wl = workloads.DECODE_TP4
    data = inputs(wl)
    out = run_fused_rank(wl, data, 1)
    for t, key, gkey, d_full in (("q", "xq", "gq", wl.q_full), ("k", "xk", "gk", wl.k_full)):
        cols = workloads.shard_cols(d_full, wl.tp, 1)
        x = torch.from_numpy(np.ascontiguousarray(data[key][:, cols]).view(np.int16)).view(torch.bfloat16).float()
        w = torch.from_numpy(data[gkey][cols])
        inv = torch.from_numpy(out[t]["inv"])[:, None]
        expect = ((x * w) * inv).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(out[t]["y"], expect)


# ------------------------------------------------------------------ full sizes

@pytest.mark.parametrize("wl", [workloads.PREFILL_TP2, workloads.LONG_PREFILL_TP4],
                         ids=lambda w: w.name)
def test_full_size_every_token(wl):
    """Full token counts in the benchmark's launch shape (each wavefront walks
    several tokens of the persistent loop): every rank, every token, every
    element against the oracle; own statistic == Phase A alone; equal factors
    on all ranks; a second launch gives the same bits."""
    data = inputs(wl)
    outs = {}
    for rank in range(wl.tp):
        print(f"[parity] full size {wl.name} rank {rank}", flush=True)
        out = run_fused_rank(wl, data, rank)
        assert out["launch"]["kernel"].startswith("rows")
        assert out["launch"]["waves"] < wl.T  # several tokens per wavefront
        outs[rank] = out
    print(f"[parity] oracle on every token: {wl.name}", flush=True)
    check_ranks_every_token(wl, data, outs, wl.name)
    for rank, out in outs.items():
        for t, key, d_full in (("q", "xq", wl.q_full), ("k", "xk", wl.k_full)):
            alone = L.qkn_partial_sumsq(to_dev_bf16(shard(data, key, d_full, wl.tp, rank)))
            assert np.array_equal(out[t]["partials"][rank], alone.cpu().numpy())
            assert np.array_equal(out[t]["inv"], outs[0][t]["inv"])
    again = run_fused_rank(wl, data, wl.tp - 1)
    for t in "qk":
        assert np.array_equal(again[t]["y"], outs[wl.tp - 1][t]["y"])


def test_full_vector_prefill_every_token():
    """The tp = 1 baseline (the compute of the all-gather path) at 8192 tokens:
    every token against the oracle."""
    wl = workloads.PREFILL_TP2.with_tp(1)
    data = inputs(workloads.PREFILL_TP2)
    print("[parity] full-vector prefill", flush=True)
    out = run_fused_rank(wl, data, 0)
    assert out["launch"]["kernel"].endswith("<8,2>/fused")
    assert out["launch"]["waves"] < wl.T
    check_rank_every_token(wl, data, 0, out, wl.name)


@pytest.mark.parametrize("opt", [None, ("waves_per_cu", 1), ("prefetch", 1), ("balance", 1),
                                 ("token_blocks", 1), ("waves_per_block", 4)],
                         ids=lambda o: "default" if o is None else f"{o[0]}={o[1]}")
def test_several_tokens_per_wave_against_oracle(opt):
    """A ragged token count (2049) with one wavefront per CU, so every
    wavefront walks eight or nine tokens of the persistent loop, under each
    scheduling option (strided tokens, the pipelined loop, equal shares,
    contiguous blocks): every token against the oracle."""
    wl = workloads.PREFILL_TP2.with_tokens(2049)
    data = inputs(wl)
    opts = [("waves_per_cu", 1)] if opt is None or opt[0] != "waves_per_cu" else []
    if opt is not None:
        opts.append(opt)
    for k, v in opts:
        L.qkn_set_option(k, v)
    try:
        out = run_fused_rank(wl, data, 1)
    finally:
        for k, _ in opts:
            L.qkn_set_option(k, 0)
    waves = out["launch"]["waves"]
    assert waves * 8 <= wl.T, out["launch"]
    check_rank_every_token(wl, data, 1, out, f"{wl.name} {opts}")


# ------------------------------------------------------------------ general path and shapes

def _single(x_bits, gamma, d_full, tp, rank, eps, peers=None, x_dev=None, y_dev=None):
    """One segment through qkn_fused_shard; peers: fp32 [tp, T] host array or None."""
    T = x_bits.shape[0]
    x = to_dev_bf16(x_bits) if x_dev is None else x_dev
    P = torch.from_numpy(np.asarray(peers, np.float32)).to(DEV) if peers is not None else \
        torch.zeros((tp, T), dtype=torch.float32, device=DEV)
    inv = torch.empty(T, dtype=torch.float32, device=DEV)
    seg = L.Seg(x=x, w=to_dev_f32(gamma), d_full=d_full, partials=P, inv_rms=inv, y=y_dev)
    L.qkn_fused_shard([seg], tp, rank, eps)
    info = L.qkn_last_launch()
    torch.cuda.synchronize()
    return bits_of(seg.y), P.cpu().numpy(), inv.cpu().numpy(), info


def _oracle_single(x_full_bits, gamma_full, tp, rank, eps):
    return Q.qknorm_shard(x_full_bits, gamma_full, tp, rank, eps)


@pytest.mark.parametrize("T,d_local,tp", [(1, 1, 1), (3, 7, 2), (33, 100, 3), (70, 4104, 2),
                                          (9, 20000, 1), (5, 40000, 2), (130, 8, 4),
                                          (67, 4096, 2), (64, 520, 4), (5, 24, 65), (4, 16, 130),
                                          (37, 5120, 1), (300, 8192, 2), (21, 16384, 1),
                                          (13, 8200, 3)])
def test_shapes_fast_and_general(T, d_local, tp):
    d_full = d_local * tp
    x_full = workloads.random_rows(T * 7 + d_local, T, d_full, "student_t")
    g_full = workloads.random_gamma(d_local, d_full)
    rank = tp // 2
    ref = _oracle_single(x_full, g_full, tp, rank, 1e-6)
    cols = workloads.shard_cols(d_full, tp, rank)
    peers = ref["partials"].astype(np.float32)
    peers[rank] = np.nan  # must not be read
    print(f"[parity] shape T={T} d={d_local} tp={tp}", flush=True)
    y, P, inv, info = _single(x_full[:, cols], g_full[cols], d_full, tp, rank, 1e-6, peers)
    compare.check_close(Q.decode_bf16(y), ref["y"], compare.OUTPUT_RTOL, "y")
    compare.check_close(P[rank], ref["partials"][rank], compare.PARTIAL_RTOL, "own partial")
    # the general kernel gives the same bits as whichever kernel ran
    L.qkn_set_option("force_generic", 1)
    try:
        peers2 = peers.copy()
        y2, P2, inv2, info2 = _single(x_full[:, cols], g_full[cols], d_full, tp, rank, 1e-6, peers2)
    finally:
        L.qkn_set_option("force_generic", 0)
    assert info2["kernel"] == "generic/fused"
    assert np.array_equal(y2, y) and np.array_equal(P2[rank], P[rank]) and np.array_equal(inv2, inv)


def test_strided_misaligned_and_in_place():
    T, d, tp, rank = 45, 512, 2, 1
    x_full = workloads.random_rows(5, T, d * tp)
    g_full = workloads.random_gamma(5, d * tp)
    ref = _oracle_single(x_full, g_full, tp, rank, 1e-6)
    peers = ref["partials"].astype(np.float32)
    shard_bits = x_full[:, workloads.shard_cols(d * tp, tp, rank)]
    base, _, _, info = _single(shard_bits, g_full[d:], d * tp, tp, rank, 1e-6, peers)
    assert info["kernel"].startswith("rows")
    compare.check_close(Q.decode_bf16(base), ref["y"], compare.OUTPUT_RTOL, "contiguous")
    # column slice of a wider buffer (aligned stride) -> fast path, same bits
    wide = torch.zeros((T, 1536), dtype=torch.bfloat16, device=DEV)
    wide[:, 512:1024] = to_dev_bf16(shard_bits)
    ystore = torch.zeros((T, 1536), dtype=torch.bfloat16, device=DEV)
    y, _, _, info = _single(shard_bits, g_full[d:], d * tp, tp, rank, 1e-6, peers,
                            x_dev=wide[:, 512:1024], y_dev=ystore[:, 8:520])
    assert info["kernel"].startswith("rows")
    assert np.array_equal(y, base)
    assert not ystore[:, :8].any() and not ystore[:, 520:].any()  # nothing outside the slice
    # misaligned by one element -> general scalar path, same bits
    odd = torch.zeros((T, 1536), dtype=torch.bfloat16, device=DEV)
    odd[:, 1:513] = to_dev_bf16(shard_bits)
    y, _, _, info = _single(shard_bits, g_full[d:], d * tp, tp, rank, 1e-6, peers,
                            x_dev=odd[:, 1:513])
    assert info["kernel"] == "generic/fused"
    assert np.array_equal(y, base)
    # in place: y is x
    xin = to_dev_bf16(shard_bits)
    y, _, _, _ = _single(shard_bits, g_full[d:], d * tp, tp, rank, 1e-6, peers, x_dev=xin, y_dev=xin)
    assert np.array_equal(y, base)


def test_special_values():
    T, d = 6, 64
    x = np.ones((T, 2 * d), np.float32)
    x[0, 3] = np.nan          # rank 0's slice: NaN poisons both slices of row 0
    x[1, d + 5] = np.inf      # inf in rank 1's slice: factor 0, inf * 0 = NaN there
    x[2] = 0.0                # zero row, eps = 0 -> NaN
    x[3] = 0.0                # (checked again below with eps > 0)
    x[4, :d] = 0.0            # rank 0 holds zeros, rank 1 ones
    bits = workloads.f32_to_bf16_bits(x)
    g = np.ones(2 * d, np.float32)
    for eps in (0.0, 1e-3):
        ref0 = _oracle_single(bits, g, 2, 0, eps)
        ref1 = _oracle_single(bits, g, 2, 1, eps)
        for rank, ref in ((0, ref0), (1, ref1)):
            peers = ref["partials"].astype(np.float32)
            y, P, inv, _ = _single(bits[:, rank * d:(rank + 1) * d], g[:d], 2 * d, 2, rank, eps, peers)
            compare.check_close(Q.decode_bf16(y), ref["y"], compare.OUTPUT_RTOL, f"eps={eps} r={rank}")
            compare.check_close(inv, ref["inv"], 1e-6, "inv")


def test_power_of_two_scaling_is_bit_exact():
    wl = workloads.DECODE_TP4
    data = inputs(wl)
    base = run_fused_rank(wl, data, 3, eps=0.0)
    for k in (-4, 3):
        scaled = dict(data)
        for key in ("xq", "xk"):
            scaled[key] = workloads.f32_to_bf16_bits(Q.decode_bf16(data[key]) * 2.0 ** k)
        out = run_fused_rank(wl, scaled, 3, eps=0.0)
        for t in "qk":
            assert np.array_equal(out[t]["y"], base[t]["y"])
            assert np.array_equal(out[t]["partials"][3], base[t]["partials"][3] * np.float32(4.0 ** k))


@pytest.mark.parametrize("opt", [("waves_per_cu", 1), ("waves_per_cu", 3), ("waves_per_block", 1),
                                 ("waves_per_block", 2), ("waves_per_block", 4)])
def test_launch_shape_does_not_change_bits(opt):
    wl = workloads.PREFILL_TP2.with_tokens(2049)
    data = inputs(wl)
    base = run_fused_rank(wl, data, 1)
    L.qkn_set_option(*opt)
    try:
        out = run_fused_rank(wl, data, 1)
    finally:
        L.qkn_set_option(opt[0], 0)
    for t in "qk":
        assert np.array_equal(out[t]["y"], base[t]["y"])
        assert np.array_equal(out[t]["partials"], base[t]["partials"])


def test_zero_tokens_leaves_outputs_alone():
    x = torch.zeros((0, 64), dtype=torch.bfloat16, device=DEV)
    seg = L.Seg(x=x, w=torch.ones(64, device=DEV), d_full=128,
                partials=torch.zeros((2, 0), device=DEV))
    L.qkn_fused_shard([seg], 2, 0, 1e-6)
    assert seg.y.shape == (0, 64)


def test_errors_raise():
    x = torch.zeros((4, 64), dtype=torch.bfloat16, device=DEV)
    seg = L.Seg(x=x, w=torch.ones(64, device=DEV), d_full=32, partials=torch.zeros((2, 4), device=DEV))
    with pytest.raises(L.QknError) as e:
        L.qkn_fused_shard([seg], 2, 0, 1e-6)
    assert e.value.status == L.QKN_EINVAL
    buf = torch.zeros(4 * 64 + 8, dtype=torch.bfloat16, device=DEV)
    x = buf[:256].view(4, 64)
    y = buf[1:257].view(4, 64)  # shifted by one element onto x
    seg = L.Seg(x=x, w=torch.ones(64, device=DEV), d_full=128,
                partials=torch.zeros((2, 4), device=DEV), y=y)
    with pytest.raises(L.QknError) as e:
        L.qkn_fused_shard([seg], 2, 0, 1e-6)
    assert e.value.status == L.QKN_EOVERLAP
