"""GPU: the fused kernel waiting for concurrently published statistics.

A rank's fused kernel publishes its own statistics as flagged slots and spins
(bounded) until the other ranks' slots of each token carry the round's epoch.
Other ranks are emulated on one GPU either by publishing kernels on another
stream (issued first: kernels on separate streams are not guaranteed to run
concurrently on one GPU) or by running every rank of the group in one launch,
where all wavefronts are resident together. Every result is checked against
the fp64 oracle on every token and every rank -- outputs within the bf16
tolerance (FP8: as a rounding of the oracle), factors and published
statistics within 1e-5 relative -- and, as an extra check, bit for bit
against qkn_fused_shard given the same statistics. Every wait is bounded by a
spin limit, so a failure shows up as status = 1 and NaN outputs, never as a
hang; the time-out case is forced from the host by never publishing.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workloads
from paper_2608_09160_amd import _lib as L

from gpu_util import (DEV, bits_of, check_group_every_token, check_rank_every_token, inputs,
                      run_fused_rank, slot_values, to_dev_act, to_dev_f32)

pytestmark = pytest.mark.gpu

SPIN = 1 << 21  # polls per slot: ~1 s at most, far above any legitimate wait here


def _rank_inputs(wl, data, rank):
    segs, peers = [], []
    for key, gkey, d_full in (("xq", "gq", wl.q_full), ("xk", "gk", wl.k_full)):
        cols = workloads.shard_cols(d_full, wl.tp, rank)
        segs.append(L.Seg(x=to_dev_act(data[key][:, cols]), w=to_dev_f32(data[gkey][cols]),
                          d_full=d_full, inv_rms=torch.empty(wl.T, dtype=torch.float32, device=DEV)))
        peers.append([to_dev_act(data[key][:, workloads.shard_cols(d_full, wl.tp, k)])
                      for k in range(wl.tp)])
    return segs, peers


def _slot_arrays(wl):
    return [torch.zeros((wl.tp, wl.T), dtype=torch.int64, device=DEV) for _ in range(2)]


def _check_rank(wl, data, rank, segs, slots, epoch):
    """One waiting rank's results against the oracle on every token (y, the
    factor, the statistic it published), then bit for bit against
    qkn_fused_shard with the same peers' statistics."""
    out = {}
    for s, t, sl in zip(segs, "qk", slots):
        partials = np.full((wl.tp, wl.T), np.nan, dtype=np.float32)
        partials[rank] = slot_values(sl[rank].cpu().numpy(), epoch)
        out[t] = {"y": bits_of(s.y), "inv": s.inv_rms.cpu().numpy(), "partials": partials}
    check_rank_every_token(wl, data, rank, out, f"{wl.name} wait")
    ref = run_fused_rank(wl, data, rank)
    for t in "qk":
        assert np.array_equal(out[t]["y"], ref[t]["y"]), (rank, t)
        assert np.array_equal(out[t]["inv"], ref[t]["inv"]), (rank, t)
        assert np.array_equal(out[t]["partials"][rank], ref[t]["partials"][rank]), (rank, t)


@pytest.mark.parametrize("wl", [workloads.DECODE_TP4, workloads.DECODE_TP4.with_dtype("fp8"),
                                workloads.PREFILL_TP2, workloads.PREFILL_TP2.with_dtype("fp8")],
                         ids=lambda w: w.name)
def test_producers_and_consumer_on_separate_streams(wl):
    """Peers publish from another stream; the consumer uses whatever it finds,
    waiting where a slot is not there yet. (Kernels on separate streams are not
    guaranteed to run at the same time on one GPU, so the producers are issued
    first: the consumer may or may not have to wait, and must be right either way.)"""
    data = inputs(wl)
    rank = 1
    segs, peers = _rank_inputs(wl, data, rank)
    slots = _slot_arrays(wl)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    s_cons, s_prod = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    print(f"[wait] producers, then consumer, on two streams: {wl.name}", flush=True)
    with torch.cuda.stream(s_prod):
        for k in range(wl.tp):
            if k != rank:
                for i in range(2):
                    L.qkn_publish_partials(peers[i][k], slots[i][k], 1)
    with torch.cuda.stream(s_cons):
        L.qkn_fused_shard_wait(segs, wl.tp, rank, wl.eps, slots, epoch=1, spin_limit=SPIN,
                               co_resident=2, status=status)
    assert L.qkn_last_launch()["kernel"].endswith("/fused_wait")
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    _check_rank(wl, data, rank, segs, slots, 1)
    # the own slots were published with the epoch and the Phase A value
    partial = L.qkn_partial_sumsq_fp8 if wl.dtype == "fp8" else L.qkn_partial_sumsq
    alone = partial(peers[0][rank]).cpu().numpy()
    assert np.array_equal(slot_values(slots[0][rank].cpu().numpy(), 1), alone)


GROUPS = [workloads.DECODE_TP4, workloads.DECODE_TP8, workloads.PREFILL_TP2.with_tokens(2048),
          workloads.Workload("tp3_T300_q1536_k384", 300, 1536, 384, 3, "normal", 7),
          workloads.PREFILL_TP2, workloads.LONG_PREFILL_TP4]


@pytest.mark.parametrize("wl", GROUPS, ids=lambda w: w.name)
def test_whole_group_in_one_launch(wl):
    """Every rank of the group in one launch: each wavefront publishes its rank's
    statistic and waits for the others'; all of them are resident at once.
    Default schedule: each token's statistics published three tokens ahead."""
    info = _run_group_and_check(wl)
    assert info["kernel"].startswith("rows_pa3<"), info


@pytest.mark.parametrize("wl", [workloads.DECODE_TP4.with_dtype("fp8"), workloads.DECODE_TP8.with_dtype("fp8"),
                                workloads.PREFILL_TP2.with_tokens(2048).with_dtype("fp8"),
                                workloads.PREFILL_TP2.with_dtype("fp8")],
                         ids=lambda w: w.name)
def test_whole_group_in_one_launch_fp8(wl):
    """FP8-E4M3 activations: the same bits as qkn_fused_shard_fp8 per rank."""
    info = _run_group_and_check(wl)
    assert info["kernel"].startswith("rows_pa3_fp8<"), info


@pytest.mark.parametrize("sched", [0, 1, 2, 3])
@pytest.mark.parametrize("wl", [workloads.DECODE_TP4, workloads.PREFILL_TP2.with_tokens(2048),
                                workloads.Workload("tp3_T7_q384_k96", 7, 384, 96, 3, "normal", 9)],
                         ids=lambda w: w.name)
def test_whole_group_other_schedules(wl, sched):
    """The same with the other schedules -- token by token (publish, then
    wait, per token; 1 also requests the next token early) and publishing one
    or two tokens ahead -- identical results, also with fewer tokens than a
    schedule keeps in flight."""
    L.qkn_set_option("wait_schedule", sched)
    try:
        info = _run_group_and_check(wl)
        assert info["kernel"].startswith(("rows<", "rows_pf<", "rows_pa<", "rows_pa2<")[sched]), info
    finally:
        L.qkn_set_option("wait_schedule", 4)


def _run_group_and_check(wl):
    """Two rounds of the whole group on the same slots; the second round's
    results against the oracle on every token and rank, equal to the first
    round's, and bit-equal per rank to qkn_fused_shard."""
    data = inputs(wl)
    slots = _slot_arrays(wl)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    segs = [L.Seg(x=to_dev_act(data[key]), w=to_dev_f32(data[gkey]), d_full=d_full,
                  inv_rms=torch.empty((wl.tp, wl.T), dtype=torch.float32, device=DEV))
            for key, gkey, d_full in (("xq", "gq", wl.q_full), ("xk", "gk", wl.k_full))]
    torch.cuda.synchronize()
    print(f"[wait] group of {wl.tp} in one launch: {wl.name}", flush=True)
    first = None
    for epoch in (11, 12):  # a second round reuses the slots with a new epoch
        L.qkn_fused_group_wait(segs, wl.tp, wl.eps, slots, epoch=epoch, spin_limit=SPIN,
                               status=status)
        info = L.qkn_last_launch()
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        assert info["kernel"].endswith("/fused_wait") and info["waves"] % wl.tp == 0
        got = {t: (bits_of(s.y), s.inv_rms.cpu().numpy()) for s, t in zip(segs, "qk")}
        if first is None:
            first = got
    for t in "qk":
        assert np.array_equal(got[t][0], first[t][0]) and np.array_equal(got[t][1], first[t][1])
    print(f"[wait] oracle on every token and rank: {wl.name}", flush=True)
    check_group_every_token(wl, data, {t: got[t][0] for t in "qk"},
                            {t: got[t][1] for t in "qk"},
                            {t: sl.cpu().numpy() for t, sl in zip("qk", slots)}, 12, wl.name)
    for r in range(wl.tp):
        ref = run_fused_rank(wl, data, r)
        for s, t, d_full, sl in zip(segs, "qk", (wl.q_full, wl.k_full), slots):
            cols = workloads.shard_cols(d_full, wl.tp, r)
            assert np.array_equal(got[t][0][:, cols], ref[t]["y"]), (r, t)
            assert np.array_equal(got[t][1][r], ref[t]["inv"]), (r, t)
            assert np.array_equal(slot_values(sl[r].cpu().numpy(), 12), ref[t]["partials"][r]), (r, t)
    return info


def test_timeout_when_nobody_publishes():
    wl = workloads.DECODE_TP4
    data = inputs(wl)
    segs, _ = _rank_inputs(wl, data, 2)
    slots = _slot_arrays(wl)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    torch.cuda.synchronize()
    print("[wait] forced time-out (no producer, 64 polls)", flush=True)
    L.qkn_fused_shard_wait(segs, wl.tp, 2, wl.eps, slots, epoch=9, spin_limit=64,
                           co_resident=1, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 1
    for s in segs:
        assert torch.isnan(s.y.float()).all()
    # this rank still published its own statistics
    own = slots[1][2].cpu().numpy().view(np.uint64)
    assert np.all((own >> np.uint64(32)) == 9)


def test_epochs_reuse_slots_without_reset():
    wl = workloads.DECODE_TP8
    data = inputs(wl)
    rank = 6
    segs, peers = _rank_inputs(wl, data, rank)
    slots = _slot_arrays(wl)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    for epoch in (5, 6):
        for s in segs:
            if s.y is not None:
                s.y.zero_()
        torch.cuda.synchronize()
        print(f"[wait] epoch {epoch}", flush=True)
        with torch.cuda.stream(torch.cuda.Stream()):
            for k in range(wl.tp):
                if k != rank:
                    for i in range(2):
                        L.qkn_publish_partials(peers[i][k], slots[i][k], epoch)
        torch.cuda.synchronize()
        L.qkn_fused_shard_wait(segs, wl.tp, rank, wl.eps, slots, epoch=epoch, spin_limit=SPIN,
                               co_resident=1, status=status)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        _check_rank(wl, data, rank, segs, slots, epoch)
    # a round whose statistics never arrive does not use the previous round's
    print("[wait] stale epoch", flush=True)
    L.qkn_fused_shard_wait(segs, wl.tp, rank, wl.eps, slots, epoch=7, spin_limit=64,
                           co_resident=1, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 1
    assert torch.isnan(segs[0].y.float()).all()


def _random_group(rng, i):
    fmt = "fp8" if rng.random() < 0.4 else "bf16"
    per = 16 if fmt == "fp8" else 8           # elements per 16-byte chunk: the register path's unit
    tp = int(rng.choice([2, 3, 4, 5, 8]))
    q_local = int(rng.integers(1, 4096 // per + 1)) * per
    k_local = int(rng.integers(1, 1024 // per + 1)) * per
    T = int(np.exp(rng.uniform(0, np.log(3000))))
    dist = str(rng.choice(["normal", "normal_lognormal", "normal_outliers", "student_t"]))
    wl = workloads.Workload(f"random{i}_T{T}_q{q_local * tp}_k{k_local * tp}_tp{tp}", T,
                            q_local * tp, k_local * tp, tp, dist, 500 + i, sigma=0.7)
    return wl.with_dtype("fp8") if fmt == "fp8" else wl, int(rng.integers(0, 5))


@pytest.mark.parametrize("seed", range(4))
def test_random_groups_against_oracle(seed):
    """Seeded random whole-group waits: token counts 1..3000, tp 2..8, slice
    widths across the register path of both formats, all five schedules;
    every token and rank against the oracle (through _run_group_and_check)."""
    rng = np.random.default_rng(7000 + seed)
    for i in range(3):
        wl, sched = _random_group(rng, 10 * seed + i)
        print(f"[wait] random group {wl.name} schedule {sched}", flush=True)
        L.qkn_set_option("wait_schedule", sched)
        try:
            _run_group_and_check(wl)
        finally:
            L.qkn_set_option("wait_schedule", 4)
