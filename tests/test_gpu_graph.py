"""GPU: the prepared entry points captured in a HIP graph (decode serving
loops replay them). Every replay must equal the eager result bit for bit; the
replays are separated by eager work that overwrites the outputs, so a replay
that wrote nothing, or wrote stale values, is caught; the eager result and
every replay are also checked against the fp64 oracle (the norm on every
token and rank it computes, the projection within its rounding bound). The
library allocates nothing and records no memset, so its launches are
capturable as they are.

The Phase B wait entry points take the round's epoch as a launch argument,
which a captured launch keeps; their graph clears the slot arrays with a
fill kernel before the waiting launch (the recipe qkn.h gives), and the
test plants stale slots carrying that epoch between replays.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workloads
from paper_2608_09160_amd import _lib as L

from oracle import compare
from oracle import projection as P_oracle
from oracle import qknorm as Q

from gpu_util import (DEV, bits_of, check_group_every_token, check_rank_every_token, inputs,
                      peer_partials, to_dev_act, to_dev_bf16, to_dev_f32)

pytestmark = pytest.mark.gpu

REPLAYS = 4


def _fused_prepared(wl, rank):
    data = inputs(wl)
    segs = []
    for key, gkey, d_full in (("xq", "gq", wl.q_full), ("xk", "gk", wl.k_full)):
        cols = workloads.shard_cols(d_full, wl.tp, rank)
        segs.append(L.Seg(x=to_dev_act(data[key][:, cols]), w=to_dev_f32(data[gkey][cols]),
                          d_full=d_full,
                          partials=peer_partials(data, key, d_full, wl.tp, wl.T, rank),
                          inv_rms=torch.empty(wl.T, dtype=torch.float32, device=DEV)))
    return L.Prepared(segs, wl.tp, rank, wl.eps), segs


def _outputs(tensors):
    torch.cuda.synchronize()
    return [t.clone() for t in tensors]


def _graph_of(fn):
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    return g


def _check_replays(fn, outs, clobber, oracle_check=None):
    """Eager result, then REPLAYS replays each equal to it bit for bit;
    oracle_check(outputs) runs on the eager result and on every replay."""
    fn()
    ref = _outputs(outs)
    if oracle_check is not None:
        oracle_check(ref)
    g = _graph_of(fn)
    for r in range(REPLAYS):
        clobber(r)                       # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        got = _outputs(outs)
        for a, b in zip(ref, got):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"replay {r}"
        if oracle_check is not None:
            oracle_check(got)


@pytest.mark.parametrize("wl,rank", [(workloads.DECODE_TP4, 1), (workloads.DECODE_TP8, 7),
                                     (workloads.DECODE_TP4.with_dtype("fp8"), 2)],
                         ids=lambda v: getattr(v, "name", str(v)))
def test_fused_shard_graph_replays(wl, rank):
    print(f"[graph] fused {wl.name} rank {rank}", flush=True)
    prep, segs = _fused_prepared(wl, rank)
    outs = [t for s in segs for t in (s.y, s.inv_rms, s.partials)]

    def clobber(r):
        for s in segs:
            s.y.view(torch.uint8).fill_(0x7F)
            s.inv_rms.fill_(float(r))
            s.partials[rank].fill_(-1.0)

    def oracle_check(got):
        out = {t: {"y": bits_of(got[3 * i]), "inv": got[3 * i + 1].cpu().numpy(),
                   "partials": got[3 * i + 2].cpu().numpy()} for i, t in enumerate("qk")}
        check_rank_every_token(wl, inputs(wl), rank, out, f"{wl.name} graph")
    _check_replays(prep, outs, clobber, oracle_check)


@pytest.mark.parametrize("T,hidden,dq,dk", [(64, 4096, 1024, 256), (1300, 1096, 264, 136)])
def test_projection_graph_replays(T, hidden, dq, dk):
    """Decode sizes split k (slice launch + reduction), larger ones run whole
    tiles + the statistic sum: both two-launch sequences replay exactly."""
    print(f"[graph] projection T={T} hidden={hidden}", flush=True)
    rng = np.random.default_rng(T)
    x = to_dev_bf16(workloads.f32_to_bf16_bits(rng.standard_normal((T, hidden), dtype=np.float32)))
    ws = [to_dev_bf16(workloads.f32_to_bf16_bits(
        rng.standard_normal((d, hidden), dtype=np.float32) / np.sqrt(hidden))) for d in (dq, dk)]
    prep = L.PreparedProj(x, [L.ProjSeg(w=w) for w in ws])
    outs = [t for s in prep.segs for t in (s.y, s.partials)]

    def clobber(r):
        for s in prep.segs:
            s.y.view(torch.uint8).fill_(0x55)
            s.partials.fill_(float(r))
        prep.workspace.fill_(0xFF)
    x_bits = bits_of(x)
    w_bits = [bits_of(w) for w in ws]
    q_exact = [P_oracle.project(x_bits, wb) for wb in w_bits]
    dot_abs = [P_oracle.dot_abs(x_bits, wb) for wb in w_bits]
    stat = [P_oracle.stored_partials(x_bits, wb) for wb in w_bits]

    def oracle_check(got):
        for i in range(2):
            yv = Q.decode_bf16(bits_of(got[2 * i]))
            compare.check_projection(yv, q_exact[i], dot_abs[i], hidden, f"graph proj seg{i} y")
            err = np.abs(got[2 * i + 1].cpu().numpy().astype(np.float64) - stat[i])
            assert np.all(err <= compare.projection_partial_bound(q_exact[i], dot_abs[i], hidden))
    _check_replays(prep, outs, clobber, oracle_check)


@pytest.mark.parametrize("wl", [workloads.DECODE_TP4, workloads.DECODE_TP8.with_dtype("fp8")],
                         ids=lambda w: w.name)
def test_group_wait_graph_with_slots_cleared_in_the_graph(wl):
    """A whole tp group in one waiting launch, captured after a fill kernel
    that clears the slot arrays. Between replays the slots are overwritten
    eagerly with wrong statistics that carry the captured epoch: a replay that
    did not clear them first would accept those. Every replay equals eager."""
    print(f"[graph] group wait {wl.name}", flush=True)
    data = inputs(wl)
    slots = [torch.zeros((wl.tp, wl.T), dtype=torch.int64, device=DEV) for _ in range(2)]
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    segs = []
    for key, gkey, d_full in (("xq", "gq", wl.q_full), ("xk", "gk", wl.k_full)):
        x = to_dev_act(data[key])
        segs.append(L.Seg(x=x, w=to_dev_f32(data[gkey]), d_full=d_full, y=torch.empty_like(x),
                          inv_rms=torch.empty((wl.tp, wl.T), dtype=torch.float32, device=DEV)))
    epoch = 21

    def step():
        for s in slots:
            s.zero_()  # a fill kernel (no memset node): epoch 0 is never a round's
        L.qkn_fused_group_wait(segs, wl.tp, wl.eps, slots, epoch=epoch, spin_limit=1 << 20,
                               status=status)
    stale = (epoch << 32) | 0x3F800000  # statistic 1.0 with the captured epoch

    def clobber(r):
        for s in segs:
            s.y.view(torch.uint8).fill_(0x7F)
            s.inv_rms.fill_(float(r))
        for s in slots:
            s.fill_(stale)

    def oracle_check(got):
        check_group_every_token(wl, data, {"q": bits_of(got[0]), "k": bits_of(got[1])},
                                {"q": got[2].cpu().numpy(), "k": got[3].cpu().numpy()},
                                {t: sl.cpu().numpy() for t, sl in zip("qk", slots)}, epoch,
                                f"{wl.name} graph")
    _check_replays(step, [s.y for s in segs] + [s.inv_rms for s in segs], clobber, oracle_check)
    assert int(status.item()) == 0


@pytest.mark.parametrize("wl,rank", [(workloads.DECODE_TP4, 3), (workloads.DECODE_TP4.with_dtype("fp8"), 0)],
                         ids=lambda v: getattr(v, "name", str(v)))
def test_prepared_apply_equals_apply_and_replays(wl, rank):
    """PreparedPartial and PreparedApply (arguments marshalled once) give
    qkn_partial_sumsq's and qkn_apply's bits, eager and from a replayed graph."""
    print(f"[graph] prepared apply {wl.name} rank {rank}", flush=True)
    data = inputs(wl)
    cols = workloads.shard_cols(wl.q_full, wl.tp, rank)
    x = to_dev_act(data["xq"][:, cols])
    w = to_dev_f32(data["gq"][cols])
    P = peer_partials(data, "xq", wl.q_full, wl.tp, wl.T, rank)
    (L.qkn_partial_sumsq_fp8 if wl.dtype == "fp8" else L.qkn_partial_sumsq)(x, out=P[rank])
    inv = torch.empty(wl.T, dtype=torch.float32, device=DEV)
    ref_y = (L.qkn_apply_fp8 if wl.dtype == "fp8" else L.qkn_apply)(x, w, P, wl.q_full, wl.eps,
                                                                     inv_rms=inv)
    ref = _outputs([ref_y, inv])
    part = L.PreparedPartial(x)
    assert torch.equal(part(), P[rank])  # the prepared Phase A gives the same statistic
    prep = L.PreparedApply(x, w, P, wl.q_full, wl.eps,
                           inv_rms=torch.empty(wl.T, dtype=torch.float32, device=DEV))
    got = _outputs([prep(), prep.inv_rms])
    for a, b in zip(ref, got):
        assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))

    def clobber(r):
        prep.y.view(torch.uint8).fill_(0x7F)
        prep.inv_rms.fill_(float(r))
    ref_o = Q.qknorm_shard(data["xq"], data["gq"], wl.tp, rank, wl.eps, fmt=wl.dtype)

    def oracle_check(got):
        yb = bits_of(got[0])
        if wl.dtype == "fp8":
            compare.check_fp8(Q.decode_e4m3(yb), ref_o["y"], "graph apply y")
        else:
            compare.check_close(Q.decode_bf16(yb), ref_o["y"], compare.OUTPUT_RTOL, "graph apply y")
        compare.check_close(got[1].cpu().numpy(), ref_o["inv"], 1e-5, "graph apply inv")
    _check_replays(prep, [prep.y, prep.inv_rms], clobber, oracle_check)
