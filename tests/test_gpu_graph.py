"""GPU: the prepared entry points captured in a HIP graph (decode serving
loops replay them). Every replay must equal the eager result bit for bit; the
replays are separated by eager work that overwrites the outputs, so a replay
that wrote nothing, or wrote stale values, is caught. The library allocates
nothing and records no memset, so its launches are capturable as they are.

Not covered here: the Phase B wait entry points, whose round epoch is an
argument of the launch; a captured launch keeps its epoch, so a graph of
waiting launches can only be replayed if the slots are re-armed between
replays (see qkn.h).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workloads
from paper_2608_09160_amd import _lib as L

from gpu_util import DEV, inputs, peer_partials, to_dev_act, to_dev_bf16, to_dev_f32

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


def _check_replays(fn, outs, clobber):
    fn()
    ref = _outputs(outs)
    g = _graph_of(fn)
    for r in range(REPLAYS):
        clobber(r)                       # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        got = _outputs(outs)
        for a, b in zip(ref, got):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"replay {r}"


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
    _check_replays(prep, outs, clobber)


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
    _check_replays(prep, outs, clobber)
