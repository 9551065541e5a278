"""Helpers for the GPU tests: move seeded inputs to the device, simulate peer
ranks, run one rank's fused kernel, and decode results for the oracle."""
from __future__ import annotations

import functools

import numpy as np
import torch

import workloads
from paper_2608_09160_amd import _lib as L

DEV = "cuda:0"


def to_dev_bf16(bits: np.ndarray) -> torch.Tensor:
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(DEV)


def to_dev_fp8(bits: np.ndarray) -> torch.Tensor:
    bits = np.ascontiguousarray(bits, dtype=np.uint8)
    return torch.from_numpy(bits).view(torch.float8_e4m3fn).to(DEV)


def to_dev_act(bits: np.ndarray) -> torch.Tensor:
    """Activation bits to the device: uint8 -> float8_e4m3fn, uint16 -> bfloat16."""
    return to_dev_fp8(bits) if np.asarray(bits).dtype == np.uint8 else to_dev_bf16(bits)


def to_dev_f32(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def bits_of(t: torch.Tensor) -> np.ndarray:
    """Activation GPU tensor -> bits on the host (uint16 for bf16, uint8 for fp8)."""
    if t.element_size() == 1:
        return t.contiguous().view(torch.uint8).cpu().numpy()
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def partial_fn(bits: np.ndarray):
    return L.qkn_partial_sumsq_fp8 if np.asarray(bits).dtype == np.uint8 else L.qkn_partial_sumsq


@functools.lru_cache(maxsize=4)
def inputs(wl: workloads.Workload):
    return workloads.generate(wl)


def shard(data, key, d_full, tp, r):
    return data[key][:, workloads.shard_cols(d_full, tp, r)]


def peer_partials(data, key, d_full, tp, T, rank, fill_own=np.nan):
    """fp32 [tp, T] on the GPU: slots of every rank but `rank` computed by
    qkn_partial_sumsq on that rank's slice (the simulated peers); the own slot
    is filled with `fill_own` so that a kernel reading it would be caught."""
    P = torch.full((tp, T), fill_own, dtype=torch.float32, device=DEV)
    for k in range(tp):
        if k == rank:
            continue
        xs = shard(data, key, d_full, tp, k)
        partial_fn(xs)(to_dev_act(xs), out=P[k])
    return P


def run_fused_rank(wl: workloads.Workload, data, rank: int, eps=None):
    """One rank's fused QK-Norm with simulated peers. Returns host results."""
    eps = wl.eps if eps is None else eps
    tp, T = wl.tp, wl.T
    segs = []
    for key, gkey, d_full in (("xq", "gq", wl.q_full), ("xk", "gk", wl.k_full)):
        cols = workloads.shard_cols(d_full, tp, rank)
        segs.append(L.Seg(x=to_dev_act(data[key][:, cols]), w=to_dev_f32(data[gkey][cols]),
                          d_full=d_full,
                          partials=peer_partials(data, key, d_full, tp, T, rank)
                          if tp > 1 else torch.empty((1, T), dtype=torch.float32, device=DEV),
                          inv_rms=torch.empty(T, dtype=torch.float32, device=DEV)))
    (L.qkn_fused_shard_fp8 if wl.dtype == "fp8" else L.qkn_fused_shard)(segs, tp, rank, eps)
    info = L.qkn_last_launch()
    torch.cuda.synchronize()
    out = {}
    for name, s in zip("qk", segs):
        out[name] = {"y": bits_of(s.y), "partials": s.partials.cpu().numpy(),
                     "inv": s.inv_rms.cpu().numpy()}
    out["launch"] = info
    return out
