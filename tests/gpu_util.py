"""Helpers for the GPU tests: move seeded inputs to the device, simulate peer
ranks, run one rank's fused kernel, and decode results for the oracle."""
from __future__ import annotations

import functools
import os
from concurrent.futures import ThreadPoolExecutor

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


# ------------------------------------------------------------------ oracle over every token
#
# The fp64 oracle (Eq. 1 on the full row, sliced; per-rank statistics as
# defined) in blocks of tokens, so that a check of every token of a full-size
# workload keeps host memory bounded. Blocks are independent (every token is
# normalised on its own), so they run on a few host threads (numpy releases
# the interpreter lock in its array operations): the whole 32768-token shard
# takes seconds instead of half a minute.

ORACLE_BLOCK = 2048
ORACLE_THREADS = max(1, min(8, len(os.sched_getaffinity(0))))


def _oracle_block(wl: workloads.Workload, data, sel):
    from oracle import qknorm as Q
    ref = {}
    for t, key, gkey in (("q", "xq", "gq"), ("k", "xk", "gk")):
        x = data[key][sel]
        full = Q.qknorm_shard(x, data[gkey], 1, 0, wl.eps, fmt=wl.dtype)
        ref[t] = {"y": full["y"], "inv": full["inv"],
                  "partials": Q.shard_partials(Q.decode(x, wl.dtype), wl.tp)}
    return ref


def for_each_oracle_block(wl: workloads.Workload, data, fn, rows=None,
                          block: int = ORACLE_BLOCK) -> None:
    """Calls fn(sel, ref) for blocks of tokens: `sel` the token indices of the
    block, ref[t] for t in "qk" the oracle's full-width output "y" [n, d_full],
    factor "inv" [n] and every rank's statistic "partials" [tp, n], all fp64.
    `rows`: the tokens to cover (default every token). An assertion raised by
    fn in any block is raised here."""
    rows = np.arange(wl.T) if rows is None else np.asarray(rows)
    starts = range(0, len(rows), block)

    def work(b0):
        sel = rows[b0:b0 + block]
        fn(sel, _oracle_block(wl, data, sel))

    with ThreadPoolExecutor(ORACLE_THREADS) as ex:
        for _ in ex.map(work, starts):
            pass


def check_y(got_bits: np.ndarray, ref_y: np.ndarray, fmt: str, what: str) -> float:
    """Outputs against the oracle: bf16 within the relative tolerance, FP8 as
    the round-to-nearest-even code of a value within the noise band. Returns
    the largest relative error (bf16) or error in half FP8 steps (FP8)."""
    from oracle import compare
    from oracle import qknorm as Q
    if fmt == "fp8":
        return compare.check_fp8(Q.decode_e4m3(got_bits), ref_y, what)
    return compare.check_close(Q.decode_bf16(got_bits), ref_y, compare.OUTPUT_RTOL, what)


def check_rank_every_token(wl: workloads.Workload, data, rank: int, out, what: str,
                           rows=None) -> None:
    """Rank `rank`'s results (as run_fused_rank returns them: per tensor its
    y slice [T, d_local], partials [tp, T] with the own row written, inv [T])
    against the oracle, element by element on every token (or on `rows`):
    y as check_y, the own statistic within 1e-5 relative, the factor within
    1e-5 relative. A tensor's "partials" or "inv" set to None is not checked."""
    check_ranks_every_token(wl, data, {rank: out}, what, rows)


def check_ranks_every_token(wl: workloads.Workload, data, outs, what: str, rows=None) -> None:
    """check_rank_every_token for several ranks' results ({rank: out}) with
    one pass of the oracle."""
    from oracle import compare
    worst = {"y": [0.0], "statistic": [0.0], "inv": [0.0]}

    def fn(sel, ref):
        for rank, out in outs.items():
            for t, d_full in (("q", wl.q_full), ("k", wl.k_full)):
                cols = workloads.shard_cols(d_full, wl.tp, rank)
                o = out[t]
                worst["y"].append(check_y(o["y"][sel], ref[t]["y"][:, cols], wl.dtype,
                                          f"{what} {t} y r{rank}"))
                if o.get("partials") is not None:
                    worst["statistic"].append(compare.check_close(
                        o["partials"][rank][sel], ref[t]["partials"][rank],
                        compare.PARTIAL_RTOL, f"{what} {t} own statistic r{rank}"))
                if o.get("inv") is not None:
                    worst["inv"].append(compare.check_close(o["inv"][sel], ref[t]["inv"], 1e-5,
                                                            f"{what} {t} inv r{rank}"))

    for_each_oracle_block(wl, data, fn, rows)
    unit = "half FP8 steps" if wl.dtype == "fp8" else "relative"
    print(f"[errors] {what}: ranks {sorted(outs)}, max y error {max(worst['y']):.3e} ({unit}), "
          f"max statistic rel error {max(worst['statistic']):.3e}, max factor rel error "
          f"{max(worst['inv']):.3e}", flush=True)


def slot_values(slots: np.ndarray, epoch: int) -> np.ndarray:
    """Published flagged slots (int64 words) -> their fp32 statistics; every
    word must carry `epoch` in its high half."""
    w = np.ascontiguousarray(slots).view(np.uint64)
    assert np.all((w >> np.uint64(32)) == np.uint64(epoch)), "a slot without the round's epoch"
    return (w & np.uint64(0xFFFFFFFF)).astype(np.uint32).view(np.float32)


def check_group_every_token(wl: workloads.Workload, data, y_bits, inv, slots, epoch: int,
                            what: str) -> None:
    """A whole tp group's results (one launch over the full tensors) against
    the oracle on every token and every rank: per tensor y [T, d_full] (the
    unsharded norm, each rank's columns written by that rank), inv [tp, T]
    (each rank's factor) and the published slots [tp, T] (each rank's
    statistic, with the round's epoch)."""
    from oracle import compare
    vals = {t: slot_values(slots[t], epoch) for t in "qk"}

    def fn(sel, ref):
        for t, d_full in (("q", wl.q_full), ("k", wl.k_full)):
            for r in range(wl.tp):
                cols = workloads.shard_cols(d_full, wl.tp, r)
                check_y(y_bits[t][sel][:, cols], ref[t]["y"][:, cols], wl.dtype,
                        f"{what} {t} y r{r}")
                compare.check_close(inv[t][r][sel], ref[t]["inv"], 1e-5, f"{what} {t} inv r{r}")
                compare.check_close(vals[t][r][sel], ref[t]["partials"][r],
                                    compare.PARTIAL_RTOL, f"{what} {t} statistic r{r}")

    for_each_oracle_block(wl, data, fn)
