#!/usr/bin/env python3
"""Benchmark of the fused sharded QK-Norm kernel on one MI355X.

Default workload: the prefill shard -- 8192 tokens, full Q/K widths 4096/1024
split over tp = 2, so this GPU (rank 0) holds Q 2048 / K 512 bf16 columns and
combines one simulated peer statistic per token and tensor. One step is one
launch of the fused kernel (Phases A, B and C for Q and K together).

Inputs are seeded synthetic data (package ``workloads``) resident in HBM. To
keep the timed launches honest about HBM -- MI355X has a 256 MB Infinity
Cache -- the benchmark rotates over enough independent buffer sets that each
launch reads data that no recent launch touched.

Prints ONE JSON line. ``value`` is whole-job throughput: algorithmic bytes of
the timed launches / wall time of the timed region (HIP events on the launch
stream). ``roofline.achieved`` divides the same bytes per launch by the mean
kernel duration, from events recorded around each launch. Side fields give
decode latencies, the full-vector (tp = 1) and two-launch baselines, a copy
kernel of the same byte count, and the fp64 oracle timed on host cores.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E peak


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default="prefill_T8192_q4096_k1024_tp2")
    p.add_argument("--rank", type=int, default=0)
    p.add_argument("--min-footprint-mb", type=int, default=1024,
                   help="total size of the rotating buffer sets")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extras", action="store_true",
                   help="only the headline workload (for profiler runs)")
    p.add_argument("--cpu-seconds", type=float, default=12.0)
    return p.parse_args()


def algorithmic_bytes(T, widths, tp, write_partials=True):
    """x read once + y written once (bf16) + gamma (fp32) once + own statistic
    written + the other ranks' statistics read (fp32), per launch."""
    b = 0
    for d in widths:
        b += 2 * T * d * 2 + 4 * d
        b += 4 * T * (tp - 1)
        if write_partials:
            b += 4 * T
    return b


class Case:
    """Rotating device buffer sets for one rank of one workload."""

    def __init__(self, wl, rank, min_footprint, torch, L, workloads, data=None, partials=True):
        self.wl, self.rank, self.torch, self.L = wl, rank, torch, L
        data = data if data is not None else workloads.generate(wl)
        dev = "cuda:0"
        tp, T = wl.tp, wl.T

        def bf16(a):
            a = np.ascontiguousarray(a, dtype=np.uint16)
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)

        shards = []
        for key, gkey, d_full in (("xq", "gq", wl.q_full), ("xk", "gk", wl.k_full)):
            cols = workloads.shard_cols(d_full, tp, rank)
            x = bf16(data[key][:, cols])
            w = torch.from_numpy(np.ascontiguousarray(data[gkey][cols])).to(dev)
            P = None
            if partials or tp > 1:
                P = torch.zeros((tp, T), dtype=torch.float32, device=dev)
                for k in range(tp):  # simulated peers (and the own slot, overwritten)
                    xk = x if k == rank else bf16(data[key][:, workloads.shard_cols(d_full, tp, k)])
                    L.qkn_partial_sumsq(xk, out=P[k])
            shards.append((x, w, P, d_full))
        set_bytes = sum(2 * x.numel() * 2 for x, _, _, _ in shards)
        self.nsets = max(2, -(-min_footprint // set_bytes))
        self.sets = []
        for i in range(self.nsets):
            segs = []
            for x, w, P, d_full in shards:
                segs.append(L.Seg(x=x.clone() if i else x, w=w, d_full=d_full,
                                  y=torch.empty_like(x),
                                  partials=(P.clone() if i else P) if P is not None else None))
            self.sets.append(segs)
        torch.cuda.synchronize()
        self.footprint = self.nsets * set_bytes
        self.bytes = algorithmic_bytes(T, (wl.q_local, wl.k_local), tp, write_partials=P is not None)

    def launch(self, i, fn="fused"):
        segs = self.sets[i % self.nsets]
        if fn == "fused":
            self.L.qkn_fused_shard(segs, self.wl.tp, self.rank, self.wl.eps)
        elif fn == "full":
            self.L.qkn_full(segs, self.wl.eps)
        elif fn == "two_step":
            for s in segs:
                self.L.qkn_partial_sumsq(s.x, out=s.partials[self.rank])
                self.L.qkn_apply(s.x, s.w, s.partials, s.d_full, self.wl.eps, y=s.y)
        else:
            raise ValueError(fn)


def time_launches(torch, fn, steps, warmup, per_launch=True):
    """Run `fn(i)` warmup + steps times on the current stream.

    Returns (region_ms, per_launch_ms list): the whole timed region between
    two events, and each launch's own duration between events recorded right
    before and after it (on the same stream)."""
    stream = torch.cuda.current_stream()
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)] if per_launch else []
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(steps):
        if per_launch:
            ev[i][0].record(stream)
        fn(warmup + i)
        if per_launch:
            ev[i][1].record(stream)
    end.record(stream)
    torch.cuda.synchronize()
    region = start.elapsed_time(end)
    each = [a.elapsed_time(b) for a, b in ev]
    return region, each


def cpu_baseline(wl, rank, data, seconds):
    """The fp64 oracle as it stands, on the host: bounded sample of the workload."""
    from oracle import qknorm as Q
    T = wl.T
    tokens = 0
    t0 = time.perf_counter()
    reps = 0
    while True:
        Q.qknorm_layerwise(data["xq"], data["xk"], data["gq"], data["gk"], wl.tp, rank, wl.eps)
        tokens += T
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    bytes_per_token = algorithmic_bytes(1, (wl.q_local, wl.k_local), wl.tp) - 4 * (wl.q_local + wl.k_local)
    gbs = bytes_per_token * tokens / el / 1e9
    try:
        ncpu = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        ncpu = os.cpu_count()
    return {"value": round(gbs, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{reps} full passes over the {T}-token workload (rank {rank}), "
                      f"{round(el, 2)} s of fp64 numpy on one thread",
            "host_cpus_visible": ncpu, "cpu_model": platform.processor() or platform.machine()}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU's share of the sharded QK-Norm; the peer ranks "
              "are simulated in device memory. Runs on more than one GPU are not supported: "
              "use --gpus 1.", file=sys.stderr)
        return 2
    os.environ.setdefault("OMP_NUM_THREADS", "1")
    import torch
    import workloads
    from paper_2608_09160_amd import _lib as L

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    L.load()
    wl = workloads.WORKLOADS[args.workload]
    data = workloads.generate(wl)
    min_fp = args.min_footprint_mb << 20

    print(f"[bench] {wl.name}: building rotating buffers", file=sys.stderr, flush=True)
    case = Case(wl, args.rank, min_fp, torch, L, workloads, data=data)
    case.launch(0)
    info = L.qkn_last_launch()
    region_ms, each = time_launches(torch, case.launch, args.steps, args.warmup)
    ms_per_step = region_ms / args.steps
    kernel_ms = float(np.mean(each))
    value = case.bytes / (ms_per_step * 1e-3) / 1e9
    achieved = case.bytes / (kernel_ms * 1e-3) / 1e9
    print(f"[bench] fused: {ms_per_step * 1e3:.2f} us/step, kernel {kernel_ms * 1e3:.2f} us "
          f"({achieved:.0f} GB/s)", file=sys.stderr, flush=True)

    extras = {}
    if not args.no_extras:
        # plain copy of the same number of bytes (x -> y of both tensors)
        src = [s.x for s in case.sets[0]]
        dst = [torch.empty_like(x) for x in src]
        copy_bytes = sum(2 * x.numel() * 2 for x in src)
        csets = [([s.x for s in segs], [s.y for s in segs]) for segs in case.sets]

        def copy(i):
            xs, ys = csets[i % len(csets)]
            for a, b in zip(xs, ys):
                b.copy_(a)
        r, e = time_launches(torch, copy, args.steps, args.warmup)
        extras["copy_same_bytes"] = {"bytes": copy_bytes, "kernel_us": round(np.mean(e) * 1e3 / 2, 3),
                                     "gbs_per_step": round(copy_bytes / (r / args.steps * 1e-3) / 1e9, 1)}
        del src, dst
        # two launches per tensor: Phase A, then Phases B+C (x read twice)
        r, e = time_launches(torch, lambda i: case.launch(i, "two_step"), args.steps, args.warmup)
        two_bytes = case.bytes + sum(2 * s.x.numel() for s in case.sets[0])
        extras["two_step_same_workload"] = {"us_per_step": round(r / args.steps * 1e3, 3),
                                            "gbs": round(two_bytes / (r / args.steps * 1e-3) / 1e9, 1),
                                            "bytes": two_bytes}
        # full-vector (tp = 1) baseline on the same tokens
        full_wl = wl.with_tp(1)
        fcase = Case(full_wl, 0, min_fp, torch, L, workloads, data=data, partials=False)
        r, e = time_launches(torch, lambda i: fcase.launch(i, "full"), args.steps, args.warmup)
        fk = float(np.mean(e))
        extras["full_vector_tp1"] = {"kernel": L.qkn_last_launch()["kernel"], "bytes": fcase.bytes,
                                     "kernel_us": round(fk * 1e3, 3),
                                     "gbs": round(fcase.bytes / (fk * 1e-3) / 1e9, 1)}
        del fcase
        # decode shapes: latency of one launch, warm (inputs just produced, cache
        # resident) and cold (rotating sets)
        lat = {}
        for name in ("decode_T64_q4096_k1024_tp4", "decode_T256_q5120_k1024_tp8",
                     "tiny_full_T16_q512_k128_tp1"):
            dwl = workloads.WORKLOADS[name]
            dcase = Case(dwl, 0, 0, torch, L, workloads, partials=dwl.tp > 1)
            fn = (lambda i, c=dcase: c.launch(i, "full")) if dwl.tp == 1 else dcase.launch
            r, e = time_launches(torch, lambda i, f=fn: f(0), 2000, 100)
            lat[name] = {"us_median": round(float(np.median(e)) * 1e3, 3),
                         "us_p10": round(float(np.percentile(e, 10)) * 1e3, 3),
                         "us_p90": round(float(np.percentile(e, 90)) * 1e3, 3),
                         "kernel": L.qkn_last_launch()["kernel"],
                         "grid": L.qkn_last_launch()["grid"]}
            del dcase
        extras["decode_latency_warm"] = lat
        # long prefill shard
        lwl = workloads.LONG_PREFILL_TP4
        lcase = Case(lwl, 0, min_fp, torch, L, workloads)
        r, e = time_launches(torch, lcase.launch, max(20, args.steps // 4), 5)
        lk = float(np.mean(e))
        extras["long_prefill_tp4"] = {"kernel": L.qkn_last_launch()["kernel"], "bytes": lcase.bytes,
                                      "kernel_us": round(lk * 1e3, 3),
                                      "gbs": round(lcase.bytes / (lk * 1e-3) / 1e9, 1)}
        del lcase
        print(f"[bench] extras done", file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        cpu = cpu_baseline(wl, args.rank, data, args.cpu_seconds)

    out = {
        "metric": "QK-Norm kernel latency (us, decode) and achieved HBM GB/s (prefill), 1 MI355X",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 in/out, fp32 accumulate",
        "data": "synthetic (seeded; package workloads)",
        "config": {"workload": wl.name, "tokens": wl.T, "tp": wl.tp, "rank": args.rank,
                   "q_local": wl.q_local, "k_local": wl.k_local, "bytes_per_step": case.bytes,
                   "rotating_sets": case.nsets, "footprint_mb": round(case.footprint / 2 ** 20),
                   "kernel": info["kernel"], "grid": info["grid"], "block": info["block"],
                   "parallelism": "1 GPU (peer ranks simulated)"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel_us": round(kernel_ms * 1e3, 3)},
        "cpu_baseline": cpu,
        "extras": extras,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
