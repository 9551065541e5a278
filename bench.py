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

if __name__ == "__main__":
    # the oracle's CPU baseline runs on one host thread: pin the thread pools
    # of numpy's libraries before numpy is imported
    for _var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[_var] = "1"

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
    p.add_argument("--summarize", metavar="DIR",
                   help="write the profiles/ summaries from rocprofv3 CSV output in DIR and exit")
    p.add_argument("--proj-only", action="store_true",
                   help="run only the projection extra (Q/K projection with Phase A in its "
                        "epilogue, and torch.mm of the same product) and print its JSON; "
                        "the command profiled for profiles/counters_proj_*.txt")
    p.add_argument("--summarize-proj", metavar="DIR",
                   help="write profiles/counters_proj_*.txt from rocprofv3 --pmc CSV output of "
                        "`bench.py --proj-only` in DIR/pmc_proj1 and DIR/pmc_proj2")
    p.add_argument("--counter-pass", action="store_true",
                   help="launch every kernel family measured in profiles/ (the headline, the "
                        "two-launch baseline, the group wait, tp = 1, the long shard, FP8, the "
                        "projection) a fixed number of times between marker launches and print "
                        "their list as JSON: the program that the rocprofv3 --pmc passes of "
                        "--summarize-counters profile")
    p.add_argument("--summarize-counters", metavar="DIR",
                   help="write profiles/counters_*.txt and profiles/issue_rate_*.md from the "
                        "rocprofv3 --pmc output of `bench.py --counter-pass` in DIR/<pass> "
                        "(one directory per entry of COUNTER_PASSES) and DIR/counter_pass.json")
    p.add_argument("--calibration-copy", action="store_true",
                   help="also run a plain device copy of Q's input (known bytes) a few times, "
                        "to scale profiler byte counters")
    return p.parse_args()


def algorithmic_bytes(T, widths, tp, write_partials=True, esz=2):
    """x read once + y written once (esz bytes per element: bf16 2, fp8 1) +
    gamma (fp32) once + own statistic written + the other ranks' statistics
    read (fp32), per launch."""
    b = 0
    for d in widths:
        b += 2 * T * d * esz + 4 * d
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
        self.fp8 = wl.dtype == "fp8"
        self.esz = 1 if self.fp8 else 2
        self.partial_fn = L.qkn_partial_sumsq_fp8 if self.fp8 else L.qkn_partial_sumsq
        self.apply_fn = L.qkn_apply_fp8 if self.fp8 else L.qkn_apply

        def bf16(a):
            if self.fp8:  # FP8 codes as uint8 device tensors (the binding takes either dtype)
                return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).to(dev)
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
                    self.partial_fn(xk, out=P[k])
            shards.append((x, w, P, d_full))
        set_bytes = sum(2 * x.numel() * self.esz for x, _, _, _ in shards)
        self.nsets = max(2, -(-min_footprint // set_bytes))
        self.sets = []
        for i in range(self.nsets):
            segs = []
            for x, w, P, d_full in shards:
                segs.append(L.Seg(x=x.clone() if i else x, w=w, d_full=d_full,
                                  y=torch.empty_like(x),
                                  partials=(P.clone() if i else P) if P is not None else None))
            self.sets.append(segs)
        full = tp == 1 and not partials
        self.calls = [L.Prepared(segs, tp, rank, wl.eps, full=full) for segs in self.sets]
        torch.cuda.synchronize()
        self.footprint = self.nsets * set_bytes
        self.bytes = algorithmic_bytes(T, (wl.q_local, wl.k_local), tp, write_partials=P is not None,
                                       esz=self.esz)

    def launch(self, i):
        self.calls[i % self.nsets]()

    def launch_two_step(self, i):
        """Phase A, then Phases B+C, per tensor: the unfused scalar-statistic path."""
        for s in self.sets[i % self.nsets]:
            self.partial_fn(s.x, out=s.partials[self.rank])
            self.apply_fn(s.x, s.w, s.partials, s.d_full, self.wl.eps, y=s.y)


class GroupCase:
    """Every rank of a tp group in one launch (qkn_fused_group_wait) over the full
    Q/K tensors, rotating buffer sets; each launch is one round (new epoch)."""

    def __init__(self, wl, min_footprint, torch, L, data):
        self.wl, self.torch, self.L = wl, torch, L
        dev = "cuda:0"

        fp8 = wl.dtype == "fp8"
        esz = 1 if fp8 else 2

        def bf16(a):
            if fp8:  # FP8 codes as uint8 device tensors (the binding takes either dtype)
                return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).to(dev)
            a = np.ascontiguousarray(a, dtype=np.uint16)
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        xs = [bf16(data["xq"]), bf16(data["xk"])]
        ws = [torch.from_numpy(data["gq"]).to(dev), torch.from_numpy(data["gk"]).to(dev)]
        set_bytes = sum(2 * x.numel() * esz for x in xs)
        self.nsets = max(2, -(-min_footprint // set_bytes))
        self.sets = []
        for i in range(self.nsets):
            segs = [L.Seg(x=x.clone() if i else x, w=w, d_full=x.shape[1], y=torch.empty_like(x))
                    for x, w in zip(xs, ws)]
            slots = [torch.zeros((wl.tp, wl.T), dtype=torch.int64, device=dev) for _ in range(2)]
            self.sets.append((segs, slots))
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.epoch = 0
        T, tp = wl.T, wl.tp
        # x read + y written, gamma, per rank: own slot written, tp - 1 slots read (8 B each)
        self.bytes = sum(2 * T * d * esz + 4 * d + 8 * T * tp * tp for d in (wl.q_full, wl.k_full))
        torch.cuda.synchronize()

    def launch(self, i):
        segs, slots = self.sets[i % self.nsets]
        self.epoch += 1
        self.L.qkn_fused_group_wait(segs, self.wl.tp, self.wl.eps, slots, epoch=self.epoch,
                                    spin_limit=1 << 22, status=self.status)


def time_region(torch, fn, steps, warmup):
    """Wall time (ms) of `steps` back-to-back calls between two events on the stream."""
    stream = torch.cuda.current_stream()
    for i in range(warmup):
        fn(i)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(steps):
        fn(warmup + i)
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end)


def time_each(torch, fn, steps, warmup):
    """Per-call durations (ms) from events recorded right before and after each call."""
    stream = torch.cuda.current_stream()
    for i in range(warmup):
        fn(i)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    torch.cuda.synchronize()
    for i in range(steps):
        ev[i][0].record(stream)
        fn(warmup + i)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in ev]


def time_cold(torch, fn, steps, flush):
    """Per-call durations (ms) from events right around each call, every call
    preceded (outside the events) by `flush()`, which evicts the caches."""
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    torch.cuda.synchronize()
    for i in range(steps):
        flush()
        ev[i][0].record(stream)
        fn(i)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in ev]


def time_launches(torch, fn, steps, warmup):
    """(region ms, per-call ms list) -- per-call events inside one timed region."""
    stream = torch.cuda.current_stream()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    start.record(stream)
    for i in range(steps):
        ev[i][0].record(stream)
        fn(warmup + i)
        ev[i][1].record(stream)
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end), [a.elapsed_time(b) for a, b in ev]


def stream_copy_ms(torch, L, nbytes: int, min_footprint: int, steps: int, warmup: int,
                   grids=(2048, 4096, 8192, 16384)):
    """Best time (ms) per launch of the streaming copy (qkn_calib_copy) of
    `nbytes` bytes in total (half read, half written) over rotating buffer sets
    of at least `min_footprint` bytes, and its grid: the practical ceiling of a
    read-once/write-once kernel moving the same bytes."""
    half = nbytes // 2 // 16 * 16
    nbuf = max(2, -(-min_footprint // (2 * half)))
    bufs = [(torch.empty(half, dtype=torch.uint8, device="cuda:0"),
             torch.empty(half, dtype=torch.uint8, device="cuda:0")) for _ in range(nbuf)]
    best = None
    for blocks in grids:
        r = time_region(torch, lambda i, b=blocks: L.qkn_calib_copy(*bufs[i % nbuf], blocks=b),
                        steps, warmup) / steps
        if best is None or r < best[0]:
            best = (r, blocks)
    del bufs
    torch.cuda.synchronize()
    return best


def token_fit(torch, L, min_fp: int, steps: int, warmup: int,
              tokens=(2048, 4096, 8192, 16384, 32768), widths=(2048, 512), tp=2, fp8=False):
    """Launch time of the fused kernel against the token count at the prefill
    shard's widths (Q 2048 + K 512 per rank, tp 2), cold (rotating buffer sets
    of >= min_fp bytes, device-random bf16 rows, or FP8-E4M3 rows with
    fp8=True), and a least-squares line time = intercept + slope * T; the same
    for the streaming copy of the same bytes. The intercept is the fixed cost
    per launch, the slope the streaming rate."""
    dev = "cuda:0"
    esz = 1 if fp8 else 2
    pts, cps = [], []
    for T in tokens:
        set_bytes = sum(2 * T * d * esz for d in widths)  # x read + y written
        nsets = max(2, -(-min_fp // set_bytes))
        calls = []
        for _ in range(nsets):
            segs = []
            for d in widths:
                if fp8:  # finite E4M3 codes (0x7F / 0xFF, the NaNs, left out) as uint8
                    x = (torch.randint(0, 0x7F, (T, d), device=dev, dtype=torch.uint8) |
                         (torch.randint(0, 2, (T, d), device=dev, dtype=torch.uint8) << 7))
                else:
                    x = torch.randn((T, d), device=dev).to(torch.bfloat16)
                P = torch.rand((tp, T), device=dev) + 0.5
                segs.append(L.Seg(x=x, w=torch.rand(d, device=dev) + 0.5, d_full=d * tp,
                                  y=torch.empty_like(x), partials=P))
            calls.append(L.Prepared(segs, tp, 0, 1e-6))
        torch.cuda.synchronize()
        ms = time_region(torch, lambda i: calls[i % nsets](), steps, warmup) / steps
        pts.append((T, ms * 1e3))
        del calls
        torch.cuda.synchronize()
        cms, _ = stream_copy_ms(torch, L, set_bytes, min_fp, steps, warmup, grids=(8192,))
        cps.append((T, cms * 1e3))
    out = {"widths": list(widths), "tp": tp, "dtype": "fp8" if fp8 else "bf16",
           "bytes_per_token": algorithmic_bytes(1, widths, tp, esz=esz) - 4 * sum(widths)}
    for key, data in (("fused", pts), ("copy", cps)):
        t = np.array([p[0] for p in data], dtype=np.float64)
        us = np.array([p[1] for p in data], dtype=np.float64)
        slope, icpt = np.polyfit(t, us, 1)
        out[key] = {"us": {int(a): round(b, 3) for a, b in data}, "intercept_us": round(icpt, 3),
                    "slope_ns_per_token": round(slope * 1e3, 4),
                    "streaming_gbs": round(out["bytes_per_token"] / (slope * 1e-6) / 1e9, 1)}
    return out


def time_graph(torch, fn, per_graph, replays):
    """Mean time (ms) per call when `per_graph` calls are replayed from one HIP graph."""
    fn(0)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            for i in range(per_graph):
                fn(i)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    stream = torch.cuda.current_stream()
    start.record(stream)
    for _ in range(replays):
        g.replay()
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / (per_graph * replays)


ROOT = os.path.dirname(os.path.abspath(__file__))
# the row kernels' templates, their instantiation tables and the host code
# that picks and launches them: counters taken before a change to any of these
# no longer describe the kernel
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_09160_amd", "csrc", f)
                  for f in ("qkn_kernels.h", "qkn_kern_rows.hip", "qkn_kern_wait.hip",
                            "qkn_kern_wait8.hip", "qkn_kern_misc.hip", "qkn.hip")]


def source_sha256() -> str:
    import hashlib
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def counters_path(kernel: str, workload: str) -> str:
    tag = kernel.replace("<", "_").replace(">", "").replace(",", "_").replace("/", "_")
    return os.path.join(ROOT, "profiles", f"counters_{tag}_{workload}.txt")


def traffic_bytes(kernel: str, workload: str):
    """HBM bytes per launch from the committed counter summary, or None when
    there is none or the kernel source changed since the counters were taken."""
    path = counters_path(kernel, workload)
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line:
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_sha256") != source_sha256():
        return None
    try:
        return int(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def trace_name(launch_name: str) -> str:
    """Profiler (demangled) name of the kernel a launch name denotes, e.g.
    "rows<4,1>/fused" -> "void qkn_rows<FmtBf16, 4, 1, 0, 0>"."""
    import re
    m = re.fullmatch(r"(rows|wide)(_pf|_pa|_pa2|_pa3)?(_fp8)?<(\d+),(\d+)>/"
                     r"(fused|apply|partial|fused_wait|publish)", launch_name)
    if not m or (m.group(1) == "wide" and m.group(2)):
        raise ValueError(f"no profiler name for {launch_name!r}")
    fam, sched_tag, fp8, n0, n1, mode = m.groups()
    fmt = "FmtFp8" if fp8 else "FmtBf16"
    mode_id = ["fused", "apply", "partial", "fused_wait", "publish"].index(mode)
    if fam == "wide":
        return f"void qkn_wide<{fmt}, {n0}, {n1}, {mode_id}>"
    sched = {None: 0, "_pf": 1, "_pa": 2, "_pa2": 3, "_pa3": 4}[sched_tag]
    return f"void qkn_rows<{fmt}, {n0}, {n1}, {mode_id}, {sched}>"


def kernel_base_name(profiler_name: str) -> str:
    """Profiler name without namespaces and parameter list, e.g.
    "void qkn_dev::qkn_rows<qkn_dev::FmtBf16, 4, 1, 0, 0>(qkn_dev::KParams)"
    -> "void qkn_rows<FmtBf16, 4, 1, 0, 0>"."""
    return (profiler_name.replace("(anonymous namespace)::", "").replace("qkn_dev::", "")
            .split("(")[0])


def summarize(outdir: str) -> None:
    """Write the kernel-trace summary of the headline kernel into profiles/
    from rocprofv3 CSV output in `outdir`: trace/*_kernel_trace.csv and
    trace_bench.json (the kernel trace of the default bench run and that run's
    JSON line), next to bench.json (an untraced run of the same session), if
    present. (The counter summaries come from --summarize-counters.)"""
    import csv
    import glob
    import statistics
    bench = json.loads(open(os.path.join(outdir, "trace_bench.json")).read().strip().splitlines()[-1])
    kernel, workload = bench["config"]["kernel"], bench["config"]["workload"]
    algo = bench["roofline"]["algorithmic_bytes"]
    tname = trace_name(kernel)
    grid_threads = bench["config"]["grid"] * bench["config"]["block"]

    trace = glob.glob(os.path.join(outdir, "trace", "*_kernel_trace.csv"))[0]
    rows = sorted(csv.DictReader(open(trace)), key=lambda r: int(r["Start_Timestamp"]))
    runs = []  # consecutive dispatches of one kernel and launch shape
    for r in rows:
        name = kernel_base_name(r["Kernel_Name"])
        key = (name, int(r["Grid_Size_X"]), int(r["Workgroup_Size_X"]))
        d = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        if runs and runs[-1][0] == key:
            runs[-1][1].append(d)
        else:
            runs.append([key, [d]])
    head = ["| kernel | grid (threads) | workgroup | dispatches | mean us | median us | min us | max us |",
            "|---|---|---|---|---|---|---|---|"]

    def row(name, g, w, ds):
        sd = sorted(ds)
        return (f"| {name} | {g} | {w} | {len(ds)} | {statistics.mean(ds) / 1e3:.3f} | "
                f"{sd[len(sd) // 2] / 1e3:.3f} | {sd[0] / 1e3:.3f} | {sd[-1] / 1e3:.3f} |")
    headline = next(ds for (n, g, _), ds in runs if n == tname and g == grid_threads and len(ds) >= 20)
    mean_us = statistics.mean(headline) / 1e3
    total = {}
    for k, ds in runs:
        total.setdefault(k, []).extend(ds)
    sha = source_sha256()
    tag = os.path.basename(counters_path(kernel, workload))[len("counters_"):-len(".txt")]
    plain = []  # the untraced bench.py run of the same session, if there is one
    if os.path.exists(os.path.join(outdir, "bench.json")):
        pb = json.loads(open(os.path.join(outdir, "bench.json")).read().strip().splitlines()[-1])
        if pb["config"]["kernel"] == kernel:
            k_us = pb["roofline"]["kernel_us"]
            plain = [f"The untraced `python bench.py` run of the same session: kernel_us {k_us} "
                     f"(timed region / launches), {abs(k_us - mean_us) / mean_us:.1%} from the "
                     f"trace's mean; value {pb['value']} GB/s, roofline.frac {pb['roofline']['frac']}."]
    cmd_trace = ("rocprofv3 --kernel-trace --stats --output-format csv -d gpurun_out/trace -o bench "
                 "-- python -u bench.py --no-cpu-baseline > gpurun_out/trace_bench.json")
    lines = [f"# Kernel trace: {kernel} on {workload}", "",
             f"Kernel source sha256 {sha}. Commands (MI355X, repository root):", "",
             f"    {cmd_trace}", "    python bench.py --summarize gpurun_out", "",
             f"Headline kernel `{tname}` (launch name `{kernel}`), the run of {len(headline)} "
             f"consecutive dispatches of the bench's timed and per-launch passes: mean "
             f"{mean_us:.3f} us -> {algo} algorithmic bytes / {mean_us:.3f} us = "
             f"{algo / (mean_us * 1e-6) / 1e9:.0f} GB/s = {algo / (mean_us * 1e-6) / 1e9 / HBM_PEAK_GBS:.1%} "
             f"of 8 TB/s. The traced bench.py line (tracing adds gaps between launches): kernel_us "
             f"{bench['roofline']['kernel_us']} (timed region / launches)."] + plain + [
             "", "Kernel names: `qkn_rows<Fmt, N0, N1, MODE, SCHED>` / `qkn_wide<Fmt, N0, N1, MODE>`, "
             "N0/N1 = 16-byte chunks per lane of the two tensors, MODE 0 fused, 1 apply (Phases B+C), "
             "2 Phase A, 3 fused with wait, 4 publish; SCHED 1 = pipelined.", "",
             "Runs of at least 20 consecutive dispatches of one kernel and shape, in order:", ""]
    lines += head + [row(*k, ds) for k, ds in runs if len(ds) >= 20]
    lines += ["", "All dispatches per kernel and shape:", ""]
    lines += head + [row(*k, ds) for k, ds in sorted(total.items(), key=lambda kv: -sum(kv[1]))]
    with open(os.path.join(ROOT, "profiles", f"trace_{tag}.md"), "w") as f:
        f.write("\n".join(lines) + "\n")

    print(f"trace: headline mean {mean_us:.3f} us over {len(headline)} dispatches; "
          f"bench kernel_us {bench['roofline']['kernel_us']}")


# rocprofv3 --pmc passes over `bench.py --counter-pass` (each within the
# per-block counter limits of one pass): HBM bytes, and the instruction-issue
# counters behind the issue-rate comparison of fused and unfused kernels
COUNTER_PASSES = (
    ("pmc_fetch", "FETCH_SIZE"),
    ("pmc_write", "WRITE_SIZE"),
    ("pmc_issue", "SQ_WAVES SQ_BUSY_CYCLES SQ_WAVE_CYCLES SQ_WAIT_ANY SQ_INSTS_VALU SQ_INSTS_SALU "
                  "SQ_INSTS_VMEM_RD SQ_INSTS_VMEM_WR"),
    ("pmc_issue2", "GRBM_GUI_ACTIVE SQ_INSTS_SMEM SQ_WAIT_INST_ANY SQ_ACTIVE_INST_ANY"),
)
COUNTER_STEPS = 20
MARKER_KERNEL = "qkn_calib_empty_kernel"
PROJ_SOURCES = [os.path.join(ROOT, "paper_2608_09160_amd", "csrc", "qkn_proj.hip")]


def proj_sha256() -> str:
    import hashlib
    h = hashlib.sha256()
    for path in PROJ_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def counter_pass(torch, L, workloads, min_fp: int) -> list:
    """Each case: a few untimed launches, then a marker launch (the empty
    calibration kernel), COUNTER_STEPS steps and another marker. Returns the case list
    (tag, workload, algorithmic bytes per step, launch names of one step)."""
    dev = "cuda:0"
    cases = []

    def run(tag, wl_name, nbytes, step, note="", launches=None):
        for i in range(2):
            step(i)
        torch.cuda.synchronize()
        names = []
        L.qkn_calib_empty()  # start marker
        for i in range(COUNTER_STEPS):
            step(2 + i)
            if i == 0:
                names.append(L.qkn_last_launch()["kernel"] if launches is None else launches)
        L.qkn_calib_empty()  # end marker
        torch.cuda.synchronize()
        cases.append({"tag": tag, "workload": wl_name, "bytes_per_step": nbytes, "note": note,
                      "launch_names": names})
        print(f"[counters] {tag} on {wl_name}", file=sys.stderr, flush=True)

    # calibration: a plain device copy of known bytes
    a = torch.empty(32 << 20, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    run("calibration_copy", "device copy of 32 MiB", 2 * a.numel(), lambda i: b.copy_(a),
        launches="torch copy_")
    del a, b
    c4 = workloads.PREFILL_TP2
    data = workloads.generate(c4)
    case = Case(c4, 0, min_fp, torch, L, workloads, data=data)
    run("fused", c4.name, case.bytes, case.launch)
    two_bytes = case.bytes + sum(2 * s.x.numel() for s in case.sets[0])
    run("two_step", c4.name, two_bytes, case.launch_two_step,
        "Phase A per tensor, then Phases B+C per tensor: four launches per step",
        launches="qkn_partial_sumsq Q, K; qkn_apply Q, K")
    del case
    g = GroupCase(c4, min_fp, torch, L, data)
    run("group_wait", c4.name, g.bytes, g.launch, "every rank of the tp = 2 group in one launch")
    del g
    full = Case(c4.with_tp(1), 0, min_fp, torch, L, workloads, data=data, partials=False)
    run("fused", c4.with_tp(1).name, full.bytes, full.launch, "tp = 1 full-vector baseline")
    del full, data
    c5 = workloads.LONG_PREFILL_TP4
    long = Case(c5, 0, min_fp, torch, L, workloads)
    run("fused", c5.name, long.bytes, long.launch)
    del long
    f8 = c4.with_dtype("fp8")
    data8 = workloads.generate(f8)
    p8 = Case(f8, 0, min_fp, torch, L, workloads, data=data8)
    run("fused", f8.name, p8.bytes, p8.launch)
    del p8
    g8 = GroupCase(f8, min_fp, torch, L, data8)
    run("group_wait", f8.name, g8.bytes, g8.launch, "every rank of the tp = 2 group in one launch")
    del g8, data8
    # the decode-sized projection (warm: the same buffers every call, as in its timing)
    dwl = workloads.DECODE_TP4
    pdata = workloads.projection_inputs(dwl)

    def bf16(arr):
        arr = np.ascontiguousarray(arr, dtype=np.uint16)
        return torch.from_numpy(arr.view(np.int16)).view(torch.bfloat16).to(dev)
    x = bf16(pdata["x"])
    wq = bf16(pdata["wq"][workloads.shard_cols(dwl.q_full, dwl.tp, 1)])
    wk = bf16(pdata["wk"][workloads.shard_cols(dwl.k_full, dwl.tp, 1)])
    prep = L.PreparedProj(x, [L.ProjSeg(w=wq), L.ProjSeg(w=wk)])
    cols, hidden = wq.shape[0] + wk.shape[0], x.shape[1]
    run("proj", dwl.name, 2 * (cols * hidden + dwl.T * hidden + dwl.T * cols), lambda i: prep(),
        "split-k projection and its reduction: two launches per call; weights warm")
    torch.cuda.synchronize()
    return cases


def _counter_rows(path: str):
    """{(dispatch id, kernel base name): {counter: value}} from one --pmc CSV, in dispatch order."""
    import csv
    import glob
    f = glob.glob(os.path.join(path, "*_counter_collection.csv"))[0]
    by = {}
    for r in csv.DictReader(open(f)):
        key = (int(r["Dispatch_Id"]), kernel_base_name(r["Kernel_Name"]))
        by.setdefault(key, {})[r["Counter_Name"]] = by.get(key, {}).get(r["Counter_Name"], 0.0) + \
            float(r["Counter_Value"])
    return [(k[1], v) for k, v in sorted(by.items())]


def _split_cases(rows, ncases):
    """The dispatches between each case's start and end marker launches."""
    segs, cur = [], None
    for name, vals in rows:
        if name.startswith(MARKER_KERNEL):
            if cur is None:
                cur = []
            else:
                segs.append(cur)
                cur = None
        elif cur is not None:
            cur.append((name, vals))
    if len(segs) != ncases:
        raise ValueError(f"{len(segs)} marker segments, {ncases} cases")
    return segs


def _per_kernel_means(seg, counter):
    """Mean per dispatch of `counter` for each kernel of a case, in first-seen order."""
    order, vals = [], {}
    for name, v in seg:
        if counter in v:
            if name not in vals:
                order.append(name)
                vals[name] = []
            vals[name].append(v[counter])
    return [(n, float(np.mean(vals[n])), len(vals[n])) for n in order]


def summarize_counters(outdir: str) -> None:
    """profiles/counters_<kernel>_<workload>.txt for every case of the counter
    pass (HBM bytes per step from FETCH_SIZE and WRITE_SIZE, each scaled by
    what it reads for a device copy of known size) and
    profiles/issue_rate_<workload>.md (instruction-issue counters of the fused,
    two-launch and group-wait kernels on the prefill shard)."""
    cases = json.loads(open(os.path.join(outdir, "counter_pass.json")).read().strip().splitlines()[-1])
    segs = {tag: _split_cases(_counter_rows(os.path.join(outdir, tag)), len(cases))
            for tag, _ in COUNTER_PASSES}
    cal = 0
    cal_f = sum(m for _, m, _ in _per_kernel_means(segs["pmc_fetch"][cal], "FETCH_SIZE"))
    cal_w = sum(m for _, m, _ in _per_kernel_means(segs["pmc_write"][cal], "WRITE_SIZE"))
    half = cases[cal]["bytes_per_step"] // 2
    sf, sw = half / 1024 / cal_f, half / 1024 / cal_w
    sha, psha = source_sha256(), proj_sha256()
    cmds = ["python -u bench.py --counter-pass > gpurun_out/counters/counter_pass.json"] + [
        f"rocprofv3 --pmc {ctrs} --output-format csv -d gpurun_out/counters/{tag} -o c -- "
        f"python -u bench.py --counter-pass" for tag, ctrs in COUNTER_PASSES] + [
        "python bench.py --summarize-counters gpurun_out/counters"]
    written = []
    for i, c in enumerate(cases):
        if i == cal:
            continue
        fetch = _per_kernel_means(segs["pmc_fetch"][i], "FETCH_SIZE")
        write = dict((n, (m, k)) for n, m, k in _per_kernel_means(segs["pmc_write"][i], "WRITE_SIZE"))
        kernels = [n for n, _, _ in fetch]
        per_step = COUNTER_STEPS
        lines = []
        hbm = 0.0
        for n, mf, k in fetch:
            mw, _ = write[n]
            reps = k / per_step  # dispatches of this kernel per step
            bf, bw = mf * 1024 * sf * reps, mw * 1024 * sw * reps
            hbm += bf + bw
            lines.append(f"  {n}: {k} dispatches ({reps:g} per step); FETCH_SIZE {mf:.1f} KiB, "
                         f"WRITE_SIZE {mw:.1f} KiB per dispatch -> {int(round(bf))} + "
                         f"{int(round(bw))} bytes per step after scaling")
        proj = c["tag"] == "proj"
        fname = (f"counters_two_step_{c['workload']}.txt" if c["tag"] == "two_step"
                 else os.path.basename(counters_path(c["launch_names"][0], c["workload"])))
        out = [f"launches of one step: {', '.join(c['launch_names'])}" +
               (f" ({c['note']})" if c.get("note") else ""),
               f"profiler names: {', '.join(kernels)}",
               f"workload: {c['workload']}",
               (f"source_sha256 (qkn_proj.hip): {psha}" if proj else f"source_sha256: {sha}"),
               "commands (on the MI355X, from the repository root):"] + [f"  {x}" for x in cmds] + [
               f"calibration copy ({half // 1024} KiB read and written): FETCH_SIZE {cal_f:.1f} KiB "
               f"-> scale {sf:.4f}; WRITE_SIZE {cal_w:.1f} KiB -> scale {sw:.4f}",
               f"per kernel, mean over the {per_step} steps between the marker launches:"] + lines + [
               f"algorithmic_bytes_per_launch: {c['bytes_per_step']}",
               f"hbm_bytes_per_launch: {int(round(hbm))}",
               f"traffic_over_algorithmic: {hbm / c['bytes_per_step']:.4f}"]
        with open(os.path.join(ROOT, "profiles", fname), "w") as f:
            f.write("\n".join(out) + "\n")
        written.append((fname, hbm / c["bytes_per_step"]))
    # issue rate on the prefill shard: fused, two-launch, group wait
    keys = ("SQ_WAVES", "SQ_BUSY_CYCLES", "SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_INSTS_VALU",
            "SQ_INSTS_SALU", "SQ_INSTS_VMEM_RD", "SQ_INSTS_VMEM_WR")
    keys2 = ("GRBM_GUI_ACTIVE", "SQ_INSTS_SMEM", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_ANY")
    c4 = cases[1]["workload"]
    rows = ["| case | kernels per step | waves | instructions (VALU+SALU+VMEM+SMEM) | "
            "SQ_BUSY_CYCLES | GRBM_GUI_ACTIVE | instructions per busy cycle | "
            "SQ_WAIT_ANY / SQ_WAVE_CYCLES | SQ_ACTIVE_INST_ANY / SQ_WAVE_CYCLES |",
            "|---|---|---|---|---|---|---|---|---|"]
    rate = {}
    for i, c in enumerate(cases):
        if c["workload"] != c4 or c["tag"] not in ("fused", "two_step", "group_wait"):
            continue
        tot = {}
        for k in keys:
            tot[k] = sum(m * (n_ / COUNTER_STEPS) for _, m, n_ in _per_kernel_means(segs["pmc_issue"][i], k))
        for k in keys2:
            tot[k] = sum(m * (n_ / COUNTER_STEPS) for _, m, n_ in _per_kernel_means(segs["pmc_issue2"][i], k))
        inst = tot["SQ_INSTS_VALU"] + tot["SQ_INSTS_SALU"] + tot["SQ_INSTS_VMEM_RD"] + \
            tot["SQ_INSTS_VMEM_WR"] + tot["SQ_INSTS_SMEM"]
        rate[c["tag"]] = inst / tot["SQ_BUSY_CYCLES"]
        rows.append(f"| {c['tag']} | {', '.join(c['launch_names'])} | {tot['SQ_WAVES']:.0f} | {inst:.3e} | "
                    f"{tot['SQ_BUSY_CYCLES']:.3e} | {tot['GRBM_GUI_ACTIVE']:.3e} | {rate[c['tag']]:.2f} | "
                    f"{tot['SQ_WAIT_ANY'] / tot['SQ_WAVE_CYCLES']:.3f} | "
                    f"{tot['SQ_ACTIVE_INST_ANY'] / tot['SQ_WAVE_CYCLES']:.3f} |")
    md = [f"# Instruction issue on the prefill shard ({c4})", "",
          f"Kernel source sha256 {sha}. Commands (MI355X, repository root):", ""] + \
         [f"    {x}" for x in cmds] + ["",
          "Counters summed over the kernels of one step (means per dispatch times dispatches per "
          "step). instructions = SQ_INSTS_VALU + SQ_INSTS_SALU + SQ_INSTS_VMEM_RD + "
          "SQ_INSTS_VMEM_WR + SQ_INSTS_SMEM; SQ_BUSY_CYCLES counts the cycles the sequencers are "
          "busy, so instructions per busy cycle is the issue-rate analogue of a GPU-wide "
          "instruction rate.", ""] + rows
    if "fused" in rate and "two_step" in rate:
        md += ["", f"Issue rate, fused over two-launch: {rate['fused'] / rate['two_step']:.2f}x."]
    with open(os.path.join(ROOT, "profiles", f"issue_rate_{c4}.md"), "w") as f:
        f.write("\n".join(md) + "\n")
    for fname, ratio in written:
        print(f"{fname}: traffic / algorithmic {ratio:.4f}")
    print("\n".join(md[-len(rows) - 2:]))


MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16


def proj_extra(torch, L, workloads, wl, rank, steps=50, graph=False):
    """The Q/K projection with the statistic against torch.mm. graph=True times
    replays of a captured graph (decode sizes, where back-to-back eager calls
    are bound by the host) and prices the launch against the HBM roofline
    (streaming W dominates); otherwise eager launches against the MFMA peak."""
    dev = "cuda:0"

    def bf16(a):
        a = np.ascontiguousarray(a, dtype=np.uint16)
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
    data = workloads.projection_inputs(wl)
    x = bf16(data["x"])
    wq = bf16(data["wq"][workloads.shard_cols(wl.q_full, wl.tp, rank)])
    wk = bf16(data["wk"][workloads.shard_cols(wl.k_full, wl.tp, rank)])
    hidden = x.shape[1]
    flops = 2 * wl.T * hidden * (wq.shape[0] + wk.shape[0])
    prep = L.PreparedProj(x, [L.ProjSeg(w=wq), L.ProjSeg(w=wk)])
    wqk_t = torch.cat([wq, wk]).t().contiguous()
    def timed(fn):  # ms per call
        if graph:
            return time_graph(torch, fn, steps, 10)
        return time_region(torch, fn, steps, 10) / steps
    ours, lib = [], []
    for _ in range(5):  # alternate, median of five regions each
        ours.append(timed(lambda i: prep()))
        lib.append(timed(lambda i: torch.mm(x, wqk_t)))
    prep()
    info = L.qkn_last_launch()
    t, tm = float(np.median(ours)), float(np.median(lib))
    tf = flops / (t * 1e-3) / 1e12
    cols = wq.shape[0] + wk.shape[0]
    if graph:
        nbytes = 2 * (cols * hidden + wl.T * hidden + wl.T * cols)  # W, x, y in bf16
        gbs = nbytes / (t * 1e-3) / 1e9
        roof = {"bound": "hbm", "bytes": nbytes, "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4)}
    else:
        roof = {"bound": "mfma", "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4)}
    return {"kernel": info["kernel"], "grid": info["grid"], "tokens": wl.T, "hidden": hidden,
            "columns": cols, "flops": flops, "kernel_us": round(t * 1e3, 2),
            "timing": "graph replay" if graph else "eager", "tflops": round(tf, 1),
            "roofline": roof, "torch_mm_us": round(tm * 1e3, 2),
            "torch_mm_tflops": round(flops / (tm * 1e-3) / 1e12, 1)}


PROJ_COUNTERS = (
    ("pmc_proj1", "SQ_WAVES SQ_BUSY_CYCLES SQ_WAVE_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_LDS "
                  "SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT SQ_INSTS_MFMA"),
    ("pmc_proj2", "GRBM_GUI_ACTIVE SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU SQ_ACTIVE_INST_LDS"),
)


def summarize_proj(outdir: str) -> None:
    """Counters of the projection kernel and of torch.mm (hipBLASLt) of the same
    product, from two rocprofv3 --pmc runs of `bench.py --proj-only`, into
    profiles/counters_proj_prefill_T8192_h4096_q2048_k512.txt (means per
    dispatch)."""
    import csv
    import collections
    cmds, rows = [], collections.defaultdict(lambda: collections.defaultdict(list))
    for sub, counters in PROJ_COUNTERS:
        path = os.path.join(outdir, sub)
        files = [f for f in os.listdir(path) if f.endswith("counter_collection.csv")]
        if not files:
            raise SystemExit(f"no counter CSV in {path}")
        cmds.append(f"rocprofv3 --pmc {counters} --output-format csv -d gpurun_out/{sub} -o p "
                    "-- python -u bench.py --proj-only")
        for r in csv.DictReader(open(os.path.join(path, files[0]))):
            name = r["Kernel_Name"]
            if "qkn_proj_gemm" in name:
                key = "qkn_proj_gemm_dl (this library)"
            elif name.startswith("Cijk"):
                key = "hipBLASLt GEMM (torch.mm)"
            else:
                continue
            rows[key][r["Counter_Name"]].append(float(r["Counter_Value"]))
    lines = ["Q/K projection, 8192 tokens x hidden 4096 -> 2048 + 512 columns (bf16, fp32 accumulation)",
             f"source_sha256 (qkn_proj.hip): {proj_sha256()}",
             "commands (on the MI355X, from the repository root):"]
    lines += ["  " + c for c in cmds]
    lines += ["  python bench.py --summarize-proj gpurun_out",
              "mean counter value per dispatch (sums over the GPU):"]
    for key in sorted(rows):
        lines.append(key + ":")
        for c in sorted(rows[key]):
            v = rows[key][c]
            lines.append(f"  {c}: {sum(v) / len(v):.0f}")
    out = os.path.join(ROOT, "profiles", "counters_proj_prefill_T8192_h4096_q2048_k512.txt")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


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
            "host_cpus_visible": ncpu, "cpu_model": cpu_model(),
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), else the machine type."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def main():
    args = parse()
    if args.summarize:
        summarize(args.summarize)
        return 0
    if args.summarize_proj:
        summarize_proj(args.summarize_proj)
        return 0
    if args.summarize_counters:
        summarize_counters(args.summarize_counters)
        return 0
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU's share of the sharded QK-Norm; the peer ranks "
              "are simulated in device memory. Runs on more than one GPU are not supported: "
              "use --gpus 1.", file=sys.stderr)
        return 2
    import torch
    import workloads
    from paper_2608_09160_amd import _lib as L

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    L.load()
    wl = workloads.WORKLOADS[args.workload]
    if args.proj_only:
        out = {"proj_partial_prefill": proj_extra(torch, L, workloads, wl, args.rank, steps=10)}
        print(json.dumps(out), flush=True)
        return 0
    if args.counter_pass:
        print(json.dumps(counter_pass(torch, L, workloads, args.min_footprint_mb << 20)), flush=True)
        return 0
    data = workloads.generate(wl)
    min_fp = args.min_footprint_mb << 20

    print(f"[bench] {wl.name}: building rotating buffers", file=sys.stderr, flush=True)
    case = Case(wl, args.rank, min_fp, torch, L, workloads, data=data)
    case.launch(0)
    info = L.qkn_last_launch()
    # timed region: exactly `steps` launches, nothing else on the stream
    torch.cuda.synchronize()
    region_ms = time_region(torch, case.launch, args.steps, args.warmup)
    torch.cuda.synchronize()
    ms_per_step = region_ms / args.steps
    value = case.bytes / (ms_per_step * 1e-3) / 1e9
    # average launch duration = timed region / launches (back-to-back on one
    # stream, as the profiler's kernel trace sees them)
    kernel_ms = ms_per_step
    achieved = case.bytes / (kernel_ms * 1e-3) / 1e9
    # for reference: events bracketing every launch (adds the events' own cost)
    each = time_each(torch, case.launch, args.steps, args.warmup)
    isolated_ms = float(np.mean(each))
    print(f"[bench] fused: {ms_per_step * 1e3:.2f} us/step ({achieved:.0f} GB/s); "
          f"isolated launch {isolated_ms * 1e3:.2f} us", file=sys.stderr, flush=True)

    extras = {}
    if args.calibration_copy:
        xq, yq = case.sets[0][0].x, case.sets[0][0].y
        for _ in range(5):
            yq.copy_(xq)
        torch.cuda.synchronize()
        extras["calibration_copy"] = {"read_bytes": xq.numel() * 2, "write_bytes": yq.numel() * 2,
                                      "launches": 5}
    if not args.no_extras:
        # the practical ceiling: a streaming copy of the same bytes in one launch
        # (qkn_calib_copy, best of four grid sizes), over rotating buffer sets as
        # large as the kernel's, so that it too reads from HBM
        copy_bytes = sum(2 * s.x.numel() * 2 for s in case.sets[0])  # read + written
        cms, cblocks = stream_copy_ms(torch, L, copy_bytes, min_fp, args.steps, args.warmup)
        extras["stream_copy_same_bytes"] = {
            "bytes": copy_bytes, "us_per_step": round(cms * 1e3, 3), "blocks": cblocks,
            "gbs": round(copy_bytes / (cms * 1e-3) / 1e9, 1),
            "fused_kernel_frac_of_copy": round(cms / ms_per_step, 4)}
        # the fixed cost per launch and the streaming rate: launch time against
        # the token count at the prefill shard's widths, kernel and copy
        extras["time_vs_tokens"] = token_fit(torch, L, min_fp, args.steps, args.warmup)
        extras["time_vs_tokens_fp8"] = token_fit(torch, L, min_fp, args.steps, args.warmup,
                                                 fp8=True)
        # the launch floor: an empty kernel replayed from a HIP graph
        us = time_graph(torch, lambda i: L.qkn_calib_empty(), 200, 10) * 1e3
        extras["empty_kernel_graph"] = {"us_per_launch_graph": round(us, 3)}
        # torch's copy of the same tensors (two launches), for context
        csets = [([s.x for s in segs], [s.y for s in segs]) for segs in case.sets]

        def copy(i):
            xs, ys = csets[i % len(csets)]
            for a, b in zip(xs, ys):
                b.copy_(a)
        r = time_region(torch, copy, args.steps, args.warmup)
        extras["torch_copy_same_bytes"] = {"bytes": copy_bytes,
                                           "us_per_step": round(r / args.steps * 1e3, 3),
                                           "gbs": round(copy_bytes / (r / args.steps * 1e-3) / 1e9, 1)}
        # two launches per tensor: Phase A, then Phases B+C (x read twice).
        # Its four calls through the generic binding take longer on the host
        # than on the GPU, so the GPU time comes from a replayed HIP graph;
        # the stream figure is reported beside it.
        r = time_region(torch, case.launch_two_step, args.steps, args.warmup)
        g = time_graph(torch, case.launch_two_step, 2 * case.nsets, max(1, args.steps // (2 * case.nsets)))
        two_bytes = case.bytes + sum(2 * s.x.numel() for s in case.sets[0])
        extras["two_step_same_workload"] = {"us_per_step": round(g * 1e3, 3),
                                            "gbs": round(two_bytes / (g * 1e-3) / 1e9, 1),
                                            "bytes": two_bytes, "timing": "HIP graph replay",
                                            "stream_us_per_step_host_bound": round(r / args.steps * 1e3, 3)}
        # full-vector (tp = 1) baseline on the same tokens
        fcase = Case(wl.with_tp(1), 0, min_fp, torch, L, workloads, data=data, partials=False)
        fk = time_region(torch, fcase.launch, args.steps, args.warmup) / args.steps
        extras["full_vector_tp1"] = {"kernel": L.qkn_last_launch()["kernel"], "bytes": fcase.bytes,
                                     "kernel_us": round(fk * 1e3, 3),
                                     "gbs": round(fcase.bytes / (fk * 1e-3) / 1e9, 1)}
        cms, _ = stream_copy_ms(torch, L, fcase.bytes, min_fp, args.steps, args.warmup)
        extras["full_vector_tp1"]["copy_us"] = round(cms * 1e3, 3)
        extras["full_vector_tp1"]["frac_of_copy"] = round(cms / fk, 4)
        del fcase
        # the Phase B wait: every rank of the tp group in one launch, each wavefront
        # publishing its statistic and waiting for the others' (same data as tp = 1)
        gcase = GroupCase(wl, min_fp, torch, L, data)
        gk = time_region(torch, gcase.launch, args.steps, args.warmup) / args.steps
        gstatus = int(gcase.status.item())
        extras["group_wait_all_ranks"] = {"kernel": L.qkn_last_launch()["kernel"],
                                          "bytes": gcase.bytes, "kernel_us": round(gk * 1e3, 3),
                                          "gbs": round(gcase.bytes / (gk * 1e-3) / 1e9, 1),
                                          "status": gstatus}
        del gcase
        f8g = wl.with_dtype("fp8")
        gcase = GroupCase(f8g, min_fp, torch, L, workloads.generate(f8g))
        gk = time_region(torch, gcase.launch, args.steps, args.warmup) / args.steps
        extras["fp8_group_wait_all_ranks"] = {"kernel": L.qkn_last_launch()["kernel"],
                                              "bytes": gcase.bytes, "kernel_us": round(gk * 1e3, 3),
                                              "gbs": round(gcase.bytes / (gk * 1e-3) / 1e9, 1),
                                              "status": int(gcase.status.item())}
        del gcase
        # decode shapes: one launch replayed from a HIP graph (inputs cache-warm,
        # as right after the projection that produced them)
        lat = {}
        for name in ("decode_T64_q4096_k1024_tp4", "decode_T256_q5120_k1024_tp8",
                     "tiny_full_T16_q512_k128_tp1"):
            dwl = workloads.WORKLOADS[name]
            dcase = Case(dwl, 0, 0, torch, L, workloads, partials=dwl.tp > 1)
            us = time_graph(torch, lambda i, c=dcase: c.launch(0), 200, 10) * 1e3
            lat[name] = {"us_per_launch_graph": round(us, 3), "kernel": L.qkn_last_launch()["kernel"],
                         "grid": L.qkn_last_launch()["grid"], "bytes": dcase.bytes}
            del dcase
        extras["decode_latency_warm"] = lat
        # cold: every launch after a streaming copy of 2 x 384 MB, which evicts
        # L2 and the 256 MB Infinity Cache; events right around each launch,
        # next to the same measurement of an empty kernel (the events' own cost)
        big = 384 << 20
        fa = torch.empty(big, dtype=torch.uint8, device="cuda:0")
        fb = torch.empty(big, dtype=torch.uint8, device="cuda:0")

        def flush():
            L.qkn_calib_copy(fa, fb, blocks=8192)
        nc = 100
        empty = np.array(time_cold(torch, lambda i: L.qkn_calib_empty(), nc, flush)) * 1e3
        cold = {"empty_kernel_event_us_median": round(float(np.median(empty)), 3)}
        for name in ("decode_T64_q4096_k1024_tp4", "decode_T256_q5120_k1024_tp8"):
            dwl = workloads.WORKLOADS[name]
            dcase = Case(dwl, 0, 0, torch, L, workloads, partials=dwl.tp > 1)
            t = np.array(time_cold(torch, lambda i, c=dcase: c.launch(0), nc, flush)) * 1e3
            cold[name] = {"event_us_median": round(float(np.median(t)), 3),
                          "event_us_p10": round(float(np.percentile(t, 10)), 3),
                          "event_us_p90": round(float(np.percentile(t, 90)), 3),
                          "over_empty_kernel_us": round(float(np.median(t) - np.median(empty)), 3)}
            del dcase
        del fa, fb
        extras["decode_latency_cold"] = cold
        # long prefill shard
        lcase = Case(workloads.LONG_PREFILL_TP4, 0, min_fp, torch, L, workloads)
        nl = max(20, args.steps // 4)
        lk = time_region(torch, lcase.launch, nl, 5) / nl
        extras["long_prefill_tp4"] = {"kernel": L.qkn_last_launch()["kernel"], "bytes": lcase.bytes,
                                      "kernel_us": round(lk * 1e3, 3),
                                      "gbs": round(lcase.bytes / (lk * 1e-3) / 1e9, 1)}
        cms, _ = stream_copy_ms(torch, L, lcase.bytes, min_fp, nl, 5)
        extras["long_prefill_tp4"]["copy_us"] = round(cms * 1e3, 3)
        extras["long_prefill_tp4"]["frac_of_copy"] = round(cms / lk, 4)
        del lcase
        # FP8-E4M3 activations (Sec. IV-C's second format): the same prefill
        # shard, and the decode shape replayed from a graph
        f8 = wl.with_dtype("fp8")
        p8 = Case(f8, args.rank, min_fp, torch, L, workloads)
        pk = time_region(torch, p8.launch, args.steps, args.warmup) / args.steps
        extras["fp8_prefill_shard"] = {"kernel": L.qkn_last_launch()["kernel"], "bytes": p8.bytes,
                                       "kernel_us": round(pk * 1e3, 3),
                                       "gbs": round(p8.bytes / (pk * 1e-3) / 1e9, 1),
                                       "frac_of_peak": round(p8.bytes / (pk * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
        cms, _ = stream_copy_ms(torch, L, p8.bytes, min_fp, args.steps, args.warmup)
        extras["fp8_prefill_shard"]["copy_us"] = round(cms * 1e3, 3)
        extras["fp8_prefill_shard"]["frac_of_copy"] = round(cms / pk, 4)
        del p8
        d8 = Case(workloads.DECODE_TP4.with_dtype("fp8"), 0, 0, torch, L, workloads)
        us = time_graph(torch, lambda i, c=d8: c.launch(0), 200, 10) * 1e3
        extras["fp8_decode_T64_tp4_graph"] = {"us_per_launch_graph": round(us, 3),
                                              "kernel": L.qkn_last_launch()["kernel"],
                                              "bytes": d8.bytes}
        del d8
        # Phase A in the Q/K projection's epilogue: the rank's column-parallel
        # projection (hidden 4096 -> Q 2048 + K 512 columns) on the matrix
        # cores, with the statistic taken from each output tile; against
        # torch.mm (hipBLASLt) of the same product without the statistic
        extras["proj_partial_prefill"] = proj_extra(torch, L, workloads, wl, args.rank)
        # the same at decode size: 64 tokens, Q 1024 + K 256 columns (tp 4)
        extras["proj_partial_decode"] = proj_extra(torch, L, workloads, workloads.DECODE_TP4, 1,
                                                   steps=20, graph=True)
        print("[bench] extras done", file=sys.stderr, flush=True)

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
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic_bytes(info["kernel"], wl.name),
                     "algorithmic_bytes": case.bytes, "kernel_us": round(kernel_ms * 1e3, 3),
                     "isolated_launch_us": round(isolated_ms * 1e3, 3),
                     # a streaming copy of the same bytes in the same run: the
                     # practical ceiling of a read-once/write-once kernel
                     "copy_ceiling": ({"us": extras["stream_copy_same_bytes"]["us_per_step"],
                                       "frac_of_peak": round(
                                           extras["stream_copy_same_bytes"]["gbs"] / HBM_PEAK_GBS, 4),
                                       "kernel_frac_of_copy":
                                           extras["stream_copy_same_bytes"]["fused_kernel_frac_of_copy"]}
                                      if "stream_copy_same_bytes" in extras else None)},
        "cpu_baseline": cpu,
        "extras": extras,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
