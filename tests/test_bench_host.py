"""Host logic of bench.py (no GPU): the algorithmic byte count behind
`value` and `roofline.achieved`, the profiler-name mapping the profile
summaries rely on, and the counter file's source check."""
import os

import bench
import workloads


def test_algorithmic_bytes_of_the_prefill_shard():
    wl = workloads.PREFILL_TP2
    # x read + y written (bf16), gamma once, own statistic written, the one
    # peer's statistic read, for Q (2048 columns) and K (512)
    expect = sum(2 * wl.T * d * 2 + 4 * d + 4 * wl.T + 4 * wl.T for d in (2048, 512))
    assert bench.algorithmic_bytes(wl.T, (wl.q_local, wl.k_local), wl.tp) == expect == 84_027_392
    # FP8 halves the activation bytes only
    fp8 = bench.algorithmic_bytes(wl.T, (2048, 512), 2, esz=1)
    assert expect - fp8 == wl.T * (2048 + 512) * 2


def test_profiler_names():
    assert bench.trace_name("rows<4,1>/fused") == "void qkn_rows<FmtBf16, 4, 1, 0, 0>"
    assert bench.trace_name("rows_pa3_fp8<2,1>/fused_wait") == "void qkn_rows<FmtFp8, 2, 1, 3, 4>"
    assert bench.trace_name("wide<16,1>/apply") == "void qkn_wide<FmtBf16, 16, 1, 1>"
    assert bench.kernel_base_name(
        "void qkn_dev::qkn_rows<qkn_dev::FmtBf16, 4, 1, 0, 0>(qkn_dev::KParams)") == \
        "void qkn_rows<FmtBf16, 4, 1, 0, 0>"
    assert bench.kernel_base_name("(anonymous namespace)::qkn_calib_copy_kernel(unsigned int*)") == \
        "qkn_calib_copy_kernel"


def test_counter_summary_is_used_only_for_the_current_source(monkeypatch):
    wl = workloads.PREFILL_TP2
    path = bench.counters_path("rows<4,1>/fused", wl.name)
    assert os.path.basename(path) == f"counters_rows_4_1_fused_{wl.name}.txt"
    text = open(path).read()
    alg = bench.algorithmic_bytes(wl.T, (wl.q_local, wl.k_local), wl.tp)
    if f"source_sha256: {bench.source_sha256()}" in text:
        # counters of the current source: used, and at least the algorithmic bytes
        assert bench.traffic_bytes("rows<4,1>/fused", wl.name) > alg
    else:
        # taken before the last kernel change: not used
        assert bench.traffic_bytes("rows<4,1>/fused", wl.name) is None
    # a summary whose recorded hash differs from the source is never used
    monkeypatch.setattr(bench, "source_sha256", lambda: "0" * 64)
    assert bench.traffic_bytes("rows<4,1>/fused", wl.name) is None


def test_every_launch_name_family_maps():
    for name, want in (("rows_pf<8,2>/apply", "void qkn_rows<FmtBf16, 8, 2, 1, 1>"),
                       ("rows_pa<4,1>/fused_wait", "void qkn_rows<FmtBf16, 4, 1, 3, 2>"),
                       ("rows_pa2_fp8<2,1>/fused_wait", "void qkn_rows<FmtFp8, 2, 1, 3, 3>"),
                       ("rows_fp8<2,0>/publish", "void qkn_rows<FmtFp8, 2, 0, 4, 0>"),
                       ("wide_fp8<8,4>/fused", "void qkn_wide<FmtFp8, 8, 4, 0>")):
        assert bench.trace_name(name) == want
    for bad in ("wide_pa3<16,1>/fused_wait", "generic/fused", "rows<4,1>/other"):
        try:
            bench.trace_name(bad)
        except ValueError:
            continue
        raise AssertionError(bad)
