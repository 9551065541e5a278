"""The C ABI without a GPU: symbols, validation, overlap rules and path choice.

Every call here either fails validation (which happens before any HIP call) or
runs with the library's "validate_only" option set, which accepts the call,
chooses a kernel without touching the GPU and returns QKN_EDRYRUN (never
QKN_OK, so a call that launched nothing cannot pass for one that ran). The pointers are fake addresses that
are never dereferenced, so these tests are safe on any machine.
"""
import ctypes
import os
import re

import pytest

from paper_2608_09160_amd import _lib as L

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "qkn.h")

BASE = 0x7f0000000000  # fake, 256-byte aligned device addresses
MB = 1 << 20
DRY = L.QKN_EDRYRUN  # what a validated call returns under validate_only: nothing launched


@pytest.fixture(scope="module")
def lib():
    return L.load()


@pytest.fixture
def dry(lib):
    assert lib.qkn_set_option(b"validate_only", 1) == 0
    yield lib
    for key in (b"validate_only", b"force_generic", b"prefetch", b"token_blocks"):
        assert lib.qkn_set_option(key, 0) == 0


def _declared_functions():
    text = "".join(open(os.path.join(os.path.dirname(HEADER), h)).read()
                   for h in sorted(os.listdir(os.path.dirname(HEADER))) if h.endswith(".h"))
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(qkn_[a-z0-9_]+)\s*\(", text)))


def test_header_symbols_exported(lib):
    names = _declared_functions()
    assert set(names) >= {"qkn_partial_sumsq", "qkn_apply", "qkn_fused_shard", "qkn_full",
                          "qkn_strerror", "qkn_last_launch", "qkn_set_option",
                          "qkn_partial_sumsq_fp8", "qkn_apply_fp8", "qkn_fused_shard_fp8",
                          "qkn_full_fp8", "qkn_proj_workspace_bytes", "qkn_proj_partial"}
    for n in names:
        assert hasattr(lib, n), n


def test_strerror(lib):
    for code in (0, -1, -2, -3, 17):
        assert isinstance(lib.qkn_strerror(code), bytes)
    assert lib.qkn_strerror(-2).startswith(b"output overlaps")


def _seg(x, ldx, w, partials, y, ldy, d_local, d_full, inv=None):
    return L.QknSeg(x, ldx, w, partials, y, ldy, inv, d_local, d_full)


def _fused(lib, segs, tp, rank, T, eps=1e-6):
    arr = (L.QknSeg * len(segs))(*segs)
    return lib.qkn_fused_shard(arr, len(segs), tp, rank, T, ctypes.c_float(eps), None)


def _q(T=64, d=1024, ld=None, rank_tp=4):
    """A well-formed Q segment at distinct fake addresses."""
    ld = ld or d
    return _seg(BASE, ld, BASE + 64 * MB, BASE + 65 * MB, BASE + 128 * MB, ld, d, d * rank_tp)


def _k(T=64, d=256, rank_tp=4):
    return _seg(BASE + 256 * MB, d, BASE + 300 * MB, BASE + 301 * MB, BASE + 400 * MB, d, d,
                d * rank_tp)


def test_valid_calls_pass_validation(dry):
    assert _fused(dry, [_q(), _k()], 4, 1, 64) == DRY
    info = L.qkn_last_launch()
    assert info["kernel"].endswith("<2,1>/fused") and info["grid"] == 0
    assert dry.qkn_partial_sumsq(BASE, 1024, 64, 1024, BASE + 64 * MB, None) == DRY
    assert L.qkn_last_launch()["kernel"].endswith("<2,0>/partial")
    assert dry.qkn_apply(BASE, 1024, BASE + 64 * MB, BASE + 65 * MB, 4, 64, 1024, 4096,
                         ctypes.c_float(1e-6), BASE + 128 * MB, 1024, None, None) == DRY
    assert L.qkn_last_launch()["kernel"].endswith("<2,0>/apply")
    full = [_seg(BASE, 4096, BASE + 64 * MB, 0, BASE + 128 * MB, 4096, 4096, 4096),
            _seg(BASE + 256 * MB, 1024, BASE + 300 * MB, 0, BASE + 400 * MB, 1024, 1024, 1024)]
    arr = (L.QknSeg * 2)(*full)
    assert dry.qkn_full(arr, 2, 8192, ctypes.c_float(1e-6), None) == DRY
    assert L.qkn_last_launch()["kernel"].endswith("<8,2>/fused")


@pytest.mark.parametrize("d,expect", [(8, "<1,0>"), (512, "<1,0>"), (520, "<2,0>"),
                                      (2048, "<4,0>"), (1536, "<4,0>"),
                                      (4096, "<8,0>"), (4104, "wide<16,0>"), (8192, "wide<16,0>"),
                                      (8200, "wide<32,0>"), (16384, "wide<32,0>"),
                                      (16392, "generic"), (100, "generic"), (1, "generic")])
def test_path_choice_by_width(dry, d, expect):
    seg = _seg(BASE, d, BASE + 64 * MB, BASE + 65 * MB, BASE + 128 * MB, d, d, 2 * d)
    assert _fused(dry, [seg], 2, 0, 16) == DRY
    name = L.qkn_last_launch()["kernel"]
    if expect in ("generic",) or expect.startswith("wide"):
        assert name.startswith(expect), name
    else:
        assert name.startswith("rows") and expect in name, name


def test_wide_path_needs_gamma_to_fit_lds(dry):
    q = _seg(BASE, 16384, BASE + 640 * MB, BASE + 641 * MB, BASE + 256 * MB, 16384, 16384, 16384)
    k = _seg(BASE + 512 * MB, 1024, BASE + 642 * MB, BASE + 643 * MB, BASE + 700 * MB, 1024, 1024, 1024)
    assert _fused(dry, [q, k], 1, 0, 16) == DRY   # 17408 gamma floats > 64 KiB of LDS
    assert L.qkn_last_launch()["kernel"] == "generic/fused"
    q = _seg(BASE, 8192, BASE + 640 * MB, BASE + 641 * MB, BASE + 256 * MB, 8192, 8192, 8192)
    assert _fused(dry, [q, k], 1, 0, 16) == DRY
    assert L.qkn_last_launch()["kernel"] == "wide<16,2>/fused"
    assert L.qkn_last_launch()["lds_bytes"] == (8192 + 1024) * 4
    # the wide tensor may come second: the launcher puts it in slot 0
    assert _fused(dry, [k, q], 1, 0, 16) == DRY
    assert L.qkn_last_launch()["kernel"] == "wide<16,2>/fused"
    # both tensors wide: the general path
    k2 = _seg(BASE + 512 * MB, 5120, BASE + 642 * MB, BASE + 643 * MB, BASE + 700 * MB, 5120, 5120, 5120)
    q2 = _seg(BASE, 5120, BASE + 640 * MB, BASE + 641 * MB, BASE + 256 * MB, 5120, 5120, 5120)
    assert _fused(dry, [q2, k2], 1, 0, 16) == DRY
    assert L.qkn_last_launch()["kernel"] == "generic/fused"


def test_prefetch_option_selects_variant(dry):
    seg = _seg(BASE, 1024, BASE + 64 * MB, BASE + 65 * MB, BASE + 128 * MB, 1024, 1024, 2048)
    assert dry.qkn_set_option(b"prefetch", 0) == 0
    assert _fused(dry, [seg], 2, 0, 16) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows<2,0>/fused"
    assert dry.qkn_set_option(b"prefetch", 1) == 0
    assert _fused(dry, [seg], 2, 0, 16) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_pf<2,0>/fused"
    assert dry.qkn_set_option(b"prefetch", 2) == L.QKN_EINVAL


def test_register_path_needs_slot_offsets_in_range(dry):
    # tp * T * 4 bytes of statistics must stay below 2^31 for the register path
    G = 1 << 34  # regions of 16 GiB apart: x and y of 8M tokens x 1024 bf16 fit
    seg = _seg(BASE, 1024, BASE + 3 * G, BASE + 2 * G, BASE + G, 1024, 1024, 64 * 1024)
    assert _fused(dry, [seg], 64, 0, (1 << 31) // (64 * 4)) == DRY
    assert L.qkn_last_launch()["kernel"] == "generic/fused"
    assert _fused(dry, [seg], 64, 0, (1 << 31) // (64 * 4) - 1) == DRY
    assert L.qkn_last_launch()["kernel"].startswith("rows")


def test_path_choice_alignment_and_options(dry):
    # misaligned x (one element off) or a stride that is not a multiple of 8
    seg = _seg(BASE + 2, 1024, BASE + 64 * MB, BASE + 65 * MB, BASE + 128 * MB, 1024, 1024, 4096)
    assert _fused(dry, [seg], 4, 0, 16) == DRY
    assert L.qkn_last_launch()["kernel"] == "generic/fused"
    seg = _seg(BASE, 1028, BASE + 64 * MB, BASE + 65 * MB, BASE + 128 * MB, 1024, 1024, 4096)
    assert _fused(dry, [seg], 4, 0, 16) == DRY
    assert L.qkn_last_launch()["kernel"] == "generic/fused"
    seg = _seg(BASE, 1024, BASE + 64 * MB + 4, BASE + 65 * MB, BASE + 128 * MB, 1024, 1024, 4096)
    assert _fused(dry, [seg], 4, 0, 16) == DRY
    assert L.qkn_last_launch()["kernel"] == "generic/fused"
    # tp beyond one slot per lane
    assert _fused(dry, [_q(rank_tp=65)], 65, 64, 16) == DRY
    assert L.qkn_last_launch()["kernel"] == "generic/fused"
    # forced general path
    assert dry.qkn_set_option(b"force_generic", 1) == 0
    assert _fused(dry, [_q(), _k()], 4, 1, 64) == DRY
    assert L.qkn_last_launch()["kernel"] == "generic/fused"
    assert L.qkn_last_launch()["lds_bytes"] == 1024 * 2


def test_zero_tokens_is_a_noop(lib):
    # T == 0 returns before any HIP call, even with NULL pointers
    assert lib.qkn_partial_sumsq(None, 8, 0, 8, None, None) == 0
    assert lib.qkn_apply(None, 8, None, None, 2, 0, 8, 16, ctypes.c_float(0.0),
                         None, 8, None, None) == 0
    seg = _seg(None, 8, None, None, None, 8, 8, 16)
    assert _fused(lib, [seg], 2, 0, 0) == 0


@pytest.mark.parametrize("case", [
    "T<0", "tp<1", "rank>=tp", "rank<0", "eps<0", "eps=nan", "eps=inf", "nseg=0", "nseg=3",
    "d_local<1", "ldx<d", "ldy<d", "d_full<d", "x=NULL", "w=NULL", "y=NULL", "partials=NULL",
    "segs=NULL"])
def test_invalid_arguments(lib, case):
    q, k = _q(), _k()
    tp, rank, T, eps, nseg = 4, 1, 64, 1e-6, 2
    if case == "T<0": T = -1
    elif case == "tp<1": tp = 0
    elif case == "rank>=tp": rank = 4
    elif case == "rank<0": rank = -1
    elif case == "eps<0": eps = -1e-6
    elif case == "eps=nan": eps = float("nan")
    elif case == "eps=inf": eps = float("inf")
    elif case == "nseg=0": nseg = 0
    elif case == "nseg=3": nseg = 3
    elif case == "d_local<1": q.d_local = 0
    elif case == "ldx<d": q.ldx = 1000
    elif case == "ldy<d": k.ldy = 255
    elif case == "d_full<d": k.d_full = 255
    elif case == "x=NULL": q.x = None
    elif case == "w=NULL": k.w = None
    elif case == "y=NULL": q.y = None
    elif case == "partials=NULL": k.partials = None
    arr = (L.QknSeg * 3)(q, k, k)
    ptr = None if case == "segs=NULL" else arr
    rc = lib.qkn_fused_shard(ptr, nseg, tp, rank, T, ctypes.c_float(eps), None)
    assert rc == L.QKN_EINVAL


def test_invalid_partial_and_apply(lib):
    f = ctypes.c_float
    assert lib.qkn_partial_sumsq(BASE, 8, 4, 0, BASE + MB, None) == L.QKN_EINVAL
    assert lib.qkn_partial_sumsq(BASE, 8, 4, 16, BASE + MB, None) == L.QKN_EINVAL
    assert lib.qkn_partial_sumsq(None, 8, 4, 8, BASE + MB, None) == L.QKN_EINVAL
    assert lib.qkn_partial_sumsq(BASE, 8, 4, 8, None, None) == L.QKN_EINVAL
    assert lib.qkn_partial_sumsq(BASE, 8, -1, 8, BASE + MB, None) == L.QKN_EINVAL
    ok = dict(x=BASE, ldx=8, w=BASE + MB, p=BASE + 2 * MB, tp=2, T=4, d=8, dfull=16, eps=1e-6,
              y=BASE + 3 * MB, ldy=8)

    def call(**kw):
        a = dict(ok, **kw)
        return lib.qkn_apply(a["x"], a["ldx"], a["w"], a["p"], a["tp"], a["T"], a["d"],
                             a["dfull"], f(a["eps"]), a["y"], a["ldy"], None, None)
    for bad in (dict(p=None), dict(w=None), dict(y=None), dict(x=None), dict(tp=0),
                dict(dfull=7), dict(ldy=7), dict(eps=-1.0), dict(T=-3)):
        assert call(**bad) == L.QKN_EINVAL, bad
    # full-vector call requires d_local == d_full
    seg = _seg(BASE, 8, BASE + MB, None, BASE + 3 * MB, 8, 8, 16)
    assert lib.qkn_full((L.QknSeg * 1)(seg), 1, 4, f(1e-6), None) == L.QKN_EINVAL


def test_overlap_rules(dry):
    T, d = 16, 1024
    # y shifted by one element onto x: partial overlap
    seg = _seg(BASE, d, BASE + 64 * MB, BASE + 65 * MB, BASE + 2, d, d, 2 * d)
    assert _fused(dry, [seg], 2, 0, T) == L.QKN_EOVERLAP
    # exactly in place: allowed
    seg = _seg(BASE, d, BASE + 64 * MB, BASE + 65 * MB, BASE, d, d, 2 * d)
    assert _fused(dry, [seg], 2, 0, T) == DRY
    # in place but a different stride: rejected
    seg = _seg(BASE, 2 * d, BASE + 64 * MB, BASE + 65 * MB, BASE, d, d, 2 * d)
    assert _fused(dry, [seg], 2, 0, T) == L.QKN_EOVERLAP
    # Q and K as column slices of one packed buffer, written in place: disjoint columns
    ld = 1024 + 256 + 256
    q = _seg(BASE, ld, BASE + 64 * MB, BASE + 65 * MB, BASE, ld, 1024, 4096)
    k = _seg(BASE + 2 * 1024, ld, BASE + 66 * MB, BASE + 67 * MB, BASE + 2 * 1024, ld, 256, 1024)
    assert _fused(dry, [q, k], 4, 3, T) == DRY
    # K's output written over Q's input columns: rejected
    k = _seg(BASE + 2 * 1024, ld, BASE + 66 * MB, BASE + 67 * MB, BASE + 2 * 512, ld, 256, 1024)
    assert _fused(dry, [q, k], 4, 3, T) == L.QKN_EOVERLAP
    # both segments sharing one partials array: their own slots collide
    q = _seg(BASE, d, BASE + 64 * MB, BASE + 65 * MB, BASE + 128 * MB, d, d, 2 * d)
    k = _seg(BASE + 256 * MB, 256, BASE + 300 * MB, BASE + 65 * MB, BASE + 400 * MB, 256, 256, 512)
    assert _fused(dry, [q, k], 2, 0, T) == L.QKN_EOVERLAP
    # ...but one array holding [2][tp][T] (disjoint per segment) is fine
    k = _seg(BASE + 256 * MB, 256, BASE + 300 * MB, BASE + 65 * MB + 2 * T * 4, BASE + 400 * MB,
             256, 256, 512)
    assert _fused(dry, [q, k], 2, 0, T) == DRY
    # inv_rms over the partials array
    q = _seg(BASE, d, BASE + 64 * MB, BASE + 65 * MB, BASE + 128 * MB, d, d, 2 * d,
             inv=BASE + 65 * MB + 8)
    assert _fused(dry, [q], 2, 0, T) == L.QKN_EOVERLAP
    # partial_out over x
    assert dry.qkn_partial_sumsq(BASE, d, T, d, BASE + 100, None) == L.QKN_EOVERLAP
    # y rows interleaved with x rows (same stride, column-disjoint): allowed
    seg = _seg(BASE, 2 * d, BASE + 64 * MB, BASE + 65 * MB, BASE + 2 * d, 2 * d, d, 2 * d)
    assert _fused(dry, [seg], 2, 0, T) == DRY
    # ...shifted by one column: overlaps
    seg = _seg(BASE, 2 * d, BASE + 64 * MB, BASE + 65 * MB, BASE + 2 * (d - 1), 2 * d, d, 2 * d)
    assert _fused(dry, [seg], 2, 0, T) == L.QKN_EOVERLAP


def test_options(lib):
    assert lib.qkn_set_option(b"waves_per_cu", 8) == 0
    assert lib.qkn_set_option(b"waves_per_cu", 0) == 0
    assert lib.qkn_set_option(b"waves_per_cu", -1) == L.QKN_EINVAL
    assert lib.qkn_set_option(b"waves_per_block", 5) == L.QKN_EINVAL
    assert lib.qkn_set_option(b"no_such_key", 1) == L.QKN_EINVAL
    assert lib.qkn_set_option(None, 1) == L.QKN_EINVAL


def test_struct_layouts_match_header(tmp_path):
    """ctypes mirrors of the C structs have the header's sizes and offsets."""
    import shutil
    import subprocess
    if not shutil.which("gcc"):
        pytest.skip("no C compiler")
    src = tmp_path / "layout.c"
    src.write_text('''#include <stdio.h>
#include <stddef.h>
#include "qkn_proj.h"
#define F(T, m) printf(#T "." #m " %zu\\n", offsetof(T, m))
int main(void) {
  printf("qkn_seg %zu\\n", sizeof(qkn_seg)); F(qkn_seg, x); F(qkn_seg, ldx); F(qkn_seg, w);
  F(qkn_seg, partials); F(qkn_seg, y); F(qkn_seg, ldy); F(qkn_seg, inv_rms);
  F(qkn_seg, d_local); F(qkn_seg, d_full);
  printf("qkn_seg8 %zu\\n", sizeof(qkn_seg8)); F(qkn_seg8, x); F(qkn_seg8, ldx); F(qkn_seg8, w);
  F(qkn_seg8, partials); F(qkn_seg8, y); F(qkn_seg8, ldy); F(qkn_seg8, inv_rms);
  F(qkn_seg8, d_local); F(qkn_seg8, d_full);
  printf("qkn_proj_seg %zu\\n", sizeof(qkn_proj_seg)); F(qkn_proj_seg, w); F(qkn_proj_seg, ldw);
  F(qkn_proj_seg, y); F(qkn_proj_seg, ldy); F(qkn_proj_seg, partials); F(qkn_proj_seg, d_local);
  printf("qkn_wait %zu\\n", sizeof(qkn_wait)); F(qkn_wait, slots); F(qkn_wait, epoch);
  F(qkn_wait, spin_limit); F(qkn_wait, co_resident); F(qkn_wait, status);
  printf("qkn_launch_info %zu\\n", sizeof(qkn_launch_info)); F(qkn_launch_info, kernel);
  F(qkn_launch_info, grid); F(qkn_launch_info, block); F(qkn_launch_info, waves);
  F(qkn_launch_info, lds_bytes);
  return 0;
}
''')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)],
                   check=True)
    c = dict(line.rsplit(" ", 1) for line in
             subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
             if line)
    for name, cls in (("qkn_seg", L.QknSeg), ("qkn_seg8", L.QknSeg), ("qkn_proj_seg", L.QknProjSeg),
                      ("qkn_wait", L.QknWait),
                      ("qkn_launch_info", L.QknLaunchInfo)):
        assert int(c[name]) == ctypes.sizeof(cls), name
        for field, _ in cls._fields_:
            assert int(c[f"{name}.{field}"]) == getattr(cls, field).offset, (name, field)


def _wait_block(**kw):
    base = dict(slots=(BASE + 512 * MB, BASE + 600 * MB), epoch=1, spin_limit=1000,
                co_resident=1, status=BASE + 700 * MB)
    base.update(kw)
    return L.QknWait((ctypes.c_void_p * 2)(*base["slots"]), base["epoch"], base["spin_limit"],
                     base["co_resident"], base["status"])


def _fused_wait(lib, segs, tp, rank, T, wait):
    arr = (L.QknSeg * len(segs))(*segs)
    return lib.qkn_fused_shard_wait(arr, len(segs), tp, rank, T, ctypes.c_float(1e-6),
                                    ctypes.byref(wait) if wait is not None else None, None)


def _q_nopart():
    q = _q()
    q.partials = None
    return q


def _k_nopart():
    k = _k()
    k.partials = None
    return k


def test_wait_entry_validation(dry):
    ok = _fused_wait(dry, [_q_nopart(), _k_nopart()], 4, 1, 64, _wait_block())
    assert ok == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_pa3<2,1>/fused_wait"  # publish three ahead
    for kw in (dict(epoch=0), dict(spin_limit=0), dict(co_resident=0), dict(status=None),
               dict(status=BASE + 700 * MB + 2), dict(slots=(None, BASE + 600 * MB)),
               dict(slots=(BASE + 512 * MB + 4, BASE + 600 * MB))):
        assert _fused_wait(dry, [_q_nopart(), _k_nopart()], 4, 1, 64, _wait_block(**kw)) == \
            L.QKN_EINVAL, kw
    assert _fused_wait(dry, [_q_nopart(), _k_nopart()], 4, 1, 64, None) == L.QKN_EINVAL
    # statistics must travel in the slots, not in partials
    assert _fused_wait(dry, [_q(), _k_nopart()], 4, 1, 64, _wait_block()) == L.QKN_EINVAL
    # slot arrays overlapping each other or an output
    assert _fused_wait(dry, [_q_nopart(), _k_nopart()], 4, 1, 64,
                       _wait_block(slots=(BASE + 512 * MB, BASE + 512 * MB + 64))) == L.QKN_EOVERLAP
    assert _fused_wait(dry, [_q_nopart(), _k_nopart()], 4, 1, 64,
                       _wait_block(slots=(BASE + 128 * MB, BASE + 600 * MB))) == L.QKN_EOVERLAP
    # outside the register path
    odd = _seg(BASE, 100, BASE + 64 * MB, None, BASE + 128 * MB, 100, 100, 400)
    assert _fused_wait(dry, [odd], 4, 1, 64, _wait_block()) == L.QKN_ENOTSUP
    # zero tokens: nothing to do
    assert _fused_wait(dry, [_q_nopart()], 4, 1, 0, _wait_block(status=None)) == 0


def test_wait_schedule_option(dry):
    try:
        for sched, prefix in ((0, "rows"), (1, "rows_pf"), (2, "rows_pa"), (3, "rows_pa2"),
                              (4, "rows_pa3")):
            assert dry.qkn_set_option(b"wait_schedule", sched) == 0
            assert _fused_wait(dry, [_q_nopart(), _k_nopart()], 4, 1, 64, _wait_block()) == DRY
            assert L.qkn_last_launch()["kernel"] == f"{prefix}<2,1>/fused_wait"
        # the option does not touch the kernels without a wait
        assert _fused(dry, [_q(), _k()], 4, 1, 64) == DRY
        assert L.qkn_last_launch()["kernel"] == "rows<2,1>/fused"
        assert dry.qkn_set_option(b"wait_schedule", 5) == L.QKN_EINVAL
        assert dry.qkn_set_option(b"wait_schedule", -1) == L.QKN_EINVAL
    finally:
        assert dry.qkn_set_option(b"wait_schedule", 4) == 0


def test_publish_entry_validation(dry):
    assert dry.qkn_publish_partials(BASE, 1024, 64, 1024, BASE + 512 * MB, 7, None) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows<2,0>/publish"
    assert dry.qkn_publish_partials(BASE, 1024, 64, 1024, BASE + 512 * MB, 0, None) == L.QKN_EINVAL
    assert dry.qkn_publish_partials(BASE, 1024, 64, 1024, BASE + 512 * MB + 4, 7, None) == L.QKN_EINVAL
    assert dry.qkn_publish_partials(None, 1024, 64, 1024, BASE + 512 * MB, 7, None) == L.QKN_EINVAL
    assert dry.qkn_publish_partials(BASE, 1024, 64, 1024, BASE + 64, 7, None) == L.QKN_EOVERLAP
    assert dry.qkn_publish_partials(BASE, 100, 64, 100, BASE + 512 * MB, 7, None) == L.QKN_ENOTSUP
    assert dry.qkn_publish_partials(BASE, 1024, 0, 1024, None, 0, None) == 0


def test_group_entry_validation(dry):
    T = 64

    def full(d_local, tp, ld=None):
        ld = ld or d_local * tp
        return _seg(BASE, ld, BASE + 64 * MB, None, BASE + 128 * MB, ld, d_local, d_local * tp)

    def call(segs, tp, wait):
        arr = (L.QknSeg * len(segs))(*segs)
        return dry.qkn_fused_group_wait(arr, len(segs), tp, T, ctypes.c_float(1e-6),
                                        ctypes.byref(wait), None)
    assert call([full(1024, 4)], 4, _wait_block()) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_pa3<2,0>/fused_wait"
    bad = full(1024, 4)
    bad.d_full = 4000
    assert call([bad], 4, _wait_block()) == L.QKN_EINVAL           # d_full != tp * d_local
    assert call([full(1024, 4, ld=2048)], 4, _wait_block()) == L.QKN_EINVAL  # ld < d_full
    withp = full(1024, 4)
    withp.partials = BASE + 900 * MB
    assert call([withp], 4, _wait_block()) == L.QKN_EINVAL
    # the slot array over the full x (T x 4096 bf16 = 512 KiB from BASE)
    assert call([full(1024, 4)], 4, _wait_block(slots=(BASE + 4096, None))) == L.QKN_EOVERLAP
    assert call([full(100, 4)], 4, _wait_block()) == L.QKN_ENOTSUP


# ------------------------------------------------------------------ FP8-E4M3

def _fused8(lib, segs, tp, rank, T, eps=1e-6):
    arr = (L.QknSeg * len(segs))(*segs)  # qkn_seg8 has qkn_seg's layout
    return lib.qkn_fused_shard_fp8(arr, len(segs), tp, rank, T, ctypes.c_float(eps), None)


@pytest.mark.parametrize("d,expect", [(16, "rows_fp8<1,0>"), (1024, "rows_fp8<1,0>"),
                                      (1040, "rows_fp8<2,0>"), (2048, "rows_fp8<2,0>"),
                                      (4096, "rows_fp8<4,0>"), (4112, "wide_fp8<8,0>"),
                                      (8192, "wide_fp8<8,0>"), (8208, "wide_fp8<16,0>"),
                                      (16384, "wide_fp8<16,0>"), (16400, "generic_fp8"),
                                      (8, "generic_fp8"), (1000, "generic_fp8")])
def test_fp8_path_choice_by_width(dry, d, expect):
    seg = _seg(BASE, d, BASE + 64 * MB, BASE + 65 * MB, BASE + 128 * MB, d, d, 2 * d)
    assert _fused8(dry, [seg], 2, 0, 16) == DRY
    name = L.qkn_last_launch()["kernel"]
    assert name.startswith(expect + ("/" if expect.startswith("generic") else "")), name


def test_fp8_entry_points_validate_like_bf16(dry):
    q = _seg(BASE, 2048, BASE + 64 * MB, BASE + 65 * MB, BASE + 128 * MB, 2048, 2048, 4096)
    k = _seg(BASE + 256 * MB, 512, BASE + 300 * MB, BASE + 301 * MB, BASE + 400 * MB, 512, 512, 1024)
    assert _fused8(dry, [q, k], 2, 1, 8192) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_fp8<2,1>/fused"
    assert dry.qkn_partial_sumsq_fp8(BASE, 2048, 64, 2048, BASE + 64 * MB, None) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_fp8<2,0>/partial"
    assert dry.qkn_apply_fp8(BASE, 2048, BASE + 64 * MB, BASE + 65 * MB, 2, 64, 2048, 4096,
                             ctypes.c_float(1e-6), BASE + 128 * MB, 2048, None, None) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_fp8<2,0>/apply"
    full = (L.QknSeg * 2)(_seg(BASE, 4096, BASE + 64 * MB, 0, BASE + 128 * MB, 4096, 4096, 4096),
                          _seg(BASE + 256 * MB, 1024, BASE + 300 * MB, 0, BASE + 400 * MB, 1024,
                               1024, 1024))
    assert dry.qkn_full_fp8(full, 2, 8192, ctypes.c_float(1e-6), None) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_fp8<4,1>/fused"
    # the prefetch option is a bf16-only variant; fp8 ignores it
    assert dry.qkn_set_option(b"prefetch", 1) == 0
    assert _fused8(dry, [q, k], 2, 1, 8192) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_fp8<2,1>/fused"
    # invalid arguments as for bf16
    assert _fused8(dry, [q, k], 2, 2, 64) == L.QKN_EINVAL
    assert _fused8(dry, [_seg(BASE, 2048, BASE + 64 * MB, 0, BASE + 128 * MB, 2048, 2048, 4096)],
                   2, 0, 64) == L.QKN_EINVAL  # partials NULL with tp > 1
    assert dry.qkn_full_fp8(full, 3, 8, ctypes.c_float(1e-6), None) == L.QKN_EINVAL
    assert dry.qkn_partial_sumsq_fp8(None, 8, 4, 8, BASE, None) == L.QKN_EINVAL
    assert dry.qkn_apply_fp8(BASE, 8, BASE + MB, None, 1, 4, 8, 8, ctypes.c_float(0.0),
                             BASE + 2 * MB, 8, None, None) == L.QKN_EINVAL


def test_fp8_alignment_and_overlap_in_bytes(dry):
    # a stride of 8 elements is 16-byte aligned for bf16 but not a whole fp8 chunk
    seg = _seg(BASE, 1032, BASE + 64 * MB, BASE + 65 * MB, BASE + 128 * MB, 1032, 1024, 2048)
    assert _fused8(dry, [seg], 2, 0, 16) == DRY
    assert L.qkn_last_launch()["kernel"] == "generic_fp8/fused"
    seg = _seg(BASE + 8, 1024, BASE + 64 * MB, BASE + 65 * MB, BASE + 128 * MB, 1024, 1024, 2048)
    assert _fused8(dry, [seg], 2, 0, 16) == DRY
    assert L.qkn_last_launch()["kernel"] == "generic_fp8/fused"
    # y directly after x (T rows of 1024 bytes) does not overlap; one byte earlier does
    T = 64
    x, y = BASE, BASE + T * 1024
    seg = _seg(x, 1024, BASE + 64 * MB, BASE + 65 * MB, y, 1024, 1024, 2048)
    assert _fused8(dry, [seg], 2, 0, T) == DRY
    seg = _seg(x, 1024, BASE + 64 * MB, BASE + 65 * MB, y - 1, 1024, 1024, 2048)
    assert _fused8(dry, [seg], 2, 0, T) == L.QKN_EOVERLAP
    # the bf16 entry sees the same y overlapping (2-byte elements)
    seg = _seg(x, 1024, BASE + 64 * MB, BASE + 65 * MB, y, 1024, 1024, 2048)
    assert _fused(dry, [seg], 2, 0, T) == L.QKN_EOVERLAP
    # in place is allowed
    seg = _seg(x, 1024, BASE + 64 * MB, BASE + 65 * MB, x, 1024, 1024, 2048)
    assert _fused8(dry, [seg], 2, 0, T) == DRY


# ------------------------------------------------------------------ projection

def _pseg(w, ldw, y, ldy, partials, d):
    return L.QknProjSeg(w, ldw, y, ldy, partials, d)


def _proj(lib, x, ldx, T, hidden, segs, ws, ws_bytes):
    arr = (L.QknProjSeg * len(segs))(*segs)
    return lib.qkn_proj_partial(x, ldx, T, hidden, arr, len(segs), ws, ws_bytes, None)


def test_proj_workspace_size(lib):
    segs = (L.QknProjSeg * 2)(_pseg(0, 0, 0, 0, 0, 2048), _pseg(0, 0, 0, 0, 0, 520))
    # many tiles: per-chunk statistics
    assert lib.qkn_proj_workspace_bytes(8192, 4096, segs, 2) == 4 * 8192 * (16 + 5)
    assert lib.qkn_proj_workspace_bytes(8192, 4096, segs, 1) == 4 * 8192 * 16
    # decode: one row tile -> 16 slices of 256 (row tiles x slices <= 16, slices >= 128
    # deep): the slices' fp32 sums
    def split_ws(T, splits, ncols, chunks):
        return 4 * splits * T * ncols
    assert lib.qkn_proj_workspace_bytes(64, 4096, segs, 2) == split_ws(64, 16, 2048 + 520, 21)
    assert lib.qkn_proj_workspace_bytes(64, 4096, segs, 1) == split_ws(64, 16, 2048, 16)
    # the slice count depends on T and hidden only
    assert lib.qkn_proj_workspace_bytes(300, 4096, segs, 2) == split_ws(300, 4, 2048 + 520, 21)
    assert lib.qkn_proj_workspace_bytes(1024, 4096, segs, 2) == split_ws(1024, 2, 2048 + 520, 21)
    assert lib.qkn_proj_workspace_bytes(1025, 4096, segs, 2) == 4 * 1025 * (16 + 5)
    # a shallow hidden caps the slices at 128 deep: 384 -> slices of 192 (three 64-wide stages)
    assert lib.qkn_proj_workspace_bytes(64, 384, segs, 2) == split_ws(64, 2, 2048 + 520, 21)
    assert lib.qkn_proj_workspace_bytes(64, 200, segs, 2) == 4 * 64 * (16 + 5)
    assert lib.qkn_proj_workspace_bytes(-1, 4096, segs, 1) == L.QKN_EINVAL
    assert lib.qkn_proj_workspace_bytes(8, 0, segs, 1) == L.QKN_EINVAL
    assert lib.qkn_proj_workspace_bytes(8, 4096, segs, 3) == L.QKN_EINVAL
    bad = (L.QknProjSeg * 1)(_pseg(0, 0, 0, 0, 0, 0))
    assert lib.qkn_proj_workspace_bytes(8, 4096, bad, 1) == L.QKN_EINVAL


def test_proj_validation(lib):
    T, h = 300, 4096
    X, W, Y, P, WS = BASE, BASE + 64 * MB, BASE + 128 * MB, BASE + 192 * MB, BASE + 200 * MB
    ok = _pseg(W, h, Y, 2048, P, 2048)
    need = lib.qkn_proj_workspace_bytes(T, h, (L.QknProjSeg * 1)(ok), 1)
    assert need > 4 * T * 16  # 3 row tiles: the split-k path
    # T == 0 is a no-op even with NULL pointers
    assert _proj(lib, None, h, 0, h, [ok], None, 0) == 0
    assert _proj(lib, X, h, T, h, [ok], WS, need - 4) == L.QKN_EINVAL          # workspace too small
    assert _proj(lib, X, h, T, h, [ok], None, need) == L.QKN_EINVAL            # no workspace
    assert _proj(lib, X, h - 8, T, h, [ok], WS, need) == L.QKN_EINVAL          # ldx < hidden
    assert _proj(lib, X, h, T, h, [_pseg(W, h - 8, Y, 2048, P, 2048)], WS, need) == L.QKN_EINVAL
    assert _proj(lib, X, h, T, h, [_pseg(W, h, Y, 2040, P, 2048)], WS, need) == L.QKN_EINVAL
    assert _proj(lib, X, h, T, h, [_pseg(W, h, Y, 2048, None, 2048)], WS, need) == L.QKN_EINVAL
    assert _proj(lib, X, h, T, h, [ok, ok, ok], WS, need) == L.QKN_EINVAL
    # alignment and multiples of 8 (the MFMA path)
    assert _proj(lib, X + 2, h, T, h, [ok], WS, need) == L.QKN_ENOTSUP
    assert _proj(lib, X, h + 4, T, h, [ok], WS, need) == L.QKN_ENOTSUP
    assert _proj(lib, X, 4100, T, 4100, [_pseg(W, 4100, Y, 2048, P, 2048)], WS, need) == L.QKN_ENOTSUP
    assert _proj(lib, X, h, T, h, [_pseg(W, h, Y, 2048, P, 2044)], WS, need) == L.QKN_ENOTSUP
    # overlaps: y onto x, partials onto y, workspace onto w; Q and K outputs as
    # disjoint column slices of one buffer are fine
    assert _proj(lib, X, h, T, h, [_pseg(W, h, X + 8192, 2048, P, 2048)], WS, need) == L.QKN_EOVERLAP
    assert _proj(lib, X, h, T, h, [_pseg(W, h, Y, 2048, Y + 64, 2048)], WS, need) == L.QKN_EOVERLAP
    assert _proj(lib, X, h, T, h, [ok], W + 4096, need) == L.QKN_EOVERLAP
    q = _pseg(W, h, Y, 2560, P, 2048)
    k = _pseg(W + 32 * MB, h, Y + 2048 * 2, 2560, P + MB, 512)
    need2 = lib.qkn_proj_workspace_bytes(T, h, (L.QknProjSeg * 2)(q, k), 2)
    assert dry_proj_ok(lib, X, h, T, h, [q, k], WS, need2)
    k_bad = _pseg(W + 32 * MB, h, Y + 2040 * 2, 2560, P + MB, 512)
    assert _proj(lib, X, h, T, h, [q, k_bad], WS, need2) == L.QKN_EOVERLAP


def dry_proj_ok(lib, *args):
    """Validation passes: with validate_only the call returns before any HIP call."""
    assert lib.qkn_set_option(b"validate_only", 1) == 0
    try:
        return _proj(lib, *args) == DRY
    finally:
        assert lib.qkn_set_option(b"validate_only", 0) == 0


def _proj_plan(lib, T, hidden, dims):
    """The kernel qkn_proj_partial chooses for these shapes (validate-only: planned for 256 CUs)."""
    X, W, Y, P, WS = BASE, BASE + 64 * MB, BASE + 1024 * MB, BASE + 2048 * MB, BASE + 3072 * MB
    segs = [_pseg(W + i * 256 * MB, hidden, Y + i * 256 * MB, d, P + i * MB, d)
            for i, d in enumerate(dims)]
    need = lib.qkn_proj_workspace_bytes(T, hidden, (L.QknProjSeg * len(segs))(*segs), len(segs))
    assert dry_proj_ok(lib, X, hidden, T, hidden, segs, WS, need)
    return L.qkn_last_launch()["kernel"]


def test_proj_plan(lib):
    # whole 128 x 128 tiles at prefill sizes
    assert _proj_plan(lib, 8192, 4096, (2048, 512)) == "proj<128x128,64,dl2,mi16>"
    assert _proj_plan(lib, 1025, 4096, (1024,)) == "proj<128x128,64,dl2,mi16>"
    # decode sizes split k, with 64-row tiles up to 64 tokens
    assert _proj_plan(lib, 64, 4096, (1024, 256)) == "proj<64x128,64,dl4,splitk>"
    assert _proj_plan(lib, 1, 4096, (1024,)) == "proj<64x128,64,dl4,splitk>"
    assert _proj_plan(lib, 65, 4096, (1024, 256)) == "proj<128x128,64,dl4,splitk>"
    assert _proj_plan(lib, 1024, 4096, (1024, 256)) == "proj<128x128,64,dl4,splitk>"
    # a forced kernel never splits
    assert lib.qkn_set_option(b"proj_tile", 2) == 0
    try:
        assert _proj_plan(lib, 8192, 4096, (2048, 512)) == "proj<128x128,64,reg>"
        assert _proj_plan(lib, 64, 4096, (1024, 256)) == "proj<128x128,64,reg>"
    finally:
        assert lib.qkn_set_option(b"proj_tile", 0) == 0
    assert lib.qkn_set_option(b"proj_tile", 3) == 0
    try:
        assert _proj_plan(lib, 8192, 4096, (2048, 512)) == "proj<128x128,64,dl2>"
    finally:
        assert lib.qkn_set_option(b"proj_tile", 0) == 0


def test_proj_tile_option(lib):
    for v in (0, 1, 2, 3):
        assert lib.qkn_set_option(b"proj_tile", v) == 0
    assert lib.qkn_set_option(b"proj_tile", 4) == L.QKN_EINVAL
    assert lib.qkn_set_option(b"proj_tile", -1) == L.QKN_EINVAL
    assert lib.qkn_set_option(b"proj_tile", 0) == 0


def test_calib_validation(dry):
    X, Y = BASE, BASE + 64 * MB
    assert dry.qkn_calib_copy(X, Y, 1 << 20, 2048, None) == DRY
    assert L.qkn_last_launch()["kernel"] == "calib_copy"
    assert dry.qkn_calib_copy(X, Y, 0, 2048, None) == 0                  # nothing to copy
    assert dry.qkn_calib_copy(X, Y, 24, 2048, None) == L.QKN_EINVAL      # not whole 16-byte vectors
    assert dry.qkn_calib_copy(X, Y, -16, 2048, None) == L.QKN_EINVAL
    assert dry.qkn_calib_copy(X, Y, 1 << 20, 0, None) == L.QKN_EINVAL
    assert dry.qkn_calib_copy(X, Y, 1 << 20, 65537, None) == L.QKN_EINVAL
    assert dry.qkn_calib_copy(X + 8, Y, 1 << 20, 2048, None) == L.QKN_EINVAL
    assert dry.qkn_calib_copy(None, Y, 1 << 20, 2048, None) == L.QKN_EINVAL
    assert dry.qkn_calib_copy(X, X + (1 << 19), 1 << 20, 2048, None) == L.QKN_EOVERLAP
    assert dry.qkn_calib_empty(None) == DRY
    assert L.qkn_last_launch()["kernel"] == "calib_empty"


def test_fp8_wait_entries(dry):
    # FP8 rows of 1024 codes: one 16-byte chunk per lane
    q = _seg(BASE, 1024, BASE + 64 * MB, None, BASE + 128 * MB, 1024, 1024, 4096)
    k = _seg(BASE + 256 * MB, 256, BASE + 300 * MB, None, BASE + 400 * MB, 256, 256, 1024)
    arr = (L.QknSeg * 2)(q, k)
    w = _wait_block()
    assert dry.qkn_fused_shard_wait_fp8(arr, 2, 4, 1, 64, ctypes.c_float(1e-6), ctypes.byref(w),
                                        None) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_pa3_fp8<1,1>/fused_wait"
    assert dry.qkn_publish_partials_fp8(BASE, 1024, 64, 1024, BASE + 512 * MB, 7, None) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_fp8<1,0>/publish"
    full = (L.QknSeg * 1)(_seg(BASE, 4096, BASE + 64 * MB, None, BASE + 128 * MB, 4096, 1024, 4096))
    assert dry.qkn_fused_group_wait_fp8(full, 1, 4, 64, ctypes.c_float(1e-6), ctypes.byref(w),
                                        None) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_pa3_fp8<1,0>/fused_wait"
    # the register path's limits are in bytes: 8 codes per row are not a 16-byte chunk
    odd = (L.QknSeg * 1)(_seg(BASE, 1032, BASE + 64 * MB, None, BASE + 128 * MB, 1032, 1032, 4128))
    assert dry.qkn_fused_shard_wait_fp8(odd, 1, 4, 1, 64, ctypes.c_float(1e-6), ctypes.byref(w),
                                        None) == L.QKN_ENOTSUP
    # validation as for bf16
    assert dry.qkn_publish_partials_fp8(BASE, 1024, 64, 1024, BASE + 512 * MB, 0, None) == L.QKN_EINVAL
    assert dry.qkn_fused_shard_wait_fp8(arr, 2, 4, 1, 64, ctypes.c_float(1e-6), None, None) == \
        L.QKN_EINVAL


def test_proj_size_limits(lib):
    """Byte offsets of the projection's buffer descriptors are 32-bit: x of
    2^31 bytes or more, or a weight slice that large, is not supported."""
    X, W, Y, P, WS = BASE, BASE + (8 << 30), BASE + (16 << 30), BASE + (24 << 30), BASE + (25 << 30)
    h = 4096
    ok = _pseg(W, h, Y, 2048, P, 2048)
    for T, expect in ((262143, 0), (262144, L.QKN_ENOTSUP)):  # T * 4096 * 2 bytes vs 2^31
        need = lib.qkn_proj_workspace_bytes(T, h, (L.QknProjSeg * 1)(ok), 1)
        if expect == 0:
            assert dry_proj_ok(lib, X, h, T, h, [ok], WS, need)
        else:
            assert _proj(lib, X, h, T, h, [ok], WS, need) == expect
    big = _pseg(W, h, Y, 262144, P, 262144)  # 262144 rows x 4096 x 2 bytes = 2^31
    need = lib.qkn_proj_workspace_bytes(64, h, (L.QknProjSeg * 1)(big), 1)
    assert _proj(lib, X, h, 64, h, [big], WS, need) == L.QKN_ENOTSUP


def test_wait_schedule_capped_for_the_widest_rows(dry):
    q = _seg(BASE, 4096, BASE + 64 * MB, None, BASE + 128 * MB, 4096, 4096, 8192)
    k = _seg(BASE + 256 * MB, 4096, BASE + 300 * MB, None, BASE + 400 * MB, 4096, 4096, 8192)
    assert _fused_wait(dry, [q, k], 2, 1, 64, _wait_block()) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_pf<8,8>/fused_wait"
    k2 = _seg(BASE + 256 * MB, 2048, BASE + 300 * MB, None, BASE + 400 * MB, 2048, 2048, 4096)
    assert _fused_wait(dry, [q, k2], 2, 1, 64, _wait_block()) == DRY
    assert L.qkn_last_launch()["kernel"] == "rows_pa3<8,4>/fused_wait"


def test_spin_limit_is_capped(dry):
    """A wait stays bounded whatever the caller asks: spin_limit above
    QKN_MAX_SPIN_LIMIT (2^22 polls) is rejected before anything is launched."""
    cap = 1 << 22
    segs = [_q_nopart(), _k_nopart()]
    assert _fused_wait(dry, segs, 4, 1, 64, _wait_block(spin_limit=cap)) == DRY
    assert _fused_wait(dry, segs, 4, 1, 64, _wait_block(spin_limit=cap + 1)) == L.QKN_EINVAL
    assert _fused_wait(dry, segs, 4, 1, 64, _wait_block(spin_limit=1 << 62)) == L.QKN_EINVAL
    full = (L.QknSeg * 1)(_seg(BASE, 4096, BASE + 64 * MB, None, BASE + 128 * MB, 4096, 1024, 4096))
    assert dry.qkn_fused_group_wait(full, 1, 4, 64, ctypes.c_float(1e-6),
                                    ctypes.byref(_wait_block(spin_limit=cap + 1)), None) == \
        L.QKN_EINVAL


def test_wait_slot_offsets_in_range(dry):
    """Flagged slots are 8 bytes: the waiting kernel addresses a token's slots
    by 32-bit byte offsets, so tp * T * 8 must stay below 2^31 (else
    QKN_ENOTSUP, never a launch whose offsets wrap)."""
    G = 1 << 38  # regions 256 GiB apart: x, y (128 GiB each) and the slot arrays fit
    tp = 4
    q = _seg(BASE, 1024, BASE + 3 * G, None, BASE + G, 1024, 1024, 4096)
    limit = (1 << 31) // (tp * 8)  # 2^26 tokens: tp * T = 2^28
    for T, expect in ((limit - 1, DRY), (limit, L.QKN_ENOTSUP)):
        w = _wait_block(slots=(BASE + 4 * G, BASE + 5 * G), status=BASE + 6 * G)
        assert _fused_wait(dry, [q], tp, 1, T, w) == expect, T
    # the statistics of the kernels without a wait are 4 bytes: twice the tokens
    qp = _seg(BASE, 1024, BASE + 3 * G, BASE + 4 * G, BASE + G, 1024, 1024, 4096)
    assert _fused(dry, [qp], tp, 1, limit) == DRY
    assert L.qkn_last_launch()["kernel"].startswith("rows")


def test_options_are_per_thread(lib):
    """A setting made in one thread does not reach another thread's launches:
    validate_only set here leaves a worker thread's calls launching normally
    (checked on validation-failing-free calls that stop at the first HIP query
    on this CPU-only machine), and a worker's settings do not come back."""
    import threading
    seg = _seg(BASE, 1024, BASE + 64 * MB, BASE + 65 * MB, BASE + 128 * MB, 1024, 1024, 2048)
    got = {}

    def worker():
        # no validate_only in this thread: the call goes on to the HIP runtime,
        # which has no device here (QKN_EHIP) -- or launches, where there is one
        got["rc"] = _fused(lib, [seg], 2, 0, 16)
        got["prefetch"] = lib.qkn_set_option(b"prefetch", 1)

    assert lib.qkn_set_option(b"validate_only", 1) == 0
    try:
        th = threading.Thread(target=worker)
        th.start()
        th.join()
        assert got["rc"] != DRY and got["prefetch"] == 0
        # this thread: still validate_only, and the worker's prefetch setting did not leak
        assert _fused(lib, [seg], 2, 0, 16) == DRY
        assert L.qkn_last_launch()["kernel"] == "rows<2,0>/fused"
    finally:
        assert lib.qkn_set_option(b"validate_only", 0) == 0


def test_proj_noalloc_validation(dry):
    """qkn_proj_partial_noalloc: the projection's checks, and a launch whose
    workspace exceeds the fixed QKN_PROJ_SCRATCH_BYTES (32 MiB) is rejected
    with QKN_ENOTSUP before any HIP call."""
    X, W, Y, P = BASE, BASE + 64 * MB, BASE + 1024 * MB, BASE + 2048 * MB

    def call(T, h, dims, x=X):
        segs = [_pseg(W + i * 256 * MB, h, Y + i * 256 * MB, d, P + i * MB, d)
                for i, d in enumerate(dims)]
        arr = (L.QknProjSeg * len(segs))(*segs)
        need = dry.qkn_proj_workspace_bytes(T, h, arr, len(segs))
        return dry.qkn_proj_partial_noalloc(x, h, T, h, arr, len(segs), None), need

    assert L.QKN_PROJ_SCRATCH_BYTES == 32 << 20
    rc, need = call(64, 4096, (1024, 256))   # decode: split-k slice sums, 5 MiB
    assert rc == DRY and need == 4 * 16 * 64 * 1280
    assert L.qkn_last_launch()["kernel"] == "proj<64x128,64,dl4,splitk>"
    rc, need = call(8192, 4096, (2048, 512))  # prefill: chunk statistics
    assert rc == DRY and L.qkn_last_launch()["kernel"] == "proj<128x128,64,dl2,mi16>"
    rc, need = call(1024, 4096, (4096, 1024))  # two slices over 5120 columns: 40 MiB
    assert need > L.QKN_PROJ_SCRATCH_BYTES and rc == L.QKN_ENOTSUP
    rc, _ = call(64, 4096, (1024, 256), x=None)
    assert rc == L.QKN_EINVAL
    rc, _ = call(0, 4096, (1024, 256), x=None)  # nothing to do
    assert rc == L.QKN_OK
