"""GPU: qkn_proj_partial_noalloc, the projection entry point for callers that
cannot allocate (its workspace is a fixed per-device array in the library).

Through the C ABI, against qkn_proj_partial with a caller's workspace: the
same kernels, so y and the statistics must be bit-identical. Two calls in a
row on the shared array, the second with fewer tokens, so the second call
runs over what the first left behind; both the split-k (decode-sized) and the
chunk-statistic (prefill-sized) workspace layouts are covered, in both
orders, and the projection oracle checks the outputs too.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workloads
from oracle import compare
from oracle import projection as P
from oracle import qknorm as Q
from paper_2608_09160_amd import _lib as L

from gpu_util import DEV, bits_of, to_dev_bf16

pytestmark = pytest.mark.gpu


def _inputs(T, hidden, dq, dk, seed):
    x = workloads.random_rows(seed, T, hidden, "normal")
    ws = [workloads.random_rows(seed + 1 + i, d, hidden, "normal", scale=hidden ** -0.5)
          for i, d in enumerate((dq, dk)) if d > 0]
    return x, ws


def _both(x_bits, w_bits, garbage_workspace=True):
    """The same projection through both entry points; the caller's workspace is
    filled with NaN bits first, so a read of an unwritten byte would show."""
    x = to_dev_bf16(x_bits)
    w_dev = [to_dev_bf16(w) for w in w_bits]
    ref_segs = [L.ProjSeg(w=w) for w in w_dev]
    need = L.qkn_proj_workspace_bytes(x.shape[0], x.shape[1], ref_segs)
    ws = torch.full((max(need, 16) // 4,), float("nan"), dtype=torch.float32,
                    device=DEV).view(torch.uint8)
    L.qkn_proj_partial(x, ref_segs, workspace=ws)
    ref_kernel = L.qkn_last_launch()["kernel"]
    # outputs allocated up front: the no-allocation call itself allocates nothing
    na_segs = [L.ProjSeg(w=w, y=torch.empty((x.shape[0], w.shape[0]), dtype=torch.bfloat16,
                                            device=DEV),
                         partials=torch.empty(x.shape[0], dtype=torch.float32, device=DEV))
               for w in w_dev]
    torch.cuda.synchronize()
    L.qkn_proj_partial_noalloc(x, na_segs)
    assert L.qkn_last_launch()["kernel"] == ref_kernel
    torch.cuda.synchronize()
    return ([(bits_of(s.y), s.partials.cpu().numpy()) for s in ref_segs],
            [(bits_of(s.y), s.partials.cpu().numpy()) for s in na_segs], ref_kernel, need)


def _check_oracle(x_bits, w, y_bits, part, what):
    hidden = x_bits.shape[1]
    q = P.project(x_bits, w)
    da = P.dot_abs(x_bits, w)
    compare.check_projection(Q.decode_bf16(y_bits), q, da, hidden, f"{what} y")
    ref = P.stored_partials(x_bits, w)
    bound = compare.projection_partial_bound(q, da, hidden)
    assert np.all(np.abs(part.astype(np.float64) - ref) <= bound), f"{what} partial"


# (T, hidden, Q columns, K columns): a larger call, then a smaller one
SEQUENCES = {
    "split_then_split": [(256, 5120, 640, 128), (64, 4096, 1024, 256)],
    "chunks_then_split": [(1500, 2048, 1024, 256), (200, 2048, 1024, 256)],
    "split_then_chunks": [(1024, 2048, 1536, 512), (1025, 1024, 512, 0)],
}


@pytest.mark.parametrize("name", list(SEQUENCES))
def test_noalloc_equals_workspace_entry_point(name):
    for i, (T, hidden, dq, dk) in enumerate(SEQUENCES[name]):
        print(f"[noalloc] {name} call {i}: T={T} hidden={hidden} q={dq} k={dk}", flush=True)
        x, ws = _inputs(T, hidden, dq, dk, 100 + 10 * i)
        ref, got, kernel, need = _both(x, ws)
        assert need <= L.QKN_PROJ_SCRATCH_BYTES
        for j, ((ry, rp), (gy, gp)) in enumerate(zip(ref, got)):
            assert np.array_equal(gy, ry), (name, i, j, kernel)
            assert np.array_equal(gp, rp), (name, i, j, kernel)
            _check_oracle(x, ws[j], gy, gp, f"{name} call {i} seg {j}")


def test_noalloc_rejects_a_workspace_beyond_its_size():
    # 1024 tokens split in two k-slices over 5120 columns: 4 * 2 * 1024 * 5120 bytes > 32 MiB
    x = torch.zeros((1024, 4096), dtype=torch.bfloat16, device=DEV)
    segs = [L.ProjSeg(w=torch.zeros((4096, 4096), dtype=torch.bfloat16, device=DEV)),
            L.ProjSeg(w=torch.zeros((1024, 4096), dtype=torch.bfloat16, device=DEV))]
    assert L.qkn_proj_workspace_bytes(1024, 4096, segs) > L.QKN_PROJ_SCRATCH_BYTES
    with pytest.raises(L.QknError) as e:
        L.qkn_proj_partial_noalloc(x, segs)
    assert e.value.status == L.QKN_ENOTSUP


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


@pytest.mark.parametrize("shape,other", [((64, 4096, 1024, 256), (300, 1024, 512, 128)),
                                         ((300, 1024, 512, 128), (64, 4096, 1024, 256))],
                         ids=["split_k", "chunk_statistics"])
def test_noalloc_graph_replays(shape, other):
    """The caller this entry point is for: a captured graph replayed while eager
    calls of another shape reuse the same fixed workspace in between. Every
    replay equals the eager result bit for bit and stays within the oracle's
    bounds. One eager call precedes the capture (it looks the array's address up)."""
    T, hidden, dq, dk = shape
    print(f"[noalloc graph] T={T} hidden={hidden} q={dq} k={dk}", flush=True)
    x_bits, w_bits = _inputs(T, hidden, dq, dk, 300)
    x = to_dev_bf16(x_bits)
    segs = [L.ProjSeg(w=to_dev_bf16(w), y=torch.empty((T, w.shape[0]), dtype=torch.bfloat16,
                                                     device=DEV),
                      partials=torch.empty(T, dtype=torch.float32, device=DEV)) for w in w_bits]
    oT, oh, oq, ok = other
    ox_bits, ow_bits = _inputs(oT, oh, oq, ok, 400)
    ox = to_dev_bf16(ox_bits)
    osegs = [L.ProjSeg(w=to_dev_bf16(w), y=torch.empty((oT, w.shape[0]), dtype=torch.bfloat16,
                                                       device=DEV),
                       partials=torch.empty(oT, dtype=torch.float32, device=DEV))
             for w in ow_bits]

    def call():
        L.qkn_proj_partial_noalloc(x, segs)

    call()
    torch.cuda.synchronize()
    ref = [(bits_of(s.y), s.partials.cpu().numpy()) for s in segs]
    for j, (y, part) in enumerate(ref):
        _check_oracle(x_bits, w_bits[j], y, part, f"eager seg {j}")
    g = _graph_of(call)
    for r in range(4):
        for s in segs:
            s.y.view(torch.uint8).fill_(0x5A)
            s.partials.fill_(float(r + 1))
        L.qkn_proj_partial_noalloc(ox, osegs)  # eager work over the same workspace
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for j, (s, (ry, rp)) in enumerate(zip(segs, ref)):
            gy, gp = bits_of(s.y), s.partials.cpu().numpy()
            assert np.array_equal(gy, ry), (r, j)
            assert np.array_equal(gp, rp), (r, j)
            if r in (0, 3):
                _check_oracle(x_bits, w_bits[j], gy, gp, f"replay {r} seg {j}")
