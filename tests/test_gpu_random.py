"""GPU parity on seeded random shapes: the fused, Phase A and Phase B+C entry
points and the projection, over random token counts, widths, tp, ranks, row
strides, column offsets (misaligned slices), eps and formats; these seeds
reach the register, wide and general paths of both formats and every
projection kernel (the launch chosen is printed per case). Each case
checks the fused kernel against the oracle's Phase A sum and Phase B factor
(oracle/qknorm.py) with the simulated peers' statistics as given, the
two-launch path against the fused one bit for bit, and the projection
against the fp64 product within the oracle's rounding bound."""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import workloads
from oracle import compare
from oracle import projection as P
from oracle import qknorm as Q
from paper_2608_09160_amd import _lib as L

from gpu_util import DEV, bits_of

pytestmark = pytest.mark.gpu


def _act(rng, T, d, fmt, pad, off):
    v = (rng.standard_normal((T, d + pad + off)) * np.exp(rng.normal(0, 0.7, (T, 1)))).astype(np.float32)
    if fmt == "fp8":
        b = Q.encode_e4m3(np.clip(v, -448, 448).astype(np.float64)).astype(np.uint8)
        full = torch.from_numpy(b).to(DEV).view(torch.float8_e4m3fn)
    else:
        b = workloads.f32_to_bf16_bits(v)
        full = torch.from_numpy(b.view(np.int16)).to(DEV).view(torch.bfloat16)
    return full[:, off:off + d], Q.decode(b, fmt)[:, off:off + d]


def _norm_case(rng, aligned):
    fmt = "fp8" if rng.random() < 0.4 else "bf16"
    tp = int(rng.choice([1, 2, 3, 4, 8, 16]))
    rank = int(rng.integers(0, tp))
    T = int(math.exp(rng.uniform(0, math.log(1500))))
    nseg = 2 if rng.random() < 0.8 else 1
    if aligned:
        widths = [int(rng.integers(1, 1025)) * 8, int(rng.integers(1, 257)) * 8][:nseg]
    else:
        widths = [int(rng.integers(1, 6000)), int(rng.integers(1, 1500))][:nseg]
    eps = float(rng.choice([0.0, 1e-6, 1e-2]))
    return fmt, tp, rank, T, widths, eps


@pytest.mark.parametrize("seed", range(8))
def test_random_norm_cases(seed):
    rng = np.random.default_rng(1000 + seed)
    for case in range(6):
        aligned = case % 2 == 0
        fmt, tp, rank, T, widths, eps = _norm_case(rng, aligned)
        desc = f"seed {seed} case {case}: {fmt} T={T} tp={tp} rank={rank} widths={widths} eps={eps}"
        print(f"[random] {desc}", flush=True)
        segs, refs = [], []
        for d in widths:
            pad = 8 * int(rng.integers(0, 5)) if aligned else int(rng.integers(0, 40))
            off = 0 if aligned else int(rng.integers(0, 9))
            x, xd = _act(rng, T, d, fmt, pad, off)
            g = rng.uniform(0.5, 1.5, d).astype(np.float32)
            d_full = d * tp + (0 if rng.random() < 0.8 else int(rng.integers(1, 100)))
            peers = (np.abs(rng.standard_normal((tp, T))) * d + 1e-3).astype(np.float32)
            own = Q.sum_of_squares(xd)
            S = peers.astype(np.float64)
            S[rank] = own
            inv = Q.rms_factor(S.sum(axis=0), d_full, eps)
            y = xd * inv[:, None] * g.astype(np.float64)[None, :]
            segs.append(L.Seg(x=x, w=torch.from_numpy(g).to(DEV), d_full=d_full,
                              partials=torch.from_numpy(peers).to(DEV),
                              inv_rms=torch.empty(T, dtype=torch.float32, device=DEV)))
            refs.append((own, inv, y, d_full))
        (L.qkn_fused_shard_fp8 if fmt == "fp8" else L.qkn_fused_shard)(segs, tp, rank, eps)
        print(f"[random]   {L.qkn_last_launch()['kernel']}", flush=True)
        torch.cuda.synchronize()
        for i, (s, (own, inv, y, d_full)) in enumerate(zip(segs, refs)):
            compare.check_close(s.partials[rank].cpu().numpy(), own, compare.PARTIAL_RTOL,
                                f"{desc} seg{i} partial")
            compare.check_close(s.inv_rms.cpu().numpy(), inv, 1e-5, f"{desc} seg{i} inv")
            yb = bits_of(s.y)
            if fmt == "fp8":
                compare.check_fp8(Q.decode_e4m3(yb), y, f"{desc} seg{i} y")
            else:
                compare.check_close(Q.decode_bf16(yb), y, compare.OUTPUT_RTOL, f"{desc} seg{i} y")
            alone = (L.qkn_partial_sumsq_fp8 if fmt == "fp8" else L.qkn_partial_sumsq)(s.x)
            assert np.array_equal(alone.cpu().numpy(), s.partials[rank].cpu().numpy()), desc
            y2 = (L.qkn_apply_fp8 if fmt == "fp8" else L.qkn_apply)(s.x, s.w, s.partials, d_full, eps)
            torch.cuda.synchronize()
            assert np.array_equal(bits_of(y2), yb), desc


@pytest.mark.parametrize("seed", range(4))
def test_random_projection_cases(seed):
    rng = np.random.default_rng(2000 + seed)
    for case in range(6):
        T = int(math.exp(rng.uniform(0, math.log(1500))))
        hidden = int(rng.integers(1, 257)) * 8
        ds = [int(rng.integers(1, 151)) * 8 for _ in range(1 if rng.random() < 0.3 else 2)]
        tile = int(rng.choice([0, 0, 1, 2, 3]))
        desc = f"seed {seed} case {case}: T={T} hidden={hidden} ds={ds} proj_tile={tile}"
        print(f"[random] {desc}", flush=True)
        xb = workloads.f32_to_bf16_bits(rng.standard_normal((T, hidden), dtype=np.float32))
        wbs = [workloads.f32_to_bf16_bits((rng.standard_normal((d, hidden)) / math.sqrt(hidden))
                                          .astype(np.float32)) for d in ds]
        x = torch.from_numpy(xb.view(np.int16)).to(DEV).view(torch.bfloat16)
        ws = [torch.from_numpy(w.view(np.int16)).to(DEV).view(torch.bfloat16) for w in wbs]
        L.qkn_set_option("proj_tile", tile)
        try:
            segs = [L.ProjSeg(w=w) for w in ws]
            L.qkn_proj_partial(x, segs)
            print(f"[random]   {L.qkn_last_launch()['kernel']}", flush=True)
            torch.cuda.synchronize()
        finally:
            L.qkn_set_option("proj_tile", 0)
        for i, (s, wb) in enumerate(zip(segs, wbs)):
            _check_projection(xb, wb, bits_of(s.y), s.partials.cpu().numpy(), f"{desc} seg{i}")


def _check_projection(x_bits, w_bits, y_bits, part, what):
    """The oracle's projection bounds (as in test_gpu_proj.py)."""
    hidden = x_bits.shape[1]
    q = P.project(x_bits, w_bits)
    da = P.dot_abs(x_bits, w_bits)
    yv = Q.decode_bf16(y_bits)
    compare.check_projection(yv, q, da, hidden, f"{what} y")
    ref = P.stored_partials(x_bits, w_bits)
    err = np.abs(part.astype(np.float64) - ref)
    assert np.all(err <= compare.projection_partial_bound(q, da, hidden)), f"{what} statistic"
    compare.check_close(part, np.sum(yv * yv, axis=1), compare.PARTIAL_RTOL,
                        f"{what} statistic vs stored row")
