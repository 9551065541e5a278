"""GPU: the measurement references (qkn_calib_copy, qkn_calib_empty).

The streaming copy must reproduce its input byte for byte for sizes that do
and do not divide the grid's stride, with few and many workgroups."""
from __future__ import annotations

import pytest
import torch

from paper_2608_09160_amd import _lib as L

from gpu_util import DEV

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nbytes,blocks", [(16, 1), (4096, 3), (1 << 20, 2048), ((1 << 22) + 48, 4096),
                                           (48, 65536)])
def test_copy_is_exact(nbytes, blocks):
    g = torch.Generator().manual_seed(nbytes)
    x = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, generator=g).to(DEV)
    y = torch.zeros(nbytes + 64, dtype=torch.uint8, device=DEV)
    print(f"[calib] copy {nbytes} B with {blocks} workgroups", flush=True)
    L.qkn_calib_copy(x, y[:nbytes], blocks=blocks)
    torch.cuda.synchronize()
    assert torch.equal(x, y[:nbytes])
    assert not y[nbytes:].any()  # nothing written past the end


def test_empty_kernel_runs():
    for _ in range(10):
        L.qkn_calib_empty()
    torch.cuda.synchronize()
    assert L.qkn_last_launch()["kernel"] == "calib_empty"
