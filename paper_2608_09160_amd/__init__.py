"""Sharded layerwise QK-Norm for AMD MI355X: HIP kernels behind a C ABI.

The computation lives in ``libqkn.so`` (``csrc/qkn.hip``, declared in
``include/qkn.h``); ``_lib`` is its ctypes binding. Build with
``python -m paper_2608_09160_amd.build``.
"""
from ._lib import (QKN_EHIP, QKN_EINVAL, QKN_EOVERLAP, QKN_OK, Prepared, QknError, Seg,  # noqa: F401
                   load, qkn_apply, qkn_full, qkn_fused_shard, qkn_last_launch,
                   qkn_partial_sumsq, qkn_set_option, qkn_strerror)
