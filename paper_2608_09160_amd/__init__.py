"""Sharded layerwise QK-Norm for AMD MI355X: HIP kernels behind a C ABI.

The computation lives in ``libqkn.so`` (kernels in ``csrc/qkn_kernels.h`` and
``csrc/qkn_proj.hip``, entry points declared in ``include/qkn.h`` and
``include/qkn_proj.h``); ``_lib`` is its ctypes binding. Build with
``python -m paper_2608_09160_amd.build``.
"""
from ._lib import (QKN_EHIP, QKN_EINVAL, QKN_ENOTSUP, QKN_EOVERLAP, QKN_OK,  # noqa: F401
                   Prepared, PreparedApply, PreparedPartial, QknError, Seg, load, qkn_apply, qkn_full, qkn_fused_shard,
                   qkn_fused_group_wait, qkn_fused_shard_wait, qkn_last_launch, qkn_partial_sumsq,
                   qkn_publish_partials, qkn_set_option, qkn_strerror)
