"""fp64 CPU oracle for sharded layerwise QK-Norm -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, the smoke check in ``__graft_entry__`` and the CPU-baseline leg
of ``bench.py`` may import this package. It shares no code with the HIP library
in ``paper_2608_09160_amd``, and the library never imports it.
"""
from . import compare, qknorm  # noqa: F401
