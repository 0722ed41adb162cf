"""fp64 CPU oracle for the HSA forward pass (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.
"""
from . import hsa_oracle  # noqa: F401
