"""ORACLE -- test infrastructure, not product code.

Python access to the plain fp64 CPU reference in ``adpsgd_oracle.c`` and to the
tiny pure-Python reference in ``tiny_ref.py``.  Only the tests, the smoke check
and the bench's CPU-baseline leg may import this package.  It imports nothing
from the GPU package; both sides take their inputs from ``workloads``.
"""
from .oracle import (  # noqa: F401
    Oracle, OracleRun, build_oracle, lib_path, philox4x32_10, normals4, problem_data,
    lr, controller_trace, num_threads, box_muller, philox_groups, normals_groups,
)
