"""CPU oracle for the pooled EmbeddingBag forward — TEST INFRASTRUCTURE.

Only tests/, the smoke check in __graft_entry__ and the CPU-baseline leg of
bench.py may import this package.  The product path (libeb and its binding)
never does.  The arithmetic lives in eb_oracle.c (plain C, fp64
accumulation); this module only marshals numpy arrays into it.
"""
from .oracle import (OracleError, OracleTable, build, double_to_half, ebo_backward_update, ebo_fm, ebo_forward,
                     ebo_forward_seq, half_to_double, lib_path, max_threads)

__all__ = ["OracleError", "OracleTable", "build", "double_to_half", "ebo_backward_update", "ebo_fm", "ebo_forward",
           "ebo_forward_seq", "half_to_double", "lib_path", "max_threads"]
