"""Barrier-free synchronization of loop-nested multi-engine kernels on MI355X.

The product is the C-ABI library ``libbfs.so`` (header ``include/bfs.h``):
a host planner for the thresholds of the paper's per-loop allocation and HIP
kernels for gfx950 whose engines are specialised wavefronts synchronising
through LDS counters.  ``bfs`` is the thin ctypes binding."""
from .bfs import (ALLOC_PER_ENGINE, ALLOC_PER_INSTR, ALLOC_PER_LOOP, KASE_FALLBACK, MODE_BARRIER, MODE_BARRIER_FREE,  # noqa: F401
                  BfsError, Plan, lib, parse_debug_log)
