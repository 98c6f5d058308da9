"""CPU oracle for the barrier-free synchronization path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  It shares no code
with the GPU library (``paper_2608_13757_amd``) and never imports it.

* ``core``    -- sequential program-order walk, Eq. (1) brute-force thresholds,
                 per-loop semaphore thresholds, barrier-scheme thresholds and
                 fp64 tile-machine values (plain C, ``bfs_oracle.c``).
* ``hazard``  -- happens-before coverage check of a dependency graph.
* ``mathref`` -- plain fp64 definitions of the fused MFMA workloads.
"""
