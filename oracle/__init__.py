"""CPU oracle for the Celeritas placement hot path (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may use this package.  The product path never imports it.
"""
