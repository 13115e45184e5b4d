"""CPU oracle of the recomputation DP -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use this package.  It shares no code with the GPU library.
"""
