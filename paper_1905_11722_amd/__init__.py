"""MI355X-native DP solver for the General Recomputation Problem of
Kusumoto et al. (NeurIPS 2019): lower-set families, the DP table fill and
the traceback run as HIP kernels for gfx950 behind the C ABI of
``include/rc.h``; ``rcdp`` is its Python binding and ``workloads`` holds
the seeded synthetic input graphs.

Importing the package loads nothing; ``rcdp.load_library()`` loads the
compiled library and raises when it is missing.
"""
