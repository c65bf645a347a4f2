"""MI355X-native scoring and per-pressure-level selection of workflow physical plans.

The compute path is the HIP library ``libdyplan.so`` (kernels for gfx950 behind
the C-ABI declared in ``include/dyplan.h``); ``dyplan`` is its ctypes binding and
``workload`` the seeded generator of paper-shaped synthetic inputs.
"""
