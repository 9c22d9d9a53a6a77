"""MI355X-native AVTP pruning-layer operator.

The compute path lives in ``libavtp.so`` (hand-written HIP kernels for gfx950
behind a C ABI, declared in ``include/avtp.h``); ``paper_2608_26806_amd.avtp``
is the ctypes binding.  ``paper_2608_26806_amd.workloads`` draws the seeded
synthetic inputs.  Importing the package loads nothing.
"""
