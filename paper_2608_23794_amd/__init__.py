"""MI355X-native Mixture of Channel Experts forward pass.

The compute path is the HIP library ``libmoce.so`` (hand-written gfx950
kernels behind a C ABI declared in ``include/moce.h``); ``binding`` marshals
arguments to it through ctypes.  ``inputs`` draws seeded synthetic workloads
and ``cost`` holds the layer's cost and traffic accounting.
"""
