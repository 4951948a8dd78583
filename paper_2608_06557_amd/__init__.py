"""MI355X-native Cascade scheduling step (arXiv 2608.06557).

The compute path lives in ``libcascade.so`` (hand-written gfx950 HIP kernels
behind a C ABI, see ``include/cascade.h``); ``paper_2608_06557_amd.cascade``
is its thin ctypes binding and loads the library on first use.
``paper_2608_06557_amd.synth`` draws the seeded synthetic workloads.
"""
