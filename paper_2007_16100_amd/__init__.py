"""SPVConv hot path (arXiv 2007.16100, Sec. 3.3) on AMD Instinct MI355X.

The compute lives in ``libspv.so`` (hand-written HIP for gfx950, C ABI in
``include/spv.h``); ``spv`` is its ctypes binding and ``synth`` draws the seeded
synthetic inputs.
"""
