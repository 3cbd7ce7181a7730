"""MI355X-native W8A8 SmoothQuant hot path (arxiv 2608.28003).

The compute lives in a C-ABI shared library of hand-written HIP kernels for
gfx950 (``libw8a8.so``, declared in ``include/w8a8.h``).  ``paper_2608_28003_amd.w8a8``
is the thin ctypes binding; it loads the library on first use and raises if it
is missing.  ``paper_2608_28003_amd.synth`` draws the seeded synthetic inputs.
"""
