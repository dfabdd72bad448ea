"""MI355X-native speculative-verification hot path (append KV, verify attention, accept).

The compute lives in libspexis.so (HIP kernels for gfx950 behind a C ABI, include/spexis.h);
``spexis`` is its Python binding, ``step`` chains the three calls, ``workloads`` draws the
seeded synthetic inputs.  Importing the package loads nothing.
"""
