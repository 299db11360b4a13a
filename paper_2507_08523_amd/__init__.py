"""MI355X-native prefix-cached paged prefill attention (InferLog hot path).

The library behind this package is ``libilpc.so`` (host prefix cache in C++,
paged K/V append and paged prefill/decode attention as HIP kernels for
gfx950), reached through a C ABI declared in ``include/ilpc.h``.  The Python
side only marshals arguments: ``paper_2507_08523_amd.ilpc`` loads the library
and raises if it is missing -- there is no fallback path.

``paper_2507_08523_amd.workload`` builds seeded synthetic log-parsing batches.
Importing this package loads nothing.
"""
