"""libhadacore: batched normalized Walsh-Hadamard transform for MI355X (gfx950).

The transform runs in hand-written HIP kernels behind a C ABI
(``include/hadacore.h``); ``hadacore`` is the thin ctypes binding and
``workloads`` holds the seeded synthetic inputs.
"""
