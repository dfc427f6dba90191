"""MI355X (gfx950) PVS dense channel and exact adaptive hybrid retrieval.

The compute path lives in ``libeahr.so`` (HIP kernels + a C ABI declared in
``include/eahr.h``); :mod:`paper_2608_07152_amd.eahr` is the thin ctypes
binding.  Importing this package does not load the library, so the data
generator (:mod:`paper_2608_07152_amd.datagen`) stays usable without it.
"""
