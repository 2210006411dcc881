"""MI355X-native per-layer paged KV-cache pack/unpack (TopKV hot path).

The compute path is ``libtopkv.so`` (HIP kernels for gfx950 behind a C ABI,
declared in ``include/topkv.h``); :mod:`paper_2607_28633_amd.topkv` is its thin
ctypes binding.  :mod:`paper_2607_28633_amd.workloads` draws seeded synthetic
inputs.  Importing this package does not load the library; importing the
binding does, and fails loudly if it is missing.
"""
