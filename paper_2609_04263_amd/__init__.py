"""MI355X-native packed low-bit KV-cache decode path.

Hot path of "Quality Recovery for Quantized KV Caches via Low-Rank Attention
Adaptation": the adapted Q/K/V projection (Sec. 3, Eq. (1)-(2)), quantize-and-
pack append into a physically packed incremental cache (Sec. 3.1, Eq. (3)),
and decode attention over the in-kernel reconstruction (Sec. 3.1-3.2).

The compute lives in hand-written HIP kernels for gfx950 behind the C ABI of
``include/kvq.h`` (``libkvq.so``); :mod:`paper_2609_04263_amd.kvq` is the thin
ctypes binding.  Importing this package does not load the GPU library;
importing :mod:`paper_2609_04263_amd.kvq` does, and fails loudly if it is
missing.
"""
