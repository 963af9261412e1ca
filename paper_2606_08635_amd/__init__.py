"""SpectrumKV per-token mixed-precision KV transfer codec for MI355X (gfx950).

The codec (arXiv 2606.08635) scores prompt tokens, assigns each one an fp16,
int8 or int4 tier (or drops it) under a normalized byte budget, packs K/V
into one compacted payload and, on the decode side, dequantizes the payload
into an fp16 paged cache.  Every step runs in the HIP kernels of ``libskv.so``;
``paper_2606_08635_amd.skv`` is the ctypes binding over its C ABI
(``include/skv.h``).  Importing this package does not load the library; the
binding loads it on first use and raises if it is missing.
"""
