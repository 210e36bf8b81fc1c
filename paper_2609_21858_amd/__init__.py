"""Keyed Poisson-race multi-draft speculative sampling on MI355X (gfx950).

The sampler lives in the HIP library ``lib/libpsd.so`` (C ABI: include/psd.h);
``paper_2609_21858_amd.psd`` is its thin ctypes binding.  Build with
``paper_2609_21858_amd.build.build()`` (hipcc, gfx950).
"""
__all__ = ["psd", "build"]
