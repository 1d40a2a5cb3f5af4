"""Reuse-aware ViT encoder (DejaVu / ReuseViT hot path) for AMD Instinct MI355X.

The computation lives in ``_lib/libdejavu.so`` (HIP kernels for gfx950 behind a C ABI
declared in ``include/dejavu.h``); ``dejavu`` is its Python binding.
"""
