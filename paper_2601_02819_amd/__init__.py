"""PHSA (Punctuation-aware Hybrid Sparse Attention) for AMD MI355X (gfx950).

The compute lives in ``libphsa.so`` (hand-written HIP kernels behind a C ABI,
declared in ``include/phsa.h``); :mod:`paper_2601_02819_amd.phsa` is a thin
ctypes binding over it that passes torch device pointers and streams.
"""
