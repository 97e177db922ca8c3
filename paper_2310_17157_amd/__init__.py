"""Deja Vu (arXiv 2310.17157) decode hot path on AMD MI355X: HIP kernels behind a C ABI.

The compute lives in libdejavu_hip.so (built from csrc/ by `python -m
paper_2310_17157_amd.build`); `binding` is its ctypes binding with the C entry
point names. Importing this package does not load the library; the first call does,
and fails loudly if it has not been built.
"""
__all__ = ["binding", "accounting", "build"]
