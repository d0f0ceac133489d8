"""DeepPCR on MI355X: Newton + Parallel Cyclic Reduction for deep sequential
networks, as a C-ABI HIP library (libdeeppcr.so) with a thin ctypes binding.

The binding (``paper_2309_16318_amd.deeppcr``) loads the library on first
use and raises if it is missing; there is no CPU fallback.
"""
