"""Factorized sparse causal attention (Sparse Transformer) for MI355X / gfx950.

The compute lives in a C-ABI shared library of hand-written HIP kernels
(``csrc/``, declared in ``include/sparse_attn.h``).  ``sparse_attn`` is a thin
ctypes binding with the same entry-point names; PyTorch provides device memory
and streams only.  Import of this package does not load the library; the first
call does, and fails loudly if it has not been built.
"""
