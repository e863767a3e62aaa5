"""Batched flow-matching action-chunk generation on AMD MI355X (gfx950).

The product is the HIP library ``librosa.so`` with the C ABI in
``include/rosa.h``; ``rosa`` is its Python binding.
"""
__all__ = ["rosa"]
