"""MI355X (gfx950) multimodal text-encoder prefill: HIP kernels behind a C ABI.

``binding`` mirrors include/mte.h one to one; ``encoder`` wraps it for torch
tensors; ``build`` compiles libmte.so. Importing ``binding`` or ``encoder``
requires the built library.
"""
