"""AF1 binary-factorized linear layer on MI355X (gfx950).

The compute path lives in ``libaf1.so`` (hand-written HIP kernels behind a
C ABI declared in ``include/af1.h``); ``af1`` holds the thin Python binding.
"""
