"""Mirror-SD verification step, native on MI355X (gfx950).

The product is ``libmsd.so`` (hand-written HIP kernels behind the C ABI in
``include/msd.h``); ``paper_2510_13161_amd.msd`` is its thin Python binding.
Submodules are imported lazily so that CPU-only users (the input generator)
do not load the HIP library.
"""
__all__ = ["msd", "synth", "build"]
