"""MI355X (gfx950) tree-verification hot path of DREAM-S speculative decoding.

The compute lives in the HIP library ``libdreams.so`` (C ABI declared in include/dreams.h); the binding in
:mod:`paper_2606_00535_amd.dreams` only marshals arguments.  Importing this package loads nothing.
"""
