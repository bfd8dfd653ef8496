"""Integer-only I-LW-DETR encoder block and deformable sampling on MI355X.

The compute path is the HIP library ``libilw.so`` (hand-written gfx950
kernels behind a C ABI declared in ``include/ilw.h``).  ``ilw`` is its thin
ctypes binding; ``synth`` draws the seeded synthetic inputs.
"""
__all__ = ["ilw", "synth"]
