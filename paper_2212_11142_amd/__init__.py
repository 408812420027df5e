"""BaCO GP + EI candidate scoring on MI355X (gfx950).

``paper_2212_11142_amd.gp`` is the ctypes binding of the HIP library built from
``csrc/`` (``build.build()``); see ``include/baco_gp.h`` for the C-ABI.
"""
__all__ = ["gp", "build"]
