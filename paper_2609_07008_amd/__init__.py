"""MLA-Online step of RedKnot-MLA (arXiv 2609.07008) for AMD MI355X (gfx950).

The computation lives in libmla_online.so (C ABI, include/mla_online.h); the
Python modules only marshal arguments: `mla` (ctypes binding) and `step`
(buffers for one attend -> merge -> o-proj step).  Importing the submodules
loads the library; this package init imports nothing heavy.
"""
__all__ = ["mla", "step", "build"]
