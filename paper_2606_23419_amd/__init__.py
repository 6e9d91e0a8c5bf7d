"""GRINQH nested-precision decode VMM for MI355X (gfx950).

``paper_2606_23419_amd.grinqh`` is the Python binding of libgrinqh.so (the
C ABI in include/grinqh.h); ``paper_2606_23419_amd.build`` compiles it.
Importing the binding without a built library raises: there is no fallback.
"""
