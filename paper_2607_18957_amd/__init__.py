"""Merged tensor loading for AMD MI355X (gfx950).

The device path lives in the C-ABI library ``libii.so`` built from ``csrc/``;
``paper_2607_18957_amd.ii`` is its Python binding. Importing this package does
not load the library, so the input generators in ``synth`` can be used on a
machine without the built extension.
"""

__all__ = ["ii", "synth"]
