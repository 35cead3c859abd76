"""MI355X (gfx950) decode-step Attention/FFN operators of disaggregated A/F serving.

The compute path is the C-ABI library ``libaflex.so`` built from ``csrc/``;
``aflex`` is its Python binding and ``synth`` the seeded input generator.
Importing the package loads nothing; ``aflex.load()`` opens the library and
raises if it has not been built.
"""
__all__ = ["aflex", "synth"]
