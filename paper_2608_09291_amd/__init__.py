"""UnionSparse W4A4 IE-BME SpMM, native to MI355X (gfx950).

The compute path lives in the HIP/C++ shared library built from ``csrc/``;
``binding`` marshals arguments to its C-ABI. Importing this package loads
nothing; the library is loaded on first use and its absence is an error.
"""
__all__ = ["binding", "synth"]
