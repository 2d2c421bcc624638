"""CPU oracle for UnionSparse's W4A4 IE-BME SpMM: TEST INFRASTRUCTURE ONLY.

A plain, slow, independent restatement of what the paper's hot path computes:
the IE-BME encoding and decoding (Section V-A), bitmap-aware row reordering
(Section V-B, Eq. 3-5), the LSPD index equations
(Section VI-B), the Payload-to-Metadata Ratio and effective compute intensity
(Eq. 1, Eq. 2) with its cross-format comparison, and the int64 masked dense
product. It shares no code, header
or table with the HIP library, and imports nothing from it.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import, call, link or execute anything in this package. The
product path never does.
"""
from . import formats, iebme, product, reorder  # noqa: F401
