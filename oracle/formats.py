"""Oracle for the cross-format byte accounting (TEST INFRASTRUCTURE ONLY).

Section III-B defines the Payload-to-Metadata Ratio (Eq. 1) and compares it
across precisions (FP16, INT8, INT4) and sparse formats; Section III-C turns
it into an effective compute intensity (Eq. 2). Here every format's arrays
are built explicitly from the dense matrix and their sizes are counted:

  * dense: every weight, no metadata;
  * CSR: scipy's compressed-sparse-row arrays, with 32-bit column indices and
    M + 1 32-bit row pointers;
  * per-area bitmaps: for every 8 x 32 area of every 16 x 64 LT, a 256-bit
    bitmap of its own nonzeros and a 32-bit offset, values of nonzeros only;
  * IE-BME: the oracle encoder of Section V-A (one union bitmap per LT shared
    by its four areas, zeros of active groups stored).

Only ``tests/`` may use this module. It shares no code with the library.
"""
from __future__ import annotations

import numpy as np
import scipy.sparse as sp

from .iebme import areas, encode, local_tiles

FORMATS = ("dense", "csr", "area_bitmap", "iebme")


def eq2(M: int, N: int, keep: float, bw: float, pmr: float) -> float:
    """Eq. 2 as printed; a format without metadata has no 1/PMR term."""
    inflation = 1.0 + 1.0 / pmr if pmr > 0 else 1.0
    return 2.0 * M * N * keep / (bw * M * keep * inflation + bw * N)


def format_bytes(W, value_bits: int, N: int) -> dict:
    W = np.asarray(W)
    M, K = W.shape
    bw = value_bits / 8.0
    nnz = int(np.count_nonzero(W))
    keep = nnz / (M * K)
    out = {}

    out["dense"] = dict(meta_bytes=0, payload_useful_bytes=bw * M * K, payload_stored_bytes=bw * M * K,
                        pmr=0.0, ci_eff=eq2(M, N, 1.0, bw, 0.0))

    csr = sp.csr_matrix(W)
    csr_meta = 4 * csr.indices.size + 4 * csr.indptr.size
    out["csr"] = dict(meta_bytes=csr_meta, payload_useful_bytes=bw * nnz,
                      payload_stored_bytes=bw * csr.data.size)

    A = areas(local_tiles(W, 16, 64), 2, 2) != 0        # (n_lt, 4, 8, 32)
    n_areas = A.shape[0] * A.shape[1]
    bitmap_bits = A.shape[2] * A.shape[3]
    area_meta = n_areas * (bitmap_bits // 8 + 4)
    out["area_bitmap"] = dict(meta_bytes=area_meta, payload_useful_bytes=bw * nnz,
                              payload_stored_bytes=bw * int(A.sum()))

    # The union masks depend only on where the nonzeros are.
    enc = encode((W != 0).astype(np.int8))
    iebme_meta = enc.n_lt * (enc.words_per_lt * 8 + 4)
    stored_values = int(enc.offsets[-1])
    out["iebme"] = dict(meta_bytes=iebme_meta, payload_useful_bytes=bw * nnz,
                        payload_stored_bytes=bw * stored_values)

    for name in FORMATS:
        r = out[name]
        if name != "dense":
            r["pmr"] = r["payload_useful_bytes"] / r["meta_bytes"] if r["meta_bytes"] else 0.0
            r["ci_eff"] = eq2(M, N, keep, bw, r["pmr"]) if keep > 0 else 0.0
        r["total_bytes"] = r["meta_bytes"] + r["payload_stored_bytes"]
        macs = M * K if name == "dense" else nnz
        r["ci_stored"] = 2.0 * macs * N / (r["total_bytes"] + bw * N * K)
    return out
