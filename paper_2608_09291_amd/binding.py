"""Python binding of the UnionSparse C-ABI (include/us.h, include/us_probe.h).

Argument marshalling only: every computation happens in the native library
(the encoder in C++, the products in HIP kernels). PyTorch provides device
memory and streams. The library must have been built in-tree
(``python -m paper_2608_09291_amd.build``); without it every call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libunionsparse.so")

US_OK = 0
STATUS = {0: "US_OK", -1: "US_ERR_ARG", -2: "US_ERR_SHAPE", -3: "US_ERR_RANGE",
          -4: "US_ERR_NOMEM", -5: "US_ERR_DEVICE", -6: "US_ERR_FORMAT"}
PAYLOAD_PAD = 16
N_MAX = 32          # widest single kernel pass
N_LIMIT = 1024      # widest activation matrix (slabs of N_MAX beyond N_MAX)
K_MAX = 130048

#: Every symbol the two public headers declare.
EXPORTS = ("us_encode", "us_encode_w2", "us_encode_reordered", "us_iebme_free", "us_pmr", "us_pmr_formats", "us_spmm_plan", "us_spmm_workspace_size", "us_spmm", "us_spmm_noalloc",
           "us_gemm_i8", "us_status_string", "us_probe_read", "us_probe_read_sink_words",
           "us_probe_copy", "us_probe_copy_lds", "us_probe_spin")


class UsError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {STATUS.get(status, status)}")
        self.status = status


class IEBME(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int32), ("K", ctypes.c_int32),
                ("lt_h", ctypes.c_int32), ("lt_w", ctypes.c_int32),
                ("ra", ctypes.c_int32), ("ca", ctypes.c_int32),
                ("n_lt", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("n_payload", ctypes.c_int64), ("payload_bytes", ctypes.c_int64),
                ("bitmaps", ctypes.POINTER(ctypes.c_uint64)),
                ("offsets", ctypes.POINTER(ctypes.c_uint32)),
                ("payload", ctypes.POINTER(ctypes.c_uint8)),
                ("perm", ctypes.POINTER(ctypes.c_uint64)), ("bits", ctypes.c_int32)]


class PMRReport(ctypes.Structure):
    _fields_ = [("nnz", ctypes.c_int64), ("stored_values", ctypes.c_int64),
                ("n_lt", ctypes.c_int64), ("payload_stored_bytes", ctypes.c_int64),
                ("bitmap_bytes", ctypes.c_int64), ("offset_bytes", ctypes.c_int64),
                ("meta_bytes", ctypes.c_int64), ("payload_useful_bytes", ctypes.c_double),
                ("pmr", ctypes.c_double), ("pmr_stored", ctypes.c_double),
                ("ci_eff", ctypes.c_double), ("perm_bytes", ctypes.c_int64)]


FORMATS = ("dense", "csr", "area_bitmap", "iebme")


class FormatReport(ctypes.Structure):
    _fields_ = [("format", ctypes.c_int32), ("value_bits", ctypes.c_int32), ("meta_bytes", ctypes.c_int64),
                ("payload_useful_bytes", ctypes.c_double), ("payload_stored_bytes", ctypes.c_double),
                ("pmr", ctypes.c_double), ("ci_eff", ctypes.c_double), ("total_bytes", ctypes.c_double),
                ("ci_stored", ctypes.c_double)]


class IEBMEDev(ctypes.Structure):
    _fields_ = [("bitmaps", ctypes.c_void_p), ("offsets", ctypes.c_void_p),
                ("payload", ctypes.c_void_p), ("M", ctypes.c_int32), ("K", ctypes.c_int32),
                ("n_lt", ctypes.c_int64), ("n_payload", ctypes.c_int64), ("perm", ctypes.c_void_p),
                ("bits", ctypes.c_int32)]


class SpmmOpts(ctypes.Structure):
    _fields_ = [("split_k", ctypes.c_int32), ("variant", ctypes.c_int32), ("chunk_lts", ctypes.c_int32),
                ("k_blocks", ctypes.c_int32)]


#: us_spmm_opts.variant values
VARIANT_AUTO, VARIANT_WHOLE, VARIANT_RING, VARIANT_BURST = 0, 1, 2, 3
K_BLOCKS_MAX = 64   # US_K_BLOCKS_MAX


_lib = None


def lib():
    """Load the native library (once); raise if it was not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run `python -m paper_2608_09291_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        L.us_encode.argtypes = [vp, i32, i32, i64, ctypes.POINTER(IEBME)]
        L.us_encode_reordered.argtypes = [vp, i32, i32, i64, ctypes.POINTER(IEBME)]
        L.us_encode_w2.argtypes = [vp, i32, i32, i64, ctypes.POINTER(IEBME)]
        L.us_iebme_free.argtypes = [ctypes.POINTER(IEBME)]
        L.us_iebme_free.restype = None
        L.us_pmr.argtypes = [ctypes.POINTER(IEBME), i32, ctypes.POINTER(PMRReport)]
        L.us_pmr_formats.argtypes = [ctypes.POINTER(IEBME), i32, i32, ctypes.POINTER(FormatReport)]
        L.us_spmm_workspace_size.argtypes = [i32, i32, i32, ctypes.POINTER(SpmmOpts),
                                             ctypes.POINTER(sz)]
        pi32 = ctypes.POINTER(i32)
        L.us_spmm_plan.argtypes = [i32, i32, i32, i32, i32, ctypes.POINTER(SpmmOpts), pi32, pi32, pi32, pi32]
        L.us_spmm.argtypes = [ctypes.POINTER(IEBMEDev), vp, i32, vp, vp, vp, vp, sz,
                              ctypes.POINTER(SpmmOpts), vp]
        L.us_spmm_noalloc.argtypes = [ctypes.POINTER(IEBMEDev), vp, i32, vp, vp, vp, ctypes.POINTER(SpmmOpts), vp]
        L.us_gemm_i8.argtypes = [vp, vp, i32, i32, i32, vp, vp]
        L.us_status_string.argtypes = [ctypes.c_int]
        L.us_status_string.restype = ctypes.c_char_p
        L.us_probe_read.argtypes = [vp, sz, vp, ctypes.c_int32, vp]
        L.us_probe_read_sink_words.argtypes = [sz]
        L.us_probe_read_sink_words.restype = sz
        L.us_probe_copy.argtypes = [vp, vp, sz, vp]
        L.us_probe_copy_lds.argtypes = [vp, vp, sz, vp]
        L.us_probe_spin.argtypes = [ctypes.c_uint64, vp]
        for name in ("us_encode", "us_encode_w2", "us_encode_reordered", "us_pmr", "us_pmr_formats", "us_spmm_workspace_size", "us_spmm_plan", "us_spmm", "us_spmm_noalloc", "us_gemm_i8",
                     "us_probe_read", "us_probe_copy", "us_probe_copy_lds", "us_probe_spin"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(fn: str, status: int):
    if status != US_OK:
        raise UsError(fn, status)


# ---------------------------------------------------------------------------
# Host encoder and byte accounting
# ---------------------------------------------------------------------------

class Encoded:
    """An IE-BME matrix produced by us_encode; owns the native arrays."""

    def __init__(self, s: IEBME):
        self._s = s

    @property
    def M(self): return self._s.M

    @property
    def K(self): return self._s.K

    @property
    def n_lt(self): return self._s.n_lt

    @property
    def nnz(self): return self._s.nnz

    @property
    def n_payload(self): return self._s.n_payload

    @property
    def bits(self): return self._s.bits

    @property
    def bitmaps(self) -> np.ndarray:
        return np.ctypeslib.as_array(self._s.bitmaps, shape=(4 * self._s.n_lt,))

    @property
    def offsets(self) -> np.ndarray:
        return np.ctypeslib.as_array(self._s.offsets, shape=(self._s.n_lt + 1,))

    @property
    def payload(self) -> np.ndarray:
        return np.ctypeslib.as_array(self._s.payload, shape=(self._s.payload_bytes,))

    @property
    def perm(self):
        """Row permutation words (one uint64 per LT), or None without reordering."""
        if not self._s.perm:
            return None
        return np.ctypeslib.as_array(self._s.perm, shape=(self._s.n_lt,))

    def struct(self) -> IEBME:
        return self._s

    def free(self):
        if self._s is not None and self._s.bitmaps:
            lib().us_iebme_free(ctypes.byref(self._s))

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def encode(W: np.ndarray, reorder: bool = False, bits: int = 4) -> Encoded:
    """us_encode, us_encode_reordered or (bits = 2) us_encode_w2 on a host int8 matrix."""
    W = np.ascontiguousarray(W, dtype=np.int8)
    if W.ndim != 2:
        raise ValueError("W must be 2-D")
    if bits == 2 and reorder:
        raise ValueError("2-bit matrices are not row-reordered")
    s = IEBME()
    name = "us_encode_w2" if bits == 2 else "us_encode_reordered" if reorder else "us_encode"
    _check(name, getattr(lib(), name)(W.ctypes.data, W.shape[0], W.shape[1], W.shape[1],
                                      ctypes.byref(s)))
    return Encoded(s)


def pmr(enc: Encoded, N: int = 0) -> dict:
    r = PMRReport()
    _check("us_pmr", lib().us_pmr(ctypes.byref(enc.struct()), N, ctypes.byref(r)))
    return {name: getattr(r, name) for name, _ in PMRReport._fields_}


def pmr_formats(enc: Encoded, value_bits: int, N: int) -> dict:
    """us_pmr_formats: {format name: report dict} for the mask of enc at value_bits bits."""
    out = (FormatReport * len(FORMATS))()
    _check("us_pmr_formats", lib().us_pmr_formats(ctypes.byref(enc.struct()), value_bits, N, out))
    return {FORMATS[r.format]: {name: getattr(r, name) for name, _ in FormatReport._fields_} for r in out}


# ---------------------------------------------------------------------------
# Device side
# ---------------------------------------------------------------------------

def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


@dataclass
class DeviceEncoded:
    """Device copies of the IE-BME arrays (torch tensors) and the C struct."""

    bitmaps: "object"
    offsets: "object"
    payload: "object"
    M: int
    K: int
    n_lt: int
    n_payload: int
    perm: "object" = None
    bits: int = 4

    def struct(self) -> IEBMEDev:
        return IEBMEDev(self.bitmaps.data_ptr(), self.offsets.data_ptr(), self.payload.data_ptr(),
                        self.M, self.K, self.n_lt, self.n_payload,
                        None if self.perm is None else self.perm.data_ptr(), self.bits)

    @property
    def nbytes(self) -> int:
        """Encoded bytes the kernel streams: bitmaps, offsets, stored payload, row permutations."""
        return (32 * self.n_lt + 4 * (self.n_lt + 1) + (self.n_payload * self.bits + 7) // 8
                + (0 if self.perm is None else 8 * self.n_lt))


def to_device(enc: Encoded, device="cuda") -> DeviceEncoded:
    import torch
    bm = torch.from_numpy(enc.bitmaps.view(np.int64).copy()).to(device)
    off = torch.from_numpy(enc.offsets.view(np.int32).copy()).to(device)
    pay = torch.from_numpy(enc.payload.copy()).to(device)
    perm = None if enc.perm is None else torch.from_numpy(enc.perm.view(np.int64).copy()).to(device)
    return DeviceEncoded(bm, off, pay, enc.M, enc.K, enc.n_lt, enc.n_payload, perm, enc.bits)


def pack_int4(Xt: np.ndarray) -> np.ndarray:
    """(N, K) int8 INT4 values -> (N, K/2) bytes, even k in the low nibble."""
    Xt = np.asarray(Xt, dtype=np.int8)
    u = (Xt.astype(np.int16) & 0xF).astype(np.uint8)
    return np.ascontiguousarray(u[:, 0::2] | (u[:, 1::2] << 4))


def workspace_size(M: int, K: int, N: int, split_k: int = 0, variant: int = 0, chunk_lts: int = 0,
                   k_blocks: int = 0) -> int:
    """us_spmm_workspace_size: device bytes us_spmm needs for these options."""
    n = ctypes.c_size_t(0)
    opts = SpmmOpts(split_k, variant, chunk_lts, k_blocks)
    _check("us_spmm_workspace_size",
           lib().us_spmm_workspace_size(M, K, N, ctypes.byref(opts), ctypes.byref(n)))
    return n.value


def spmm_plan(M: int, K: int, N: int, split_k: int = 0, variant: int = 0, reordered: bool = False,
              bits: int = 4, chunk_lts: int = 0, k_blocks: int = 0, full: bool = False):
    """us_spmm_plan: (K slices per workgroup, LTs per chunk or slice, staging 1 whole / 2 ring /
    3 single pass), and with full=True also the K blocks across workgroups."""
    opts = SpmmOpts(split_k, variant, chunk_lts, k_blocks)
    a, b, c, d = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    _check("us_spmm_plan", lib().us_spmm_plan(M, K, N, bits, int(bool(reordered)), ctypes.byref(opts),
                                              ctypes.byref(a), ctypes.byref(b), ctypes.byref(c), ctypes.byref(d)))
    return (a.value, b.value, c.value, d.value) if full else (a.value, b.value, c.value)


def spmm(w: DeviceEncoded, x_packed, N: int, y, scale=None, y_f32=None, split_k: int = 0,
         ws=None, stream=None, wstruct: IEBMEDev = None, variant: int = 0, chunk_lts: int = 0,
         k_blocks: int = 0) -> None:
    """us_spmm: y[n, m] = sum_k W[m, k] X[k, n] (+ optional dequant into y_f32)."""
    s = wstruct if wstruct is not None else w.struct()
    opts = SpmmOpts(split_k, variant, chunk_lts, k_blocks)
    _check("us_spmm", lib().us_spmm(
        ctypes.byref(s), x_packed.data_ptr(), N, y.data_ptr(),
        None if scale is None else scale.data_ptr(),
        None if y_f32 is None else y_f32.data_ptr(),
        None if ws is None else ws.data_ptr(), 0 if ws is None else ws.numel() * ws.element_size(),
        ctypes.byref(opts), _stream_handle(stream)))


NOALLOC_SCRATCH_BYTES = 4 << 20   # US_NOALLOC_SCRATCH_BYTES


def spmm_noalloc(w: DeviceEncoded, x_packed, N: int, y, scale=None, y_f32=None, split_k: int = 0,
                 stream=None, wstruct: IEBMEDev = None, variant: int = 0, chunk_lts: int = 0,
                 k_blocks: int = 0) -> None:
    """us_spmm_noalloc: us_spmm with the library's own per-device workspace."""
    s = wstruct if wstruct is not None else w.struct()
    opts = SpmmOpts(split_k, variant, chunk_lts, k_blocks)
    _check("us_spmm_noalloc", lib().us_spmm_noalloc(
        ctypes.byref(s), x_packed.data_ptr(), N, y.data_ptr(),
        None if scale is None else scale.data_ptr(),
        None if y_f32 is None else y_f32.data_ptr(),
        ctypes.byref(opts), _stream_handle(stream)))


def gemm_i8(w, x, M: int, K: int, N: int, y, stream=None) -> None:
    """us_gemm_i8: dense int8 (M, K) times int8 (N, K)^T into int32 (N, M)."""
    _check("us_gemm_i8", lib().us_gemm_i8(w.data_ptr(), x.data_ptr(), M, K, N, y.data_ptr(),
                                          _stream_handle(stream)))


PROBE_READ_SHAPES = 4      # US_PROBE_READ_SHAPES


def probe_read(src, nbytes: int, sink, shape: int = 0, stream=None) -> None:
    """us_probe_read: one streaming read of nbytes in launch shape `shape`."""
    _check("us_probe_read", lib().us_probe_read(src.data_ptr(), nbytes, sink.data_ptr(), shape,
                                                _stream_handle(stream)))


def probe_read_sink_words(nbytes: int) -> int:
    return int(lib().us_probe_read_sink_words(nbytes))


def probe_copy(src, dst, nbytes: int, stream=None) -> None:
    _check("us_probe_copy", lib().us_probe_copy(src.data_ptr(), dst.data_ptr(), nbytes,
                                                _stream_handle(stream)))


def probe_copy_lds(src, dst, nbytes: int, stream=None) -> None:
    """us_probe_copy_lds: the copy with non-temporal buffer loads straight into LDS."""
    _check("us_probe_copy_lds", lib().us_probe_copy_lds(src.data_ptr(), dst.data_ptr(), nbytes,
                                                        _stream_handle(stream)))


def probe_spin(ns: int, stream=None) -> None:
    _check("us_probe_spin", lib().us_probe_spin(int(ns), _stream_handle(stream)))
