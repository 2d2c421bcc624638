"""Oracle for the IE-BME representation (TEST INFRASTRUCTURE ONLY).

Plain numpy restatement of the paper's Index-Efficient Bitmap Encoding:
Section V-A ("Area Partitioning", "Shared Union Mask", "IE-BME Storage
Layout") and the Low-Bit Shared-Memory Parallel Decoding index equations of
Section VI-B. Each step follows the paper's order and notation; no step is
fused or reordered for speed. Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may use this package. It shares no code
with the HIP path.

Readings taken where the paper is silent:
  * local tile (LT) 16 x 64, given only in the caption of the encoding figure;
  * R_A = C_A = 2, so Q = 4 areas of 8 x 32;
  * area index q = a * C_A + c, for row partition a and column partition c;
  * areas are contiguous blocks: rows [a*H_L/R_A, (a+1)*H_L/R_A), columns
    [c*K_L/C_A, (c+1)*K_L/C_A);
  * LTs are numbered row-block-major: t = mb * (K / K_L) + kb;
  * union-mask bit (i, j) is linear bit L = i * K_B + j; bit L lives in 64-bit
    word L // 64 of its LT at bit L % 64 (leftmost column = least significant);
  * offsets are counted in INT4 values and stored as uint32, n_LT + 1 entries;
  * payload nibble n sits in byte n // 2, in the low half when n is even, as
    4-bit two's complement; 16 zero bytes of tail padding follow the payload;
  * a signed b-bit quantizer (Section V-A) covers [-2^(b-1), 2^(b-1) - 1]; with
    b = 2 (the W2A4 setting of the evaluation) the payload packs four values
    per byte, value n at bits 2 (n mod 4) .. 2 (n mod 4) + 1 of byte n // 4,
    everything else (mask, offsets in values, stream order) unchanged.

Value order within an LT. The storage-layout passage puts area q's value at
rank rho at CV[o_t + q P_t + rho] (``order="areas"``, the paper's order).
The library stores the same values in a second order (``order="area_rows"``):
the C_A areas of one area row alternate value by value, area (a, c) at rank
rho at CV[o_t + a C_A P_t + C_A rho + c], so that one read at a rank serves
every area of the row. Offsets, bitmaps, P_t and the byte count are the same
in both orders; only the positions of the values inside an LT differ.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

INT4_MIN, INT4_MAX = -8, 7
TAIL_PAD_BYTES = 16
VALUE_BITS = (4, 2)                     # W4A4 and W2A4 payloads


def value_range(bits: int):
    """Alphabet bounds of the signed b-bit quantizer."""
    if bits not in VALUE_BITS:
        raise ValueError(f"payload values are 4 or 2 bits, not {bits}")
    return -(1 << (bits - 1)), (1 << (bits - 1)) - 1


@dataclass
class Encoded:
    """The three IE-BME arrays of Section V-A plus the tile geometry."""

    M: int
    K: int
    lt_h: int
    lt_w: int
    ra: int
    ca: int
    bitmaps: np.ndarray   # uint64, words_per_lt words per LT ("Union Bitmaps")
    offsets: np.ndarray   # uint32, n_lt + 1 entries ("Union Value Offsets")
    payload: np.ndarray   # uint8, packed b-bit values ("Compressed Values") + tail pad
    P: np.ndarray         # int64 per LT: P_t = ||B_t||_0
    nnz: int
    bits: int = 4         # bits per payload value
    order: str = "areas"  # value order within an LT (see the module docstring)

    @property
    def Q(self) -> int:
        return self.ra * self.ca

    @property
    def n_lt(self) -> int:
        return (self.M // self.lt_h) * (self.K // self.lt_w)

    @property
    def n_payload(self) -> int:
        return int(self.offsets[-1])

    @property
    def area_shape(self):
        return self.lt_h // self.ra, self.lt_w // self.ca

    @property
    def words_per_lt(self) -> int:
        hb, kb = self.area_shape
        return hb * kb // 64


def check_weights(W, bits: int = 4) -> np.ndarray:
    W = np.asarray(W)
    lo, hi = value_range(bits)
    if W.ndim != 2 or not np.issubdtype(W.dtype, np.integer):
        raise ValueError("W must be a 2-D integer matrix")
    if W.size and (W.min() < lo or W.max() > hi):
        raise ValueError(f"W values must lie in the signed {bits}-bit range [{lo}, {hi}]")
    return W.astype(np.int64)


def local_tiles(W: np.ndarray, lt_h: int, lt_w: int) -> np.ndarray:
    """Cut W into LTs, numbered t = mb * (K / lt_w) + kb: shape (n_lt, lt_h, lt_w)."""
    M, K = W.shape
    nmb, nkb = M // lt_h, K // lt_w
    return W.reshape(nmb, lt_h, nkb, lt_w).transpose(0, 2, 1, 3).reshape(nmb * nkb, lt_h, lt_w)


def areas(T: np.ndarray, ra: int, ca: int) -> np.ndarray:
    """Area partitioning (Section V-A): W_t^(q)(i, j), shape (n_lt, Q, H_L/R_A, K_L/C_A).

    Area q = a * C_A + c holds rows [a*hb, (a+1)*hb) and columns [c*kb, (c+1)*kb).
    """
    n_lt, lt_h, lt_w = T.shape
    hb, kb = lt_h // ra, lt_w // ca
    return T.reshape(n_lt, ra, hb, ca, kb).transpose(0, 1, 3, 2, 4).reshape(n_lt, ra * ca, hb, kb)


VALUE_ORDERS = ("areas", "area_rows")


def value_address(off, P, q, rho, ca: int, order: str):
    """Position in the compressed-values array of area q's value at rank rho
    of an LT with offset off and P active union-mask entries.

    "areas": o_t + q P_t + rho (the storage-layout passage of Section V-A);
    "area_rows": area q = a C_A + c at o_t + a C_A P_t + C_A rho + c.
    """
    if order == "areas":
        return off + q * P + rho
    if order == "area_rows":
        a, c = q // ca, q % ca
        return off + a * ca * P + ca * rho + c
    raise ValueError(f"unknown value order {order!r}")


def encode(W, lt_h: int = 16, lt_w: int = 64, ra: int = 2, ca: int = 2, bits: int = 4,
           order: str = "areas") -> Encoded:
    """IE-BME encoding of a masked b-bit matrix (Section V-A)."""
    if order not in VALUE_ORDERS:
        raise ValueError(f"unknown value order {order!r}")
    W = check_weights(W, bits)
    M, K = W.shape
    if M % lt_h or K % lt_w or lt_h % ra or lt_w % ca:
        raise ValueError("shape must tile exactly into LTs and areas")
    hb, kb = lt_h // ra, lt_w // ca
    if (hb * kb) % 64:
        raise ValueError("the union mask of an LT must fill whole 64-bit words")
    Q = ra * ca

    # Area partitioning: one grouped position (i, j) shared by all Q areas.
    A = areas(local_tiles(W, lt_h, lt_w), ra, ca)
    n_lt = A.shape[0]

    # Shared union mask: B_t(i, j) = 1 if any area value at (i, j) is nonzero.
    B = np.any(A != 0, axis=1)                        # (n_lt, hb, kb)

    # P_t = number of active union-mask entries.
    P = B.reshape(n_lt, -1).sum(axis=1).astype(np.int64)

    # Union Value Offsets: o_t = sum over earlier tiles of Q * P_tau.
    offsets = np.zeros(n_lt + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(Q * P)
    if offsets[-1] > np.iinfo(np.uint32).max:
        raise ValueError("payload exceeds the uint32 offset range")

    # Union Bitmaps: row-major scan, leftmost bit = LSB, packed into 64-bit words.
    nbits = hb * kb
    mask_bits = B.reshape(n_lt, nbits // 64, 64).astype(np.uint64)
    shifts = np.arange(64, dtype=np.uint64)
    words = np.bitwise_or.reduce(mask_bits << shifts, axis=2)
    bitmaps = words.reshape(-1).astype(np.uint64)

    # Compressed Values: compact rank rho_t(i, j) = active entries before (i, j)
    # in row-major order; CV[o_t + q * P_t + rho] = W_t^(q)(i, j) in the
    # paper's order, or at value_address(...) in the chosen order.
    flat = B.reshape(n_lt, nbits)
    rho = np.cumsum(flat, axis=1) - flat
    t_idx, pos = np.nonzero(flat)
    vals = A.reshape(n_lt, Q, nbits)[t_idx, :, pos]                       # (n_active, Q)
    addr = value_address(offsets[t_idx][:, None], P[t_idx][:, None], np.arange(Q, dtype=np.int64)[None, :],
                         rho[t_idx, pos][:, None], ca, order)
    cv = np.zeros(int(offsets[-1]), dtype=np.int64)
    cv[addr.ravel()] = vals.ravel()

    return Encoded(M, K, lt_h, lt_w, ra, ca, bitmaps, offsets.astype(np.uint32),
                   pack_values(cv, bits), P, int(np.count_nonzero(W)), bits, order)


def pack_values(v: np.ndarray, bits: int) -> np.ndarray:
    """b-bit values -> bytes: value n at bits b (n mod 8/b) of byte n // (8/b).

    Adds the zeroed tail pad; values are stored as b-bit two's complement.
    """
    if bits == 4:
        return pack_nibbles(v)
    value_range(bits)
    per = 8 // bits
    v = np.asarray(v, dtype=np.int64)
    u = (v & ((1 << bits) - 1)).astype(np.uint8)
    out = np.zeros(-(-v.size // per) + TAIL_PAD_BYTES, dtype=np.uint8)
    for k in range(per):
        part = u[k::per]
        out[: part.size] |= (part << (bits * k)).astype(np.uint8)
    return out


def unpack_values(b: np.ndarray, n: int, bits: int) -> np.ndarray:
    """Inverse of pack_values for the first n values (sign-extended to int64)."""
    if bits == 4:
        return unpack_nibbles(b, n)
    value_range(bits)
    per = 8 // bits
    b = np.asarray(b, dtype=np.uint8)[: -(-n // per)].astype(np.int64)
    u = np.empty(b.size * per, dtype=np.int64)
    for k in range(per):
        u[k::per] = (b >> (bits * k)) & ((1 << bits) - 1)
    u = u[:n]
    return np.where(u >= (1 << (bits - 1)), u - (1 << bits), u)


def pack_nibbles(v: np.ndarray) -> np.ndarray:
    """INT4 values -> bytes: value n in byte n // 2, low half when n is even.

    Adds the zeroed tail pad. Values are stored as 4-bit two's complement.
    """
    v = np.asarray(v, dtype=np.int64)
    n = v.size
    u = (v & 0xF).astype(np.uint8)
    out = np.zeros((n + 1) // 2 + TAIL_PAD_BYTES, dtype=np.uint8)
    out[: n // 2] = u[0 : 2 * (n // 2) : 2] | (u[1 : 2 * (n // 2) : 2] << 4)
    if n % 2:
        out[n // 2] = u[n - 1]
    return out


def unpack_nibbles(b: np.ndarray, n: int) -> np.ndarray:
    """Inverse of pack_nibbles for the first n values (sign-extended to int64)."""
    b = np.asarray(b, dtype=np.uint8)
    u = np.empty(2 * ((n + 1) // 2), dtype=np.int64)
    u[0::2] = b[: (n + 1) // 2] & 0xF
    u[1::2] = b[: (n + 1) // 2] >> 4
    u = u[:n]
    return np.where(u >= 8, u - 16, u)


def union_mask(enc: Encoded) -> np.ndarray:
    """Unpack the Union Bitmaps back to B_t: bool (n_lt, hb, kb)."""
    hb, kb = enc.area_shape
    w = enc.bitmaps.reshape(enc.n_lt, enc.words_per_lt, 1)
    bits = (w >> np.arange(64, dtype=np.uint64)) & np.uint64(1)
    return bits.reshape(enc.n_lt, hb, kb).astype(bool)


def decode(enc: Encoded) -> np.ndarray:
    """Inverse of encode: rebuild the dense INT4 matrix from the three arrays.

    Every active (i, j) of LT t takes W_t^(q)(i, j) = CV[o_t + q * P_t + rho_t(i, j)]
    (or the value at value_address in the encoding's order); every inactive
    position is zero in all Q areas.
    """
    hb, kb = enc.area_shape
    Q, n_lt = enc.Q, enc.n_lt
    B = union_mask(enc).reshape(n_lt, hb * kb)
    P = B.sum(axis=1).astype(np.int64)
    off = enc.offsets.astype(np.int64)
    if not np.array_equal(off[1:] - off[:-1], Q * P):
        raise ValueError("offsets disagree with the union bitmaps")
    cv = unpack_values(enc.payload, int(off[-1]), enc.bits)
    rho = np.cumsum(B, axis=1) - B
    A = np.zeros((n_lt, Q, hb * kb), dtype=np.int64)
    t_idx, pos = np.nonzero(B)
    addr = value_address(off[t_idx][:, None], P[t_idx][:, None], np.arange(Q, dtype=np.int64)[None, :],
                         rho[t_idx, pos][:, None], enc.ca, enc.order)
    A[t_idx, :, pos] = cv[addr]
    # Undo the area partitioning, then the LT tiling.
    T = (A.reshape(n_lt, enc.ra, enc.ca, hb, kb).transpose(0, 1, 3, 2, 4)
         .reshape(n_lt, enc.lt_h, enc.lt_w))
    nmb, nkb = enc.M // enc.lt_h, enc.K // enc.lt_w
    return T.reshape(nmb, nkb, enc.lt_h, enc.lt_w).transpose(0, 2, 1, 3).reshape(enc.M, enc.K)


# --------------------------------------------------------------------------
# LSPD index generation (Section VI-B, "Thread-to-Segment Mapping",
# "Bitmap-Guided Offset Generation", "Area Gathering and Register Packing").
# --------------------------------------------------------------------------

def lspd_idx_base(Bt: np.ndarray, r: int, g: int, G: int) -> int:
    """idx_base(r, g): active bits in all rows above r plus those of row r before j_g = g*G."""
    jg = g * G
    return int(Bt[:r, :].sum() + Bt[r, :jg].sum())


def lspd_segment(Bt: np.ndarray, r: int, g: int, G: int, streams: list) -> list:
    """Gather one G-bit segment of union-mask row r from every area stream.

    Returns, per area q, the G decoded values of the segment: an active bit at
    segment position p with seg_rank k reads V^(q)[idx_base + k]; inactive
    positions are zero and read nothing.
    """
    base = lspd_idx_base(Bt, r, g, G)
    out = []
    for V in streams:
        vals, k = [], 0
        for p in range(G):
            if Bt[r, g * G + p]:
                vals.append(int(V[base + k]))   # global_idx = idx_base + seg_rank
                k += 1
            else:
                vals.append(0)
        out.append(vals)
    return out


def lspd_decode_tile(enc: Encoded, t: int, G: int) -> np.ndarray:
    """Decode LT t segment by segment with the LSPD index equations: (lt_h, lt_w)."""
    hb, kb = enc.area_shape
    Bt = union_mask(enc)[t]
    Pt = int(Bt.sum())
    o = int(enc.offsets[t])
    cv = unpack_values(enc.payload, int(enc.offsets[-1]), enc.bits)
    rhos = np.arange(Pt, dtype=np.int64)
    streams = [cv[value_address(o, Pt, q, rhos, enc.ca, enc.order)] for q in range(enc.Q)]
    A = np.zeros((enc.Q, hb, kb), dtype=np.int64)
    for r in range(hb):
        for g in range(kb // G):
            seg = lspd_segment(Bt, r, g, G, streams)
            for q in range(enc.Q):
                A[q, r, g * G:(g + 1) * G] = seg[q]
    T = np.zeros((enc.lt_h, enc.lt_w), dtype=np.int64)
    for q in range(enc.Q):
        a, c = divmod(q, enc.ca)
        T[a * hb:(a + 1) * hb, c * kb:(c + 1) * kb] = A[q]
    return T


# --------------------------------------------------------------------------
# Payload-to-Metadata Ratio (Eq. 1) and effective compute intensity (Eq. 2).
# --------------------------------------------------------------------------

def pmr_report(enc: Encoded, N: int = 0, bytes_per_weight: float = None) -> dict:
    """Byte accounting of an encoded matrix (Section III-B/C).

    Metadata = union bitmaps + one offset per LT (the sentinel offset is not
    counted). ``pmr`` is Eq. 1 with the useful payload B_w * nnz; ``pmr_stored``
    uses the stored payload, which also holds the zeros kept inside active
    groups. ``ci_eff`` is Eq. 2 evaluated as printed, for activation width N.
    """
    if bytes_per_weight is None:
        bytes_per_weight = enc.bits / 8                             # B_w
    n_lt = enc.n_lt
    bitmap_bytes = 8 * enc.words_per_lt * n_lt
    offset_bytes = 4 * n_lt
    meta = bitmap_bytes + offset_bytes
    stored_values = int(enc.offsets[-1])
    payload_useful = bytes_per_weight * enc.nnz                  # B_w * M * K * (1 - s)
    payload_stored = bytes_per_weight * stored_values
    pmr = payload_useful / meta
    per = 8 // enc.bits
    rep = dict(nnz=enc.nnz, stored_values=stored_values, n_lt=n_lt,
               payload_stored_bytes=-(-stored_values // per),
               bitmap_bytes=bitmap_bytes, offset_bytes=offset_bytes, meta_bytes=meta,
               payload_useful_bytes=payload_useful, pmr=pmr,
               pmr_stored=payload_stored / meta, ci_eff=0.0)
    if N > 0:
        rep["ci_eff"] = ci_eff(enc.M, enc.K, N, 1.0 - enc.nnz / (enc.M * enc.K), pmr,
                               bytes_per_weight)
    return rep


def ci_eff(M: int, K: int, N: int, s: float, pmr: float, bytes_per_weight: float = 0.5) -> float:
    """Eq. 2: 2 M N (1-s) / (B_w M (1-s) (1 + 1/PMR) + B_w N). K does not appear."""
    keep = 1.0 - s
    if keep <= 0.0 or pmr <= 0.0:
        return 0.0
    bw = bytes_per_weight
    return 2.0 * M * N * keep / (bw * M * keep * (1.0 + 1.0 / pmr) + bw * N)
