"""Pins for the oracle's second value order ("area_rows").

The paper stores area q's value at rank rho at CV[o_t + q P_t + rho] (Section
V-A, storage layout). The library stores the same values with the areas of an
area row alternating: area (a, c) at CV[o_t + a C_A P_t + C_A rho + c]. Nothing
in the paper fixes that order, so it is pinned to its definition: payload bytes
worked out by hand for a small LT, and round trips (decode of the encoding is
the matrix) over both orders, both value widths and several tile geometries.
A swapped a / c, a missing factor C_A or a wrong nibble order fails one of them.
"""
import numpy as np
import pytest

from oracle import iebme
from paper_2608_09291_amd import synth


def _two_active_lt(vals):
    """A 16 x 64 LT whose union mask has exactly (0, 0) and (0, 1) active.

    vals[q] = (value at rank 0, value at rank 1) of area q = 2 a + c, area
    (a, c) covering rows 8a.., columns 32c.."""
    W = np.zeros((16, 64), dtype=np.int8)
    for q, (v0, v1) in enumerate(vals):
        a, c = divmod(q, 2)
        W[8 * a, 32 * c] = v0
        W[8 * a, 32 * c + 1] = v1
    return W


def test_hand_example_4bit():
    # Areas: q0 = (1, 2), q1 = (3, 4), q2 = (5, 6), q3 = (7, -1); P_t = 2.
    W = _two_active_lt([(1, 2), (3, 4), (5, 6), (7, -1)])
    paper = iebme.encode(W, order="areas")
    rows = iebme.encode(W, order="area_rows")
    assert int(paper.P[0]) == 2 and list(paper.offsets) == [0, 8] == list(rows.offsets)
    # Paper order: 1 2 | 3 4 | 5 6 | 7 -1, two values per byte, low nibble first.
    assert paper.payload[:4].tolist() == [0x21, 0x43, 0x65, 0xF7]
    # Area rows: area row 0 alternates q0, q1 by rank: 1 3 2 4; area row 1: 5 7 6 -1.
    assert rows.payload[:4].tolist() == [0x31, 0x42, 0x75, 0xF6]
    assert np.array_equal(paper.bitmaps, rows.bitmaps)
    assert not rows.payload[4:].any()


def test_hand_example_2bit():
    # 2-bit values, four per byte, value n at bits 2 (n mod 4).
    W = _two_active_lt([(1, -2), (-1, 0), (0, 1), (-2, -1)])
    rows = iebme.encode(W, bits=2, order="area_rows")
    paper = iebme.encode(W, bits=2, order="areas")
    # Paper order 1 -2 -1 0 | 0 1 -2 -1 -> codes 1 2 3 0 | 0 1 2 3.
    assert paper.payload[:2].tolist() == [0b00111001, 0b11100100]
    # Area rows: 1 -1 -2 0 | 0 -2 1 -1 -> codes 1 3 2 0 | 0 2 1 3.
    assert rows.payload[:2].tolist() == [0b00101101, 0b11011000]


@pytest.mark.parametrize("bits", [4, 2])
@pytest.mark.parametrize("sparsity", [0.0, 0.5, 0.9, 1.0])
def test_round_trip_both_orders(bits, sparsity):
    W, _, _ = synth.random_problem(64, 512, 1, sparsity, 11, bits=bits)
    for order in iebme.VALUE_ORDERS:
        enc = iebme.encode(W, bits=bits, order=order)
        assert np.array_equal(iebme.decode(enc), W)


@pytest.mark.parametrize("lt_h,lt_w,ra,ca", [(16, 64, 2, 2), (8, 128, 1, 4), (32, 64, 4, 2), (16, 128, 2, 4)])
def test_round_trip_geometries(lt_h, lt_w, ra, ca):
    W, _, _ = synth.random_problem(2 * lt_h, 2 * lt_w, 1, 0.6, 12)
    rows = iebme.encode(W, lt_h=lt_h, lt_w=lt_w, ra=ra, ca=ca, order="area_rows")
    paper = iebme.encode(W, lt_h=lt_h, lt_w=lt_w, ra=ra, ca=ca, order="areas")
    assert np.array_equal(iebme.decode(rows), W)
    assert np.array_equal(rows.offsets, paper.offsets) and np.array_equal(rows.bitmaps, paper.bitmaps)
    # Within every LT the two orders hold the same values.
    n = rows.n_payload
    a = iebme.unpack_values(rows.payload, n, 4)
    b = iebme.unpack_values(paper.payload, n, 4)
    off = rows.offsets.astype(np.int64)
    for t in range(rows.n_lt):
        assert sorted(a[off[t]:off[t + 1]]) == sorted(b[off[t]:off[t + 1]])


def test_lspd_decode_reads_either_order():
    W, _, _ = synth.random_problem(32, 128, 1, 0.5, 13)
    tiles = iebme.local_tiles(W.astype(np.int64), 16, 64)
    for order in iebme.VALUE_ORDERS:
        enc = iebme.encode(W, order=order)
        for t in range(enc.n_lt):
            assert np.array_equal(iebme.lspd_decode_tile(enc, t, 8), tiles[t])


def test_unknown_order_is_refused():
    with pytest.raises(ValueError):
        iebme.encode(np.zeros((16, 64), dtype=np.int8), order="columns")
