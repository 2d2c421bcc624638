"""Cross-format byte accounting (Section III-B/C): oracle pins and native parity.

Pins tie oracle/formats.py to things other than its own formulas: a tile
counted by hand, the IE-BME/area-bitmap metadata ratio fixed by the layouts,
Eq. 1's linearity in the value width, scipy's CSR arrays, and the i.i.d.
expectation of IE-BME's stored values. The native us_pmr_formats must then
match the oracle field by field.
"""
import numpy as np
import pytest

from oracle import formats, iebme
from paper_2608_09291_amd import binding, synth


def test_hand_counted_tile():
    # One 16 x 64 LT with nonzeros at (0, 0), (8, 0), (0, 32), (3, 5), (15, 63).
    W = np.zeros((16, 64), dtype=np.int8)
    for r, c in [(0, 0), (8, 0), (0, 32), (3, 5), (15, 63)]:
        W[r, c] = 3
    rep = formats.format_bytes(W, 4, 2)
    assert rep["csr"]["meta_bytes"] == 4 * 5 + 4 * 17
    assert rep["area_bitmap"]["meta_bytes"] == 4 * (32 + 4)
    assert rep["area_bitmap"]["payload_stored_bytes"] == 0.5 * 5
    # Union mask: (0,0) is shared by rows 0 and 8 and columns 0 and 32 -> one
    # group; (3,5) and (15,63) -> (7, 31) are two more: 3 groups x 4 areas.
    assert rep["iebme"]["meta_bytes"] == 36
    assert rep["iebme"]["payload_stored_bytes"] == 0.5 * 12
    assert rep["dense"]["payload_stored_bytes"] == 0.5 * 1024
    assert rep["iebme"]["pmr"] == pytest.approx(2.5 / 36)
    # Eq. 2 by hand: M = 16, N = 2, 1 - s = 5/1024, B_w = 1/2. With PMR = 2.5/36
    # the denominator is 205/128 and the numerator 5/16: CI = 8/41; with the
    # area bitmaps' PMR = 2.5/144 it is 40/421.
    assert rep["iebme"]["ci_eff"] == pytest.approx(8 / 41, rel=1e-14)
    assert rep["area_bitmap"]["ci_eff"] == pytest.approx(40 / 421, rel=1e-14)


@pytest.mark.parametrize("s", [0.3, 0.5, 0.7, 0.95])
def test_layout_ratio_and_precision_scaling(s):
    W, _, _ = synth.random_problem(64, 512, 1, s, 3)
    r4, r16 = formats.format_bytes(W, 4, 8), formats.format_bytes(W, 16, 8)
    # Same useful payload, four times the metadata of one shared union mask.
    assert r4["area_bitmap"]["pmr"] == pytest.approx(r4["iebme"]["pmr"] / 4, rel=1e-15)
    for f in ("csr", "area_bitmap", "iebme"):
        assert r16[f]["pmr"] == pytest.approx(4 * r4[f]["pmr"], rel=1e-15)   # Eq. 1 is linear in B_w
        assert r16[f]["meta_bytes"] == r4[f]["meta_bytes"]


def test_csr_against_row_counts():
    W, _, _ = synth.random_problem(48, 256, 1, 0.6, 4)
    per_row = [int(np.count_nonzero(W[m])) for m in range(48)]
    rep = formats.format_bytes(W, 8, 1)
    assert rep["csr"]["meta_bytes"] == 4 * sum(per_row) + 4 * (48 + 1)


def test_iebme_stored_values_iid_expectation():
    s = 0.6
    W, _, _ = synth.random_problem(512, 2048, 1, s, 5)
    rep = formats.format_bytes(W, 4, 1)
    n_lt = (512 // 16) * (2048 // 64)
    expect = 0.5 * n_lt * 4 * 256 * (1 - s ** 4)
    assert rep["iebme"]["payload_stored_bytes"] == pytest.approx(expect, rel=0.01)


def test_eq2_limits():
    # Dense with s = 0 and no metadata: 2 M N / (B_w M + B_w N).
    W = np.ones((32, 128), dtype=np.int8)
    rep = formats.format_bytes(W, 8, 16)
    assert rep["dense"]["ci_eff"] == pytest.approx(2 * 32 * 16 / (32 + 16))
    assert rep["dense"]["ci_stored"] == pytest.approx(2 * 32 * 128 * 16 / (32 * 128 + 16 * 128))


@pytest.mark.parametrize("bits", [16, 8, 4, 2])
@pytest.mark.parametrize("M,K,s,N,seed", [(16, 64, 0.5, 1, 1), (64, 512, 0.4, 8, 2), (128, 1024, 0.7, 32, 3),
                                          (32, 256, 0.0, 4, 4), (32, 256, 1.0, 4, 5)])
def test_native_matches_oracle(bits, M, K, s, N, seed):
    W, _, _ = synth.random_problem(M, K, 1, s, seed)
    got = binding.pmr_formats(binding.encode(W), bits, N)
    want = formats.format_bytes(W, bits, N)
    for f in formats.FORMATS:
        for key, v in want[f].items():
            assert got[f][key] == pytest.approx(v, rel=1e-12, abs=1e-12), (f, key)


def test_native_argument_errors():
    enc = binding.encode(np.zeros((16, 64), dtype=np.int8))
    for bits, N in [(3, 1), (32, 1), (4, 0)]:
        with pytest.raises(binding.UsError):
            binding.pmr_formats(enc, bits, N)
