"""The native 2-bit encoder (us_encode_w2, the W2A4 setting) against the oracle.

The oracle's 2-bit packing is pinned in test_w2_pins.py; here the native
arrays must equal the oracle's byte for byte, and the byte accounting must
follow Eq. 1 with B_w = 1/4.
"""
import ctypes

import numpy as np
import pytest

from oracle import iebme
from paper_2608_09291_amd import binding, synth


@pytest.mark.parametrize("M,K,s,seed,skew", [
    (16, 64, 0.5, 0, False), (48, 192, 0.3, 1, False), (64, 256, 0.7, 2, False),
    (32, 128, 0.0, 3, False), (32, 128, 1.0, 4, False), (80, 320, 0.9, 5, False),
    (256, 512, 0.6, 6, True), (512, 512, 0.5, 7, False)])
def test_w2_encoder_matches_oracle(M, K, s, seed, skew):
    W, _, _ = synth.random_problem(M, K, 1, s, seed, row_skew=skew, bits=2)
    enc, ref = binding.encode(W, bits=2), iebme.encode(W, bits=2, order="area_rows")
    assert enc.bits == 2 and enc.perm is None
    assert enc.n_lt == ref.n_lt and enc.nnz == ref.nnz and enc.n_payload == ref.n_payload
    assert np.array_equal(enc.bitmaps, ref.bitmaps)
    assert np.array_equal(enc.offsets, ref.offsets)
    assert np.array_equal(enc.payload, ref.payload)


@pytest.mark.parametrize("N", [0, 1, 8, 32])
def test_w2_pmr_matches_oracle(N):
    W, _, _ = synth.random_problem(128, 512, 1, 0.5, 9, bits=2)
    got, want = binding.pmr(binding.encode(W, bits=2), N), iebme.pmr_report(iebme.encode(W, bits=2, order="area_rows"), N)
    for key in ("nnz", "stored_values", "n_lt", "payload_stored_bytes", "bitmap_bytes", "offset_bytes",
                "meta_bytes"):
        assert got[key] == want[key], key
    for key in ("payload_useful_bytes", "pmr", "pmr_stored", "ci_eff"):
        assert got[key] == pytest.approx(want[key], rel=1e-12), key


@pytest.mark.parametrize("value", [2, -3, 7, -8])
def test_w2_range_errors(value):
    W = np.zeros((32, 128), dtype=np.int8)
    W[5, 77] = value
    s = binding.IEBME()
    assert binding.lib().us_encode_w2(W.ctypes.data, 32, 128, 128, ctypes.byref(s)) == -3
    assert not s.bitmaps


def test_w2_refuses_reordering_in_the_binding():
    with pytest.raises(ValueError):
        binding.encode(np.zeros((16, 64), dtype=np.int8), reorder=True, bits=2)


@pytest.mark.slow
def test_w2_encoder_full_size():
    w = synth.WORKLOADS["ffn_down_4096x11008_s50"]
    W = synth.weights(w, bits=2)
    enc, ref = binding.encode(W, bits=2), iebme.encode(W, bits=2, order="area_rows")
    assert np.array_equal(enc.offsets, ref.offsets)
    assert np.array_equal(enc.payload, ref.payload)
    assert np.array_equal(enc.bitmaps, ref.bitmaps)
