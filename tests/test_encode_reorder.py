"""The native reordering encoder (us_encode_reordered) against the oracle.

The oracle's row reordering (Section V-B) is pinned in test_reorder_pins.py.
Both sides resolve DP ties the same documented way, so the whole encoding
(bitmaps, offsets, payload and permutation words) must agree byte for byte;
what is unique whatever the tie rule (each LT's optimal union-mask size,
and the decoded matrix) is checked as well.
"""
import ctypes

import numpy as np
import pytest

from oracle import iebme, reorder
from paper_2608_09291_amd import binding, synth


def _check_against_oracle(W):
    enc = binding.encode(W, reorder=True)
    ref, perms = reorder.encode_reordered(W, order="area_rows")
    assert enc.n_lt == ref.n_lt and enc.nnz == ref.nnz and enc.n_payload == ref.n_payload
    assert np.array_equal(enc.perm, reorder.perm_words(perms))
    assert np.array_equal(enc.bitmaps, ref.bitmaps)
    assert np.array_equal(enc.offsets, ref.offsets)
    assert np.array_equal(enc.payload, ref.payload)
    return enc, ref, perms


@pytest.mark.parametrize("M,K,s,seed,skew", [
    (16, 64, 0.5, 0, False), (48, 192, 0.3, 1, False), (64, 256, 0.7, 2, False),
    (32, 128, 0.0, 3, False), (32, 128, 1.0, 4, False), (80, 320, 0.9, 5, False),
    (128, 512, 0.6, 6, True), (64, 1024, 0.5, 7, False)])
def test_reordered_encoder_matches_oracle(M, K, s, seed, skew):
    W, _, _ = synth.random_problem(M, K, 1, s, seed, row_skew=skew)
    enc, ref, perms = _check_against_oracle(W)
    # Unique whatever the tie rule: the optimal size of every LT's union mask.
    _, _, costs = reorder.reorder(W)
    assert np.array_equal(np.diff(enc.offsets.astype(np.int64)), 4 * costs)
    assert np.array_equal(reorder.undo_reorder(iebme.decode(ref), perms), W.astype(np.int64))


def test_reordered_encoder_planted_pairs():
    # Rows in identical pairs over disjoint columns: one optimum, known permutation.
    rng = np.random.default_rng(3)
    W = np.zeros((32, 128), dtype=np.int8)
    for mb in range(2):
        for kb in range(2):
            rows = rng.permutation(16)
            cols = rng.permutation(32)
            for k in range(8):
                u, v = sorted(rows[2 * k:2 * k + 2])
                for j in cols[4 * k:4 * k + 4]:
                    c = int(rng.integers(2))
                    W[16 * mb + u, 64 * kb + 32 * c + j] = W[16 * mb + v, 64 * kb + 32 * c + j] = 5
    enc, _, _ = _check_against_oracle(W)
    assert enc.n_payload == 4 * 32 * 4        # 32 active union-mask entries per LT


def test_reordering_never_grows_the_payload():
    W, _, _ = synth.random_problem(256, 1024, 1, 0.5, 21)
    plain, reo = binding.encode(W), binding.encode(W, reorder=True)
    P_plain = np.diff(plain.offsets.astype(np.int64))
    P_reo = np.diff(reo.offsets.astype(np.int64))
    assert np.all(P_reo <= P_plain)
    assert reo.nnz == plain.nnz
    assert plain.perm is None


def test_reordered_pmr_counts_permutations():
    W, _, _ = synth.random_problem(64, 256, 1, 0.5, 4)
    enc = binding.encode(W, reorder=True)
    rep = binding.pmr(enc, N=8)
    assert rep["perm_bytes"] == 8 * enc.n_lt
    assert rep["meta_bytes"] == 36 * enc.n_lt          # Eq. 1 metadata is unchanged
    assert binding.pmr(binding.encode(W), N=8)["perm_bytes"] == 0


@pytest.mark.parametrize("case,status", [("m_not_16", -2), ("k_not_64", -2), ("ldw_small", -1),
                                         ("value_8", -3)])
def test_reordered_encode_errors(case, status):
    W = np.zeros((32, 128), dtype=np.int8)
    M, K, ldw = 32, 128, 128
    if case == "m_not_16":
        M = 24
    elif case == "k_not_64":
        K = 96
    elif case == "ldw_small":
        ldw = 64
    elif case == "value_8":
        W[7, 9] = 8
    s = binding.IEBME()
    assert binding.lib().us_encode_reordered(W.ctypes.data, M, K, ldw, ctypes.byref(s)) == status
    assert not s.perm and not s.bitmaps


@pytest.mark.slow
def test_reordered_encoder_full_size_sampled():
    """The bench matrix: costs of sampled LTs equal the oracle's optimum."""
    w = synth.WORKLOADS["ffn_down_4096x11008_s50"]
    W = synth.weights(w)
    enc = binding.encode(W, reorder=True)
    P = np.diff(enc.offsets.astype(np.int64)) // 4
    rng = np.random.default_rng(0)
    nkb = W.shape[1] // 64
    for t in rng.choice(enc.n_lt, size=40, replace=False):
        mb, kb = divmod(int(t), nkb)
        T = W[16 * mb:16 * mb + 16, 64 * kb:64 * kb + 64]
        pi, total = reorder.reorder_tile(T)
        assert P[t] == total
        assert int(enc.perm[t]) == int(reorder.perm_words(np.array([pi]))[0])
