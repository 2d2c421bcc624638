"""Pins that tie the CPU oracle to the paper and to plain mathematics.

Each test checks the oracle against something other than itself: values the
paper prints for its worked examples, closed forms for special matrices,
invariants of the format, brute force on tiny inputs, and statistics of
i.i.d. masks. A plausible slip in the oracle (a transposed operand, an
inclusive rank, a swapped area order, a wrong nibble half) fails at least one.
"""
import itertools

import numpy as np
import pytest

from oracle import iebme, product
from paper_2608_09291_amd import synth

# --------------------------------------------------------------------------
# Worked examples printed in the paper
# --------------------------------------------------------------------------


def _lt_with_mask(rows_hex, hb, kb, ra, ca, rng):
    """An (ra*hb) x (ca*kb) tile whose union mask is rows_hex (LSB = leftmost).

    Every active position gets a nonzero value in a varying, nonempty subset
    of the areas, so the union (not any single area) produces the mask.
    """
    W = np.zeros((ra * hb, ca * kb), dtype=np.int8)
    for i, h in enumerate(rows_hex):
        for j in range(kb):
            if (h >> j) & 1:
                subset = [q for q in range(ra * ca) if rng.random() < 0.5] or [int(rng.integers(ra * ca))]
                for q in subset:
                    a, c = divmod(q, ca)
                    W[a * hb + i, c * kb + j] = synth.nonzero_int4(rng, 1)[0]
    return W


def test_union_bitmap_worked_example(golden):
    g = golden["union_bitmap"]
    lt_h, lt_w = g["lt_shape"]
    ra, ca = g["ra"], g["ca"]
    hb, kb = lt_h // ra, lt_w // ca
    rows = [int(h, 16) for h in g["mask_rows_lsb_is_leftmost"]]
    rng = np.random.default_rng(7)
    lt = _lt_with_mask(rows, hb, kb, ra, ca, rng)
    W = np.concatenate([lt, np.zeros_like(lt)], axis=1)   # a second, empty LT after it
    enc = iebme.encode(W, lt_h=lt_h, lt_w=lt_w, ra=ra, ca=ca)
    assert enc.words_per_lt == 1
    word = int(enc.bitmaps[0])
    for i, h in enumerate(rows):
        assert (word >> (16 * i)) & 0xFFFF == h
        assert bin(h).count("1") == g["active_bits_per_row"]
    assert word == 0xB6DA5B6D6DB636DB
    assert int(enc.P[0]) == g["P_t"]
    assert int(enc.offsets[1]) == g["next_offset"] == g["Q_times_P_t"]
    assert int(enc.offsets[2]) == g["next_offset"]          # the empty LT adds nothing
    assert np.array_equal(iebme.decode(enc), W)


def test_zero_retention_example(golden):
    # Group [1, 3, 5, 0] across areas 0..3 at (0, 0); group [0, 0, 0, 0] at (0, 1);
    # one more single-area group at (0, 2) to give the streams length 2.
    W = np.zeros((16, 64), dtype=np.int8)
    vals = [1, 3, 5, 0]
    for q, v in enumerate(vals):
        a, c = divmod(q, 2)
        W[8 * a + 0, 32 * c + 0] = v
    W[8, 2] = -8                     # area 2 only, position (0, 2)
    enc = iebme.encode(W)
    B = iebme.union_mask(enc)[0]
    assert B[0, 0] and not B[0, 1] and B[0, 2]
    assert int(enc.P[0]) == 2
    assert enc.n_payload == 8        # Q * P_t values, the kept zero included
    cv = iebme.unpack_nibbles(enc.payload, enc.n_payload)
    streams = cv.reshape(4, 2)       # V^(q)[rho]
    assert list(streams[:, 0]) == vals
    assert list(streams[:, 1]) == [0, 0, -8, 0]
    assert golden["zero_retention"]["printed_group"][3] == 0


def test_lspd_segment_example(golden):
    g = golden["lspd_segment"]
    G = g["G"]
    bits = [int(c) for c in g["segment_bits_left_to_right"]]
    assert [p for p, b in enumerate(bits) if b] == g["active_positions"]
    # Union mask row 1, segment 1 holds the pattern; row 0 has 3 active bits
    # and segment 0 of row 1 has 2, so idx_base = 5.
    Bt = np.zeros((8, 32), dtype=bool)
    Bt[0, [4, 9, 30]] = True
    Bt[1, [1, 6]] = True
    Bt[1, G:2 * G] = bits
    base = iebme.lspd_idx_base(Bt, 1, 1, G)
    assert base == 5
    streams = [np.arange(100, 140) + 1000 * q for q in range(4)]
    seg = iebme.lspd_segment(Bt, 1, 1, G, streams)
    for q in range(4):
        want = [0] * G
        for p, k in zip(g["active_positions"], g["payload_index_offsets"]):
            want[p] = int(streams[q][base + k])
        assert seg[q] == want
    # As an LSB-first byte the segment is 0x2D.
    assert sum(b << p for p, b in enumerate(bits)) == 0x2D


# --------------------------------------------------------------------------
# Closed forms for special matrices
# --------------------------------------------------------------------------


def test_all_zero_matrix():
    W = np.zeros((32, 128), dtype=np.int8)
    enc = iebme.encode(W)
    assert enc.n_lt == 4
    assert not enc.bitmaps.any()
    assert enc.offsets.tolist() == [0] * 5
    assert enc.payload.size == iebme.TAIL_PAD_BYTES and not enc.payload.any()
    assert enc.nnz == 0
    assert np.array_equal(iebme.decode(enc), W)
    rep = iebme.pmr_report(enc, N=8)
    assert rep["meta_bytes"] == 36 * 4 and rep["pmr"] == 0.0 and rep["ci_eff"] == 0.0


def test_dense_matrix_closed_form():
    """No zeros: P_t = 256, o_t = 1024 t, payload = areas 0..3 row-major, in LT order."""
    rng = np.random.default_rng(3)
    M, K = 32, 128
    W = synth.nonzero_int4(rng, (M, K))
    enc = iebme.encode(W)
    assert np.all(enc.bitmaps == np.uint64(0xFFFFFFFFFFFFFFFF))
    assert np.array_equal(enc.offsets, 1024 * np.arange(5))
    expect = []
    for mb in range(M // 16):               # row-block-major LT order
        for kb in range(K // 64):
            T = W[16 * mb:16 * mb + 16, 64 * kb:64 * kb + 64]
            for a in range(2):              # q = a * 2 + c
                for c in range(2):
                    expect.extend(T[8 * a:8 * a + 8, 32 * c:32 * c + 32].ravel().tolist())
    # Nibble n in byte n // 2, low half for even n, 4-bit two's complement.
    by = enc.payload
    for n in range(0, len(expect), 97):
        b = int(by[n // 2])
        nib = (b & 0xF) if n % 2 == 0 else (b >> 4)
        assert (nib - 16 if nib >= 8 else nib) == expect[n]
    rep = iebme.pmr_report(enc)
    assert rep["pmr"] == pytest.approx(0.5 * 1024 / 36)


def test_nibble_twos_complement():
    packed = iebme.pack_nibbles(np.array([-8, -1, 7, 0, 3]))
    assert packed[:3].tolist() == [0xF8, 0x07, 0x03]
    assert iebme.unpack_nibbles(packed, 5).tolist() == [-8, -1, 7, 0, 3]


# --------------------------------------------------------------------------
# Invariants, round trip, LSPD equivalence
# --------------------------------------------------------------------------


@pytest.mark.parametrize("M,K,s,seed", [(16, 64, 0.5, 0), (48, 192, 0.3, 1), (64, 256, 0.7, 2),
                                        (32, 128, 0.0, 3), (32, 128, 1.0, 4), (80, 320, 0.9, 5)])
def test_round_trip_and_invariants(M, K, s, seed):
    W, _, _ = synth.random_problem(M, K, 1, s, seed)
    enc = iebme.encode(W)
    assert np.array_equal(iebme.decode(enc), W)
    # offsets[n_lt] = 4 * total popcount of the bitmaps
    pop = sum(bin(int(x)).count("1") for x in enc.bitmaps)
    assert int(enc.offsets[-1]) == 4 * pop
    # stored - nnz = zeros kept inside active groups, counted directly from W
    kept_zeros = 0
    for mb, kb in itertools.product(range(M // 16), range(K // 64)):
        T = W[16 * mb:16 * mb + 16, 64 * kb:64 * kb + 64]
        groups = np.stack([T[8 * a:8 * a + 8, 32 * c:32 * c + 32] for a in range(2) for c in range(2)])
        active = (groups != 0).any(axis=0)
        kept_zeros += int(((groups == 0) & active[None]).sum())
    rep = iebme.pmr_report(enc)
    assert rep["stored_values"] - rep["nnz"] == kept_zeros
    assert rep["meta_bytes"] == 36 * enc.n_lt
    assert rep["pmr"] == pytest.approx(0.5 * np.count_nonzero(W) / (36 * enc.n_lt))


@pytest.mark.parametrize("G", [8, 16, 32])
def test_lspd_decode_matches_definition(G):
    W, _, _ = synth.random_problem(32, 128, 1, 0.6, 11)
    enc = iebme.encode(W)
    dense = iebme.decode(enc)
    for t in range(enc.n_lt):
        mb, kb = divmod(t, 2)
        assert np.array_equal(iebme.lspd_decode_tile(enc, t, G),
                              dense[16 * mb:16 * mb + 16, 64 * kb:64 * kb + 64])


def test_expected_active_groups_iid():
    """E[P_t] = 256 (1 - s^4) for an i.i.d. mask (a group is inactive iff all 4 are pruned)."""
    s = 0.5
    W, _, _ = synth.random_problem(1024, 1024, 1, s, 21)   # 1024 LTs
    enc = iebme.encode(W)
    mean = enc.P.mean()
    p = 1 - s ** 4
    sd = np.sqrt(256 * p * (1 - p) / enc.n_lt)
    assert abs(mean - 256 * p) < 5 * sd


def test_rejects_bad_input():
    with pytest.raises(ValueError):
        iebme.encode(np.zeros((15, 64), dtype=np.int8))
    with pytest.raises(ValueError):
        iebme.encode(np.zeros((16, 60), dtype=np.int8))
    with pytest.raises(ValueError):
        iebme.encode(np.full((16, 64), 8, dtype=np.int8))
    enc = iebme.encode(synth.random_problem(16, 64, 1, 0.5, 0)[0])
    enc.offsets[1] += 4
    with pytest.raises(ValueError):
        iebme.decode(enc)


# --------------------------------------------------------------------------
# The product, its epilogue and Eq. 1 / Eq. 2
# --------------------------------------------------------------------------


def _brute(W, Xt):
    M, K = W.shape
    N = Xt.shape[0]
    Y = [[0] * N for _ in range(M)]
    for m in range(M):
        for n in range(N):
            acc = 0
            for k in range(K):
                acc += int(W[m][k]) * int(Xt[n][k])
            Y[m][n] = acc
    return np.array(Y, dtype=np.int64)


@pytest.mark.parametrize("M,K,N,s", [(16, 64, 1, 0.5), (32, 128, 3, 0.7), (16, 128, 8, 0.0)])
def test_product_brute_force(M, K, N, s):
    W, Xt, _ = synth.random_problem(M, K, N, s, 5)
    want = _brute(W, Xt)
    assert np.array_equal(product.matmul_c(W, Xt), want)
    assert np.array_equal(product.matmul_np(W, Xt), want)
    assert np.array_equal(product.matmul_np(iebme.decode(iebme.encode(W)), Xt), want)


def test_product_extremes_fit_int32():
    K = 11008
    W = np.full((16, K), -8, dtype=np.int8)
    Xt = np.full((2, K), -8, dtype=np.int8)
    Y = product.to_int32(product.matmul_c(W, Xt))
    assert np.all(Y == 64 * K)


def test_dequant_is_one_rounding():
    Y = np.array([[3, -7], [16777215, 1]], dtype=np.int64)
    sc = np.array([0.1, 0.5], dtype=np.float32)
    got = product.dequant(Y, sc)
    # float64 holds the product of two float32 values exactly, so rounding it
    # once to float32 is the correctly rounded float32 product.
    want = (Y.astype(np.float64) * sc.astype(np.float64)[:, None]).astype(np.float32)
    assert got.dtype == np.float32 and np.array_equal(got, want)
    # By hand: fl32(0.1) = 0.100000001490116..., times 3 = 0.3000000044703...,
    # whose float32 neighbours are 0x3E999999 and 0x3E99999A; the nearer is 0x3E99999A.
    assert got[0, 0].view(np.uint32) == 0x3E99999A
    assert got[1, 0] == 8388607.5          # (2**24 - 1) / 2 is exact in float32
    assert got[1, 1] == 0.5


def test_ci_eq2_hand_value():
    # M=4096, N=8, s=0.5, PMR=64/9: numerator 2*4096*8*0.5 = 32768;
    # denominator 0.5*4096*0.5*(1 + 9/64) + 0.5*8 = 1024*73/64 + 4 = 1172 -> 32768/1172.
    assert iebme.ci_eff(4096, 11008, 8, 0.5, 64 / 9) == pytest.approx(32768 / 1172)
    # K cancels; infinite PMR leaves payload-only traffic.
    assert iebme.ci_eff(4096, 1, 8, 0.5, 64 / 9) == iebme.ci_eff(4096, 10 ** 6, 8, 0.5, 64 / 9)
    assert iebme.ci_eff(4096, 64, 8, 0.5, 1e300) == pytest.approx(32768 / (1024 + 4))
