"""Host-side checks of the C-ABI library (no GPU needed).

* the shared library loads and exports every symbol the headers declare;
* us_encode is byte-identical to the oracle's encoding;
* us_pmr agrees with the oracle's byte accounting (Eq. 1, Eq. 2);
* every argument error is reported before any work.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import iebme
from paper_2608_09291_amd import binding, synth

# The value order the library's encoders write: the areas of an area row
# interleaved by rank.
LIB_ORDER = "area_rows"

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_symbols():
    names = set()
    for h in ("us.h", "us_probe.h"):
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(us_[a-z0-9_]+)\s*\(", text))
    return names


def test_library_exports_every_declared_symbol():
    L = binding.lib()
    declared = _declared_symbols()
    assert declared == set(binding.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name


def test_status_strings():
    L = binding.lib()
    for code in binding.STATUS:
        assert L.us_status_string(code)


def _assert_same_encoding(enc, ref):
    assert enc.n_lt == ref.n_lt and enc.nnz == ref.nnz and enc.n_payload == ref.n_payload
    assert np.array_equal(enc.bitmaps, ref.bitmaps)
    assert np.array_equal(enc.offsets, ref.offsets)
    assert np.array_equal(enc.payload, ref.payload)


@pytest.mark.parametrize("M,K,s,seed,skew", [
    (16, 64, 0.5, 0, False), (48, 192, 0.3, 1, False), (64, 256, 0.7, 2, False),
    (32, 128, 0.0, 3, False), (32, 128, 1.0, 4, False), (80, 320, 0.9, 5, False),
    (256, 512, 0.6, 6, True), (512, 512, 0.5, 7, False)])
def test_encoder_matches_oracle(M, K, s, seed, skew):
    W, _, _ = synth.random_problem(M, K, 1, s, seed, row_skew=skew)
    _assert_same_encoding(binding.encode(W), iebme.encode(W, order=LIB_ORDER))


def test_encoder_matches_oracle_worked_tile(golden):
    # A 16 x 64 tile whose union-mask rows 0..3 repeat the paper's 16-bit rows twice.
    rows = [int(h, 16) for h in golden["union_bitmap"]["mask_rows_lsb_is_leftmost"]]
    rng = np.random.default_rng(1)
    W = np.zeros((16, 64), dtype=np.int8)
    for i, h in enumerate(rows):
        for j in range(32):
            if (h >> (j % 16)) & 1:
                q = int(rng.integers(4))
                a, c = divmod(q, 2)
                W[8 * a + i, 32 * c + j] = synth.nonzero_int4(rng, 1)[0]
    _assert_same_encoding(binding.encode(W), iebme.encode(W, order=LIB_ORDER))


@pytest.mark.slow
def test_encoder_matches_oracle_full_size():
    w = synth.WORKLOADS["ffn_down_4096x11008_s50"]
    W = synth.weights(w)
    enc, ref = binding.encode(W), iebme.encode(W, order=LIB_ORDER)
    _assert_same_encoding(enc, ref)
    rep = binding.pmr(enc, N=8)
    assert rep["pmr"] == pytest.approx(iebme.pmr_report(ref, N=8)["pmr"], rel=1e-12)


@pytest.mark.parametrize("N", [0, 1, 8, 32])
def test_pmr_matches_oracle(N):
    W, _, _ = synth.random_problem(128, 512, 1, 0.5, 9)
    enc, ref = binding.encode(W), iebme.encode(W, order=LIB_ORDER)
    got, want = binding.pmr(enc, N), iebme.pmr_report(ref, N)
    for key in ("nnz", "stored_values", "n_lt", "payload_stored_bytes", "bitmap_bytes",
                "offset_bytes", "meta_bytes"):
        assert got[key] == want[key], key
    for key in ("payload_useful_bytes", "pmr", "pmr_stored", "ci_eff"):
        assert got[key] == pytest.approx(want[key], rel=1e-12), key


def test_pmr_detects_corrupt_offsets():
    W, _, _ = synth.random_problem(32, 128, 1, 0.5, 3)
    enc = binding.encode(W)
    enc.offsets[2] += 4
    r = binding.PMRReport()
    assert binding.lib().us_pmr(ctypes.byref(enc.struct()), 0, ctypes.byref(r)) == -6


def _encode_status(W, M=None, K=None, ldw=None, null_out=False):
    W = np.ascontiguousarray(W, dtype=np.int8)
    M = W.shape[0] if M is None else M
    K = W.shape[1] if K is None else K
    ldw = K if ldw is None else ldw
    s = binding.IEBME()
    out = None if null_out else ctypes.byref(s)
    return binding.lib().us_encode(W.ctypes.data, M, K, ldw, out), s


@pytest.mark.parametrize("case,status", [
    ("m_not_16", -2), ("k_not_64", -2), ("zero_m", -2), ("negative_k", -2),
    ("ldw_small", -1), ("null_out", -1), ("value_8", -3), ("value_minus_9", -3)])
def test_encode_errors(case, status):
    W = np.zeros((32, 128), dtype=np.int8)
    kw = {}
    if case == "m_not_16":
        kw = dict(M=24)
    elif case == "k_not_64":
        kw = dict(K=96)
    elif case == "zero_m":
        kw = dict(M=0)
    elif case == "negative_k":
        kw = dict(K=-64)
    elif case == "ldw_small":
        kw = dict(ldw=64)
    elif case == "null_out":
        kw = dict(null_out=True)
    elif case == "value_8":
        W[3, 5] = 8
    elif case == "value_minus_9":
        W[31, 127] = -9
    got, s = _encode_status(W, **kw)
    assert got == status
    assert not s.bitmaps and s.n_lt == 0          # nothing written on error


def test_encode_null_weights():
    s = binding.IEBME()
    assert binding.lib().us_encode(None, 16, 64, 64, ctypes.byref(s)) == -1


def test_encode_with_row_stride():
    W, _, _ = synth.random_problem(32, 128, 1, 0.5, 12)
    big = np.zeros((32, 200), dtype=np.int8)
    big[:, :128] = W
    big[:, 128:] = 99                 # outside the matrix: never read
    s = binding.IEBME()
    assert binding.lib().us_encode(big.ctypes.data, 32, 128, 200, ctypes.byref(s)) == 0
    enc = binding.Encoded(s)
    _assert_same_encoding(enc, iebme.encode(W, order=LIB_ORDER))


def _dev_struct(M=32, K=128, n_lt=None, n_payload=0, ptr=0x1000):
    n_lt = (M // 16) * (K // 64) if n_lt is None else n_lt
    return binding.IEBMEDev(ptr, ptr, ptr, M, K, n_lt, n_payload)


@pytest.mark.parametrize("case,status", [
    ("null_w", -1), ("null_x", -1), ("null_y", -1), ("scale_without_yf", -1),
    ("m_not_16", -2), ("k_not_64", -2), ("k_too_big", -2), ("n_zero", -2), ("n_1025", -2),
    ("n_lt_wrong", -6), ("payload_odd", -6), ("payload_too_big", -6),
    ("split_3", -1), ("variant", -1), ("misaligned_x", -1), ("misaligned_perm", -1),
    ("bits_3", -6), ("bits_2_reordered", -1), ("single_pass_no_split", -1), ("k_blocks_chunked", -1),
    ("k_blocks_no_ws", -1), ("k_blocks_small_ws", -1), ("k_blocks_65", -1), ("single_pass_n17", -1),
    ("single_pass_ch_5", -1), ("misaligned_ws", -1)])
def test_spmm_argument_errors_before_launch(case, status):
    """Every argument error returns before touching the GPU (pointers are fake)."""
    L = binding.lib()
    w = _dev_struct()
    x, y, sc, yf = 0x2000, 0x3000, None, None
    N = 8
    opts = binding.SpmmOpts(0, 0)
    wp = ctypes.byref(w)
    ws, ws_bytes = None, 0
    if case == "null_w":
        wp = None
    elif case == "null_x":
        x = None
    elif case == "null_y":
        y = None
    elif case == "scale_without_yf":
        sc = 0x4000
    elif case == "m_not_16":
        w.M = 40
    elif case == "k_not_64":
        w.K = 100
    elif case == "k_too_big":
        w.K, w.M = 131072, 16
        w.n_lt = 2048
    elif case == "n_zero":
        N = 0
    elif case == "n_1025":
        N = 1025
    elif case == "n_lt_wrong":
        w.n_lt += 1
    elif case == "payload_odd":
        w.n_payload = 6
    elif case == "payload_too_big":
        w.n_payload = 32 * 128 + 4
    elif case == "split_3":
        opts.split_k = 3
    elif case == "variant":
        opts.variant = 4
    elif case == "single_pass_no_split":           # the single pass needs an explicit split
        opts.variant = 3
    elif case == "k_blocks_chunked":               # K blocks across workgroups: single pass only
        opts.k_blocks = 2
    elif case == "k_blocks_no_ws":
        opts.split_k, opts.variant, opts.k_blocks = 1, 3, 2
    elif case == "k_blocks_small_ws":
        opts.split_k, opts.variant, opts.k_blocks = 1, 3, 2
        ws, ws_bytes = 0x6000, 4 * 32 * 8
    elif case == "k_blocks_65":
        opts.split_k, opts.variant, opts.k_blocks = 1, 3, 65
        ws, ws_bytes = 0x6000, 1 << 20
    elif case == "single_pass_n17":
        opts.split_k, opts.variant = 1, 3
        N = 17
    elif case == "single_pass_ch_5":
        opts.split_k, opts.variant, opts.chunk_lts = 1, 3, 5
    elif case == "misaligned_ws":
        ws, ws_bytes = 0x6002, 1 << 20
    elif case == "misaligned_x":
        x = 0x2002
    elif case == "misaligned_perm":
        w.perm = 0x5004
    elif case == "bits_3":
        w.bits = 3
    elif case == "bits_2_reordered":
        w.bits, w.perm = 2, 0x5000
    got = L.us_spmm(wp, x, N, y, sc, yf, ws, ws_bytes, ctypes.byref(opts), None)
    assert got == status


def test_gemm_argument_errors():
    L = binding.lib()
    assert L.us_gemm_i8(None, 0x10, 16, 64, 1, 0x20, None) == -1
    assert L.us_gemm_i8(0x10, 0x10, 17, 64, 1, 0x20, None) == -2
    assert L.us_gemm_i8(0x10, 0x10, 16, 64, 1025, 0x20, None) == -2
    assert L.us_gemm_i8(0x18, 0x10, 16, 64, 1, 0x20, None) == -1


def test_workspace_size():
    # No workspace unless the K range is split across workgroups; then int32
    # accumulators for min(N, 16) columns and one ticket per 16-row block.
    assert binding.workspace_size(4096, 11008, 8) == 0
    assert binding.workspace_size(4096, 11008, 8, split_k=4, variant=3) == 0
    for N in (1, 8, 16, 32):
        assert binding.workspace_size(4096, 11008, N, split_k=4, variant=3, k_blocks=4) == \
            4 * 4096 * min(N, 16) + 4 * 256
    with pytest.raises(binding.UsError):
        binding.workspace_size(4096, 11008, 0)
    with pytest.raises(binding.UsError):
        binding.workspace_size(4096, 11008, 8, k_blocks=2)          # needs the single pass


def test_probe_argument_errors():
    L = binding.lib()
    assert L.us_probe_read(None, 16, 0x10, 0, None) == -1
    assert L.us_probe_read(0x10, 15, 0x10, 0, None) == -1
    assert L.us_probe_read(0x10, 16, 0x10, -1, None) == -1
    assert L.us_probe_read(0x10, 16, 0x10, binding.PROBE_READ_SHAPES, None) == -1
    assert L.us_probe_copy(0x10, 0x18, 16, None) == -1
    assert L.us_probe_copy_lds(0x10, 0x18, 16, None) == -1
    assert L.us_probe_copy_lds(0x10, 0x20, (1 << 31) + 16, None) == -1
    assert L.us_probe_spin(2 * 10 ** 9, None) == -1


def test_pack_int4_layout():
    Xt = np.array([[-8, 7, 0, -1]], dtype=np.int8)
    assert binding.pack_int4(Xt).tolist() == [[0x78, 0xF0]]


# The launch plan (host only; with no GPU visible the library plans for a
# 256-CU MI355X, which is also what the GPU reports).
@pytest.mark.parametrize("M,K,N,plan", [
    (4096, 11008, 8, (16, 11, 1)),     # one generation of 16-wavefront workgroups
    (12288, 4096, 8, (4, 16, 2)),      # the ring lets three workgroups share a CU
    (28672, 8192, 1, (2, 16, 1)),      # a cost tie at up to 4 columns goes to fewer wavefronts: 2 x 16
    (12288, 4096, 1, (4, 16, 1)),      # the same tie: 4 x 16 rather than 8 x 8
    (28672, 7168, 8, (4, 4, 1)),       # 4-LT chunks keep seven wavefronts per SIMD in one generation
    (12288, 49152, 4, (4, 16, 1)),     # the same tie, level in time with 8 x 8
    (1024, 4096, 1, (16, 4, 1)),       # 64 row blocks for 256 CUs: the tie keeps more wavefronts
    (28672, 7168, 1, (2, 8, 1)),       # fewer wavefronts on a tie, but at least 8 per CU (not 1 x 16)
    (28672, 8192, 2, (2, 11, 1)),      # up to 4 columns, a linear stage rather than a ring
    (28672, 8192, 32, (2, 4, 1)),      # two column blocks, 1792 row blocks: two generations would cost more
    (4096, 11008, 32, (16, 4, 1)),     # 256 row blocks: one generation, so 16 slices of three 4-LT chunks
])
def test_plan_choices(M, K, N, plan):
    assert binding.spmm_plan(M, K, N) == plan


@pytest.mark.parametrize("reordered", [False, True])
@pytest.mark.parametrize("M,K", [(16, 64), (512, 512), (4096, 11008), (12288, 4096), (48, 130048)])
@pytest.mark.parametrize("N", [1, 8, 16, 17, 32])
def test_plan_invariants(M, K, N, reordered):
    nkb = K // 64
    for split in (0, 1, 2, 4, 8, 16):
        for variant in (0, 1, 2):
            if variant == 2 and N > 16:
                with pytest.raises(binding.UsError):
                    binding.spmm_plan(M, K, N, split, variant, reordered)
                continue
            try:
                s, ch, stg = binding.spmm_plan(M, K, N, split, variant, reordered)
            except binding.UsError:
                # A forced ring with a fixed split may fit no configuration;
                # automatic choices always fit.
                assert variant == 2 and split != 0
                continue
            assert s in (1, 2, 4, 8, 16) and s <= nkb
            if split:
                assert s == min(split, 1 << (nkb.bit_length() - 1))
            assert ch in ((4, 8) if N > 16 else (4, 8, 11, 16))
            assert stg in (1, 2) and (variant == 0 or stg == variant)
            assert stg == 1 or ch in (11, 16)


def test_plan_argument_errors():
    L = binding.lib()
    a, b, c, d = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    ok = ctypes.byref(binding.SpmmOpts(0, 0))
    ra, rb, rc, rd = ctypes.byref(a), ctypes.byref(b), ctypes.byref(c), ctypes.byref(d)
    assert L.us_spmm_plan(32, 128, 8, 4, 0, ok, None, rb, rc, rd) == -1
    assert L.us_spmm_plan(40, 128, 8, 4, 0, ok, ra, rb, rc, rd) == -2
    assert L.us_spmm_plan(32, 128, 1025, 4, 1, ok, ra, rb, rc, rd) == -2
    bad = ctypes.byref(binding.SpmmOpts(3, 0))
    assert L.us_spmm_plan(32, 128, 8, 4, 0, bad, ra, rb, rc, rd) == -1
    bad = ctypes.byref(binding.SpmmOpts(0, 5))
    assert L.us_spmm_plan(32, 128, 8, 4, 1, bad, ra, rb, rc, rd) == -1
    assert L.us_spmm_plan(32, 128, 8, 3, 0, ok, ra, rb, rc, rd) == -1
    assert L.us_spmm_plan(32, 128, 8, 2, 1, ok, ra, rb, rc, rd) == -1
    # The K-block output may be omitted.
    assert L.us_spmm_plan(32, 128, 8, 4, 0, ok, ra, rb, rc, None) == 0


@pytest.mark.parametrize("bits,reordered", [(4, False), (4, True), (2, False)])
@pytest.mark.parametrize("M,K", [(16, 64), (512, 512), (1024, 4096), (4096, 11008)])
@pytest.mark.parametrize("N", [1, 8, 16])
def test_single_pass_plans(M, K, N, bits, reordered):
    """Single-pass plans (variant 3): every wavefront gets 1..ch LTs of its
    workgroup's K block, the stage fits the LDS, and the plan echoes the
    forced choices; impossible ones are refused."""
    nkb = K // 64
    accepted = 0
    for split in (1, 2, 4, 8, 16):
        for kb in (1, 2, 4, 8):
            for ch in (0, 4, 8, 11, 16, 22, 32):
                rmin, rmax = nkb // kb, -(-nkb // kb)
                try:
                    s, c, stg, k = binding.spmm_plan(M, K, N, split, 3, reordered, bits, ch, kb, full=True)
                except binding.UsError:
                    # Refused: no slice length fits, or the stage does not fit the LDS.
                    continue
                accepted += 1
                assert (s, stg, k) == (split, 3, kb)
                assert c in (4, 8, 11, 16, 22, 32) and (ch == 0 or c == ch)
                assert rmin >= split and -(-rmax // split) <= c
                if ch == 0:      # the shortest slice length that holds every wavefront's LTs
                    assert all(-(-rmax // split) > c2 for c2 in (4, 8, 11, 16, 22, 32) if c2 < c)
    assert accepted > 0
