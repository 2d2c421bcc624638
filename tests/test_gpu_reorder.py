"""GPU parity of us_spmm on row-reordered IE-BME matrices (Section V-B).

The encoder moves rows inside every LT; the kernel must route each reordered
row back to its original output row, so Y is the plain product of the
original W and X, bit for bit, and the expected values come from the oracle's
int64 product of the original (not reordered) matrix.
"""
import numpy as np
import pytest

from paper_2608_09291_amd import binding, synth
from test_gpu_spmm import SMALL, _random_cases, announce, check, run_spmm, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,K,N,s,seed", SMALL)
def test_reordered_small_parity(torch_cuda, M, K, N, s, seed):
    announce(f"reordered small M={M} K={K} N={N} s={s} seed={seed}")
    W, Xt, sc = synth.random_problem(M, K, N, s, seed)
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc, reorder=True)
    check(Y, Yf, W, Xt, sc)


@pytest.mark.parametrize("split_k", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("N", [1, 8, 16, 32])
def test_reordered_every_split(torch_cuda, split_k, N):
    M, K = 64, 2496                                    # 39 LTs per row block
    announce(f"reordered split M={M} K={K} N={N} split={split_k}")
    W, Xt, sc = synth.random_problem(M, K, N, 0.5, 700 + split_k)
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc, split_k=split_k, reorder=True)
    check(Y, Yf, W, Xt, sc)


@pytest.mark.parametrize("variant", [1, 2])
@pytest.mark.parametrize("M,K,N,s,split_k", [
    (32, 2368, 8, 0.5, 2),       # 37 LTs per row block
    (32, 2368, 1, 0.3, 1),
    (48, 4736, 16, 0.5, 1),      # 74 LTs: several chunks, odd last chunk
    (64, 1216, 4, 0.0, 1),       # every group active
    (64, 704, 8, 0.5, 1),        # 11 LTs: one ring chunk of 11
])
def test_reordered_staging_variants(torch_cuda, variant, M, K, N, s, split_k):
    announce(f"reordered staging variant={variant} M={M} K={K} N={N} s={s} split={split_k}")
    W, Xt, sc = synth.random_problem(M, K, N, s, 800 + 7 * variant + split_k)
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc, split_k=split_k, variant=variant, reorder=True)
    check(Y, Yf, W, Xt, sc)


@pytest.mark.parametrize("M,K,N,s,split_k,variant,seed", _random_cases(30, seed=20261203))
def test_reordered_random_shapes(torch_cuda, M, K, N, s, split_k, variant, seed):
    announce(f"reordered random M={M} K={K} N={N} s={s} split={split_k} variant={variant} seed={seed}")
    W, Xt, sc = synth.random_problem(M, K, N, s, seed)
    try:
        Y, Yf = run_spmm(torch_cuda, W, Xt, sc, split_k=split_k, variant=variant, reorder=True)
    except binding.UsError:
        assert variant == 2 and split_k != 0
        return
    check(Y, Yf, W, Xt, sc)


def test_reordered_planted_pairs(torch_cuda):
    """Identical row pairs over disjoint columns: permutations far from the identity."""
    announce("reordered planted pairs M=64 K=1024 N=16")
    rng = np.random.default_rng(12)
    M, K = 64, 1024
    W = np.zeros((M, K), dtype=np.int8)
    for mb in range(M // 16):
        for kb in range(K // 64):
            rows = rng.permutation(16)
            cols = rng.permutation(32)
            for k in range(8):
                u, v = rows[2 * k:2 * k + 2]
                for j in cols[4 * k:4 * k + 4]:
                    for c in range(2):
                        if rng.random() < 0.7:
                            W[16 * mb + u, 64 * kb + 32 * c + j] = synth.nonzero_int4(rng, 1)[0]
                            W[16 * mb + v, 64 * kb + 32 * c + j] = synth.nonzero_int4(rng, 1)[0]
    Xt = rng.integers(-8, 8, size=(16, K), dtype=np.int8)
    enc = binding.encode(W, reorder=True)
    assert np.any(enc.perm != enc.perm[0])             # the LTs really are permuted differently
    Y, _ = run_spmm(torch_cuda, W, Xt, reorder=True)
    check(Y, None, W, Xt)


def test_reordered_single_rows(torch_cuda):
    """Each LT row alone, with its partner rows empty: every lane row's routing."""
    announce("reordered single rows M=16 K=128 N=16")
    rng = np.random.default_rng(13)
    Xt = rng.integers(-8, 8, size=(16, 128), dtype=np.int8)
    for r in range(16):
        W = np.zeros((16, 128), dtype=np.int8)
        W[r, :] = synth.nonzero_int4(rng, 128)
        W[(r + 5) % 16, ::3] = 7
        Y, _ = run_spmm(torch_cuda, W, Xt, reorder=True)
        check(Y, None, W, Xt)


_cache = {}


@pytest.mark.parametrize("name,N", [("ffn_down_4096x11008_s50", 8), ("qkv_12288x4096_s50", 8),
                                    ("ffn_13824x5120_skew60", 16), ("ffn_28672x8192_s70", 1),
                                    ("ffn_28672x8192_s70", 32)])
def test_reordered_full_size_parity(torch_cuda, name, N):
    announce(f"reordered full {name} N={N}")
    if name not in _cache:
        _cache.clear()
        w = synth.WORKLOADS[name]
        W = synth.weights(w)
        _cache[name] = (w, W, binding.to_device(binding.encode(W, reorder=True)))
    w, W, dev = _cache[name]
    Xt = synth.activations(w, N)
    sc = synth.scales(w) if w.dequant else None
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc, dev=dev)
    check(Y, Yf, W, Xt, sc)
