"""GPU parity of us_spmm on 2-bit IE-BME matrices (the W2A4 setting, Section VII).

Weights are signed 2-bit values packed four to a byte; the kernel places
them as 64 v and shifts the sums by 10. Y must equal the oracle's int64
product of the same W and X bit for bit.
"""
import numpy as np
import pytest

from paper_2608_09291_amd import binding, synth
from test_gpu_spmm import SMALL, _random_cases, announce, check, run_spmm, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,K,N,s,seed", SMALL)
def test_w2_small_parity(torch_cuda, M, K, N, s, seed):
    announce(f"w2 small M={M} K={K} N={N} s={s} seed={seed}")
    W, Xt, sc = synth.random_problem(M, K, N, s, seed, bits=2)
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc, bits=2)
    check(Y, Yf, W, Xt, sc)


@pytest.mark.parametrize("split_k", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("N", [1, 8, 16, 32])
def test_w2_every_split(torch_cuda, split_k, N):
    M, K = 64, 2496                                    # 39 LTs per row block
    announce(f"w2 split M={M} K={K} N={N} split={split_k}")
    W, Xt, sc = synth.random_problem(M, K, N, 0.5, 900 + split_k, bits=2)
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc, split_k=split_k, bits=2)
    check(Y, Yf, W, Xt, sc)


@pytest.mark.parametrize("variant", [1, 2])
@pytest.mark.parametrize("M,K,N,s,split_k", [
    (32, 2368, 8, 0.5, 2),
    (32, 2368, 1, 0.3, 1),
    (48, 4736, 16, 0.5, 1),      # 74 LTs: several chunks
    (64, 1216, 4, 0.0, 1),       # every group active
    (64, 704, 8, 0.5, 1),        # 11 LTs in one chunk
])
def test_w2_staging_variants(torch_cuda, variant, M, K, N, s, split_k):
    announce(f"w2 staging variant={variant} M={M} K={K} N={N} s={s} split={split_k}")
    W, Xt, sc = synth.random_problem(M, K, N, s, 950 + 7 * variant + split_k, bits=2)
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc, split_k=split_k, variant=variant, bits=2)
    check(Y, Yf, W, Xt, sc)


@pytest.mark.parametrize("M,K,N,s,split_k,variant,seed", _random_cases(30, seed=20261204))
def test_w2_random_shapes(torch_cuda, M, K, N, s, split_k, variant, seed):
    announce(f"w2 random M={M} K={K} N={N} s={s} split={split_k} variant={variant} seed={seed}")
    W, Xt, sc = synth.random_problem(M, K, N, s, seed, bits=2)
    try:
        Y, Yf = run_spmm(torch_cuda, W, Xt, sc, split_k=split_k, variant=variant, bits=2)
    except binding.UsError:
        assert variant == 2 and split_k != 0
        return
    check(Y, Yf, W, Xt, sc)


def test_w2_extreme_values_at_k_max(torch_cuda):
    """All -2 weights times all -8 activations at the largest K: Y = 16 K."""
    K = binding.K_MAX
    announce(f"w2 extreme M=16 K={K} N=2")
    W = np.full((16, K), -2, dtype=np.int8)
    W[1::2, :] = 1
    Xt = np.full((2, K), -8, dtype=np.int8)
    Xt[1, ::2] = 7
    Y, _ = run_spmm(torch_cuda, W, Xt, bits=2)
    check(Y, None, W, Xt)
    assert Y[0, 0] == 16 * K


def test_w2_single_positions(torch_cuda):
    """Each LT position alone: every lane, segment and 2-bit slot of the placement."""
    announce("w2 single positions M=16 K=64 N=16")
    rng = np.random.default_rng(19)
    Xt = rng.integers(-8, 8, size=(16, 64), dtype=np.int8)
    for r in range(16):
        for kk in range(0, 64, 5):
            W = np.zeros((16, 64), dtype=np.int8)
            W[r, kk] = -2 if (r + kk) % 2 else 1
            W[(r + 3) % 16, (kk + 9) % 64] = -1
            Y, _ = run_spmm(torch_cuda, W, Xt, bits=2)
            check(Y, None, W, Xt)


_cache = {}


@pytest.mark.parametrize("name,N", [("ffn_down_4096x11008_s50", 8), ("qkv_12288x4096_s50", 1),
                                    ("qkv_12288x4096_s50", 32), ("ffn_13824x5120_skew60", 16),
                                    ("ffn_28672x8192_s70", 1)])
def test_w2_full_size_parity(torch_cuda, name, N):
    announce(f"w2 full {name} N={N}")
    if name not in _cache:
        _cache.clear()
        w = synth.WORKLOADS[name]
        W = synth.weights(w, bits=2)
        _cache[name] = (w, W, binding.to_device(binding.encode(W, bits=2)))
    w, W, dev = _cache[name]
    Xt = synth.activations(w, N)
    sc = synth.scales(w) if w.dequant else None
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc, dev=dev)
    check(Y, Yf, W, Xt, sc)
