"""GPU parity for activation widths beyond one kernel pass (N > 32, prefill sizes).

us_spmm and us_gemm_i8 run such N as slabs of 32 columns, each slab with its
own launch configuration and its own offsets into X, Y and the dequantised
Y. Y must equal the oracle's int64 product for every column, including the
ragged last slab.
"""
import numpy as np
import pytest

from oracle import product
from paper_2608_09291_amd import binding, synth
from test_gpu_spmm import announce, check, run_spmm, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,K,N,s,seed", [
    (32, 640, 33, 0.5, 1),       # one full slab and a 1-column slab
    (48, 1280, 48, 0.3, 2),
    (64, 1024, 64, 0.5, 3),      # two full slabs
    (16, 2496, 65, 0.7, 4),
    (128, 768, 100, 0.5, 5),     # 32 + 32 + 32 + 4
    (64, 4096, 128, 0.6, 6),
    (32, 512, 256, 0.5, 7),
    (16, 128, 1024, 0.5, 8),     # the widest accepted
])
def test_wide_n_parity(torch_cuda, M, K, N, s, seed):
    announce(f"wide N M={M} K={K} N={N} s={s}")
    W, Xt, sc = synth.random_problem(M, K, N, s, seed)
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc)
    check(Y, Yf, W, Xt, sc)


@pytest.mark.parametrize("split_k", [1, 4, 16])
def test_wide_n_every_split(torch_cuda, split_k):
    announce(f"wide N split={split_k}")
    W, Xt, sc = synth.random_problem(64, 2496, 70, 0.5, 20 + split_k)
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc, split_k=split_k)
    check(Y, Yf, W, Xt, sc)


def test_wide_n_two_bit_and_reordered(torch_cuda):
    announce("wide N with 2-bit weights and with reordering")
    W, Xt, sc = synth.random_problem(48, 1280, 72, 0.5, 31, bits=2)
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc, bits=2)
    check(Y, Yf, W, Xt, sc)
    W, Xt, sc = synth.random_problem(48, 1280, 72, 0.5, 32)
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc, reorder=True)
    check(Y, Yf, W, Xt, sc)


def test_wide_n_full_size(torch_cuda):
    w = synth.WORKLOADS["ffn_down_4096x11008_s50"]
    announce("wide N full 4096x11008 N=96")
    W = synth.weights(w)
    Xt = synth.activations(w, 96)
    assert np.array_equal(Xt[:32], synth.activations(w, 32))     # the first 32 columns never change
    sc = synth.scales(w)
    Y, Yf = run_spmm(torch_cuda, W, Xt, sc)
    check(Y, Yf, W, Xt, sc)


@pytest.mark.parametrize("N", [33, 64, 100])
def test_wide_n_dense_gemm(torch_cuda, N):
    torch = torch_cuda
    announce(f"dense gemm N={N}")
    rng = np.random.default_rng(N)
    M, K = 64, 512
    W = rng.integers(-128, 128, size=(M, K), dtype=np.int8)
    Xt = rng.integers(-128, 128, size=(N, K), dtype=np.int8)
    y = torch.full((N, M), -1, dtype=torch.int32, device="cuda")
    binding.gemm_i8(torch.from_numpy(W).cuda(), torch.from_numpy(Xt).cuda(), M, K, N, y)
    torch.cuda.synchronize()
    assert np.array_equal(y.cpu().numpy().T, product.to_int32(product.matmul_c(W, Xt)))
