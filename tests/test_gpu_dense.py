"""GPU parity of the dense INT8 GEMM comparison point and the measurement probes."""
import sys

import numpy as np
import pytest

from oracle import product
from paper_2608_09291_amd import binding, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.lib()
    return torch


def announce(msg):
    sys.stderr.write(f"[gpu case] {msg}\n")
    sys.stderr.flush()


@pytest.mark.parametrize("M,K,N,seed", [(16, 64, 1, 0), (64, 640, 8, 1), (128, 4096, 17, 2),
                                        (4096, 11008, 8, 3), (512, 2048, 32, 4)])
def test_gemm_i8_parity(torch_cuda, M, K, N, seed):
    announce(f"gemm M={M} K={K} N={N}")
    torch = torch_cuda
    rng = np.random.default_rng(seed)
    W = rng.integers(-128, 128, size=(M, K), dtype=np.int8)
    Xt = rng.integers(-128, 128, size=(N, K), dtype=np.int8)
    w = torch.from_numpy(W).cuda()
    x = torch.from_numpy(Xt).cuda()
    y = torch.full((N, M), -7, dtype=torch.int32, device="cuda")
    binding.gemm_i8(w, x, M, K, N, y)
    torch.cuda.synchronize()
    assert np.array_equal(y.cpu().numpy().T, product.to_int32(product.matmul_c(W, Xt)))


def test_probe_read_and_copy(torch_cuda):
    torch = torch_cuda
    announce("probe read/copy 8 MiB")
    n = 8 << 20
    rng = np.random.default_rng(1)
    host = rng.integers(0, 256, size=n, dtype=np.uint8)
    src = torch.from_numpy(host).cuda()
    words = binding.probe_read_sink_words(n)
    expect = np.bitwise_xor.reduce(host.view(np.uint32))
    for shape in range(binding.PROBE_READ_SHAPES):
        sink = torch.zeros(words, dtype=torch.int32, device="cuda")
        binding.probe_read(src, n, sink, shape)
        torch.cuda.synchronize()
        assert np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32)) == expect, shape
    dst = torch.zeros(n, dtype=torch.uint8, device="cuda")
    binding.probe_copy(src, dst, n)
    torch.cuda.synchronize()
    assert np.array_equal(dst.cpu().numpy(), host)
    # Through LDS, also with a ragged tail (not a whole 1 KB step).
    for m in (n, n - 16 * 37):
        dst = torch.zeros(n, dtype=torch.uint8, device="cuda")
        binding.probe_copy_lds(src, dst, m)
        torch.cuda.synchronize()
        got = dst.cpu().numpy()
        assert np.array_equal(got[:m], host[:m]) and not got[m:].any(), m


def test_probe_spin_returns(torch_cuda):
    torch = torch_cuda
    announce("probe spin 2 ms")
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    binding.probe_spin(2_000_000)
    end.record()
    torch.cuda.synchronize()
    assert 1.5 <= start.elapsed_time(end) < 200
