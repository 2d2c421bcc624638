"""us_spmm_noalloc (no workspace argument: the library's per-device array)
against us_spmm with a caller workspace, through the C-ABI.

Two calls in a row, the second with a smaller matrix and fewer columns,
each with the K range split across workgroups so that the array is used;
the outputs must be bit-identical to us_spmm's (whose results the other GPU
tests check against the oracle), and to the oracle. Also an automatic plan
(no split, the array unused) and the size limit.
"""
import ctypes

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


def _both(torch, M, K, N, seed, opts):
    W, Xt, sc = synth.random_problem(M, K, N, 0.5, seed)
    dev = binding.to_device(binding.encode(W))
    xp = torch.from_numpy(binding.pack_int4(Xt)).cuda()
    s = torch.from_numpy(sc).cuda()
    outs = []
    for use_noalloc in (True, False):
        y = torch.full((N, M), -1, dtype=torch.int32, device="cuda")
        yf = torch.full((N, M), float("nan"), dtype=torch.float32, device="cuda")
        if use_noalloc:
            binding.spmm_noalloc(dev, xp, N, y, s, yf, **opts)
        else:
            nbytes = binding.workspace_size(M, K, N, **opts)
            ws = torch.zeros(max(1, nbytes // 4), dtype=torch.int32, device="cuda")
            binding.spmm(dev, xp, N, y, s, yf, ws=ws, **opts)
        torch.cuda.synchronize()
        outs.append((y.cpu().numpy(), yf.cpu().numpy()))
    (y0, f0), (y1, f1) = outs
    assert np.array_equal(y0, y1)
    assert np.array_equal(f0.view(np.uint32), f1.view(np.uint32))
    Y = product.to_int32(product.matmul_c(W, Xt))
    assert np.array_equal(y0.T, Y)
    assert np.array_equal(f0.T.view(np.uint32), product.dequant(Y, sc).view(np.uint32))


def test_noalloc_matches_us_spmm_twice(torch_cuda):
    # The second call reuses the array left by the first, with another shape.
    _both(torch_cuda, 1024, 4096, 16, 11, dict(split_k=8, variant=3, k_blocks=4))
    _both(torch_cuda, 512, 2048, 5, 12, dict(split_k=4, variant=3, k_blocks=3))


def test_noalloc_automatic_plan(torch_cuda):
    _both(torch_cuda, 256, 1600, 8, 13, {})


def test_noalloc_size_limit(torch_cuda):
    # A split whose workspace exceeds the array is refused before any launch.
    L = binding.lib()
    M, K, N = 65536, 64, 16
    need = binding.workspace_size(M, K, N, split_k=1, variant=3, k_blocks=2)
    assert need > binding.NOALLOC_SCRATCH_BYTES
    w = binding.IEBMEDev(0x1000, 0x1000, 0x1000, M, K, M // 16, 0)
    opts = binding.SpmmOpts(1, 3, 0, 2)
    assert L.us_spmm_noalloc(ctypes.byref(w), 0x2000, N, 0x3000, None, None, ctypes.byref(opts), None) == -2
