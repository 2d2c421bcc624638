"""Every kernel configuration, forced, against the oracle; and the largest matrix.

The host normally picks the configuration; here each (chunk length, staging)
pair is forced with us_spmm_opts for every kernel family (4-bit in stored
order at N <= 4, N <= 16 and N <= 32, row-reordered, 2-bit), once with one
chunk per slice and once with several, so that every instantiation that can
be launched runs at least once.
"""
import numpy as np
import pytest

from paper_2608_09291_amd import binding, synth
from test_gpu_spmm import announce, check, run_spmm, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

CFGS = [(4, 1), (8, 1), (11, 1), (16, 1), (16, 2), (11, 2)]     # (chunk LTs, staging)


def _cases():
    out = []
    for family in ("plain", "reordered", "w2"):
        for N in (3, 12, 24):
            for ch, stg in CFGS:
                if N > 16 and (ch > 8 or stg == 2):
                    continue
                for nlt, split in ((ch, 2), (3 * ch + 1, 1)):       # one chunk / several chunks
                    out.append((family, N, ch, stg, nlt, split))
    return out


@pytest.mark.parametrize("family,N,ch,stg,nlt,split", _cases())
def test_forced_configuration(torch_cuda, family, N, ch, stg, nlt, split):
    K = 64 * nlt * split
    M = 32
    announce(f"config {family} N={N} chunk={ch} staging={stg} K={K} split={split}")
    bits = 2 if family == "w2" else 4
    W, Xt, sc = synth.random_problem(M, K, N, 0.4, 40 + ch + 3 * N + nlt, bits=bits)
    plan = binding.spmm_plan(M, K, N, split, stg, reordered=family == "reordered", bits=bits, chunk_lts=ch)
    assert plan == (split, ch, stg)
    dev = binding.to_device(binding.encode(W, reorder=family == "reordered", bits=bits))
    xp = torch_cuda.from_numpy(binding.pack_int4(Xt)).cuda()
    y = torch_cuda.full((N, M), -1, dtype=torch_cuda.int32, device="cuda")
    s = torch_cuda.from_numpy(sc).cuda()
    yf = torch_cuda.full((N, M), float("nan"), dtype=torch_cuda.float32, device="cuda")
    binding.spmm(dev, xp, N, y, s, yf, split_k=split, variant=stg, chunk_lts=ch)
    torch_cuda.cuda.synchronize()
    check(y.cpu().numpy().T, yf.cpu().numpy().T, W, Xt, sc)


def test_largest_matrix(torch_cuda):
    """M K just below 2^32 with every position active: offsets near the uint32
    limit and a 2 GiB payload. Checked on sampled rows, one by one."""
    torch = torch_cuda
    M, K, N = 33024, binding.K_MAX, 2
    assert M * K < 2 ** 32 and (M + 16) * K >= 2 ** 32
    announce(f"largest M={M} K={K} N={N}")
    # A dense, deterministic INT4 pattern without zeros: W[m, k] is the
    # ((7 m + 3 k + (k >> 6)(m >> 4)) mod 15)-th nonzero INT4 value. It
    # depends on the row block j = m >> 4 only through j mod 15, so 15
    # distinct 16-row blocks are built and copied.
    values = np.array([v for v in range(-8, 8) if v != 0], dtype=np.int8)
    table = values[np.arange(64) % 15]                 # index sums stay below 64
    k = np.arange(K, dtype=np.int64)
    b = ((3 * k) % 15).astype(np.uint8)
    kk = ((k >> 6) % 15).astype(np.uint8)
    blocks = []
    for j in range(15):
        a = ((7 * (16 * j + np.arange(16))) % 15).astype(np.uint8)[:, None]
        c = (kk * np.uint8(j)) % np.uint8(15)
        blocks.append(table[a + (b + c)[None, :]])
    W = np.empty((M, K), dtype=np.int8)
    for j in range(M // 16):
        W[16 * j:16 * j + 16] = blocks[j % 15]
    assert not (W == 0).any()
    rng = np.random.default_rng(5)
    Xt = rng.integers(-8, 8, size=(N, K), dtype=np.int8)
    enc = binding.encode(W)
    assert enc.n_payload == M * K                      # all 1024 positions of every LT
    assert int(enc.offsets[-1]) == M * K
    dev = binding.to_device(enc)
    del enc
    xp = torch.from_numpy(binding.pack_int4(Xt)).cuda()
    y = torch.full((N, M), -1, dtype=torch.int32, device="cuda")
    binding.spmm(dev, xp, N, y)
    torch.cuda.synchronize()
    Y = y.cpu().numpy().T
    rows = np.unique(np.concatenate([rng.integers(0, M, size=48), [0, 1, 15, 16, M - 17, M - 16, M - 1]]))
    for m in rows:
        want = W[m].astype(np.int64) @ Xt.T.astype(np.int64)
        assert np.array_equal(Y[m], want), (m, Y[m], want)
