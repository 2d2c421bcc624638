"""Pipelined chunks, forced, against the oracle.

Above 16 activation columns, and at up to 16 with chunks of 11 or 16 LTs, a
slice of several chunks requests the first payload pieces of its next chunk
during the current chunk's last steps. The kernel has separate code for the
first chunk, the chunks in between and the last one, so these cases cover
slices of exactly two chunks (no middle chunk), two chunks with a one-LT
tail, and five chunks, at N = 17 (one column past the 16-column kernels) and
N = 32 with 4- and 8-LT chunks, and at N = 12 and 16 with 11- and 16-LT
chunks, for every weight form (reordered chunks longer than 4 LTs keep the
unpipelined order and are covered too). The row block's K range is one LT
short of an equal split, so the wavefronts of a workgroup hold slices of
different lengths (and, for some, a different number of chunks).
"""
import pytest

from paper_2608_09291_amd import binding, synth
from test_gpu_spmm import announce, check, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu


def _cases():
    out = []
    for family in ("plain", "reordered", "w2"):
        for Ns, chs in (((17, 32), (4, 8)), ((12, 16), (11, 16))):
            for N in Ns:
                for ch in chs:
                    for nlt in (ch + 1, 2 * ch, 5 * ch):
                        for split in (1, 4):
                            out.append((family, N, ch, nlt, split))
    return out


@pytest.mark.parametrize("family,N,ch,nlt,split", _cases())
def test_pipelined_chunks(torch_cuda, family, N, ch, nlt, split):
    torch = torch_cuda
    nkb = nlt * split - (1 if split > 1 else 0)            # slices of nlt and nlt - 1 LTs
    K, M = 64 * nkb, 48
    announce(f"pipelined {family} N={N} chunk={ch} K={K} split={split}")
    bits = 2 if family == "w2" else 4
    W, Xt, sc = synth.random_problem(M, K, N, 0.45, 700 + 7 * ch + N + nlt + split, bits=bits)
    reorder = family == "reordered"
    assert binding.spmm_plan(M, K, N, split, 1, reordered=reorder, bits=bits, chunk_lts=ch) == (split, ch, 1)
    dev = binding.to_device(binding.encode(W, reorder=reorder, bits=bits))
    xp = torch.from_numpy(binding.pack_int4(Xt)).cuda()
    y = torch.full((N, M), -1, dtype=torch.int32, device="cuda")
    s = torch.from_numpy(sc).cuda()
    yf = torch.full((N, M), float("nan"), dtype=torch.float32, device="cuda")
    binding.spmm(dev, xp, N, y, s, yf, split_k=split, variant=1, chunk_lts=ch)
    torch.cuda.synchronize()
    check(y.cpu().numpy().T, yf.cpu().numpy().T, W, Xt, sc)
