"""The single-pass kernel family (us_spmm_opts.variant = 3), forced, against the oracle.

Every instantiation family (4-bit at N <= 4 and N <= 16, row-reordered,
2-bit) for each slice length, with one workgroup per row block and with
the K range split across workgroups (the paper's split-K batches with a
reduction workspace); the workspace must be left zero-filled by every
call, so that the next call (here: a second, narrower one) needs no
clearing. Expected values come from the oracle only.
"""
import numpy as np
import pytest

from paper_2608_09291_amd import binding, synth
from test_gpu_spmm import announce, check, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

CHS = (4, 8, 11, 16, 22, 32)


def _run(torch, W, Xt, sc, split, ch, kb, reorder=False, bits=4, ws=None, dev=None):
    M, K = W.shape
    N = Xt.shape[0]
    if dev is None:
        dev = binding.to_device(binding.encode(W, reorder=reorder, bits=bits))
    xp = torch.from_numpy(binding.pack_int4(Xt)).cuda()
    y = torch.full((N, M), -1, dtype=torch.int32, device="cuda")
    s = None if sc is None else torch.from_numpy(sc).cuda()
    yf = None if sc is None else torch.full((N, M), float("nan"), dtype=torch.float32, device="cuda")
    binding.spmm(dev, xp, N, y, s, yf, split_k=split, variant=3, chunk_lts=ch, k_blocks=kb, ws=ws)
    torch.cuda.synchronize()
    return y.cpu().numpy().T, (None if yf is None else yf.cpu().numpy().T)


def _cases():
    out = []
    for family in ("plain", "reordered", "w2"):
        for N in (1, 3, 8, 16):
            for ch in CHS:
                for split, kb in ((2, 1), (1, 3), (4, 2)):
                    out.append((family, N, ch, split, kb))
    return out


@pytest.mark.parametrize("family,N,ch,split,kb", _cases())
def test_forced_single_pass(torch_cuda, family, N, ch, split, kb):
    torch = torch_cuda
    # K gives every wavefront exactly ch LTs except the last K block, which is shorter.
    nkb = ch * split * kb - (ch - 1 if kb > 1 else 0)
    M, K = 48, 64 * nkb
    announce(f"single pass {family} N={N} ch={ch} split={split} k_blocks={kb} K={K}")
    bits = 2 if family == "w2" else 4
    W, Xt, sc = synth.random_problem(M, K, N, 0.45, 700 + ch + 5 * N + 11 * kb, bits=bits)
    plan = binding.spmm_plan(M, K, N, split, 3, reordered=family == "reordered", bits=bits, chunk_lts=ch,
                             k_blocks=kb, full=True)
    assert plan == (split, ch, 3, kb)
    nbytes = binding.workspace_size(M, K, N, split_k=split, variant=3, chunk_lts=ch, k_blocks=kb)
    ws = torch.zeros(max(1, nbytes // 4), dtype=torch.int32, device="cuda") if kb > 1 else None
    Y, Yf = _run(torch, W, Xt, sc, split, ch, kb, reorder=family == "reordered", bits=bits, ws=ws)
    check(Y, Yf, W, Xt, sc)
    if ws is not None:
        assert int(ws.count_nonzero().item()) == 0, "workspace not left zero-filled"


def test_workspace_reuse_across_calls(torch_cuda):
    """Two calls in a row on one workspace, the second with another shape: no
    clearing between them."""
    torch = torch_cuda
    ws = torch.zeros(binding.workspace_size(1024, 4096, 16, split_k=4, variant=3, k_blocks=4) // 4,
                     dtype=torch.int32, device="cuda")
    for (M, K, N, kb) in ((1024, 4096, 16, 4), (512, 2048, 5, 3), (1024, 4096, 1, 2)):
        announce(f"workspace reuse M={M} K={K} N={N} k_blocks={kb}")
        W, Xt, sc = synth.random_problem(M, K, N, 0.5, 800 + N)
        Y, Yf = _run(torch, W, Xt, sc, 4, 0, kb, ws=ws)
        check(Y, Yf, W, Xt, sc)
        assert int(ws.count_nonzero().item()) == 0


def test_too_small_workspace_is_refused(torch_cuda):
    torch = torch_cuda
    W, Xt, sc = synth.random_problem(64, 1024, 8, 0.5, 9)
    need = binding.workspace_size(64, 1024, 8, split_k=2, variant=3, k_blocks=2)
    ws = torch.zeros(need // 4 - 1, dtype=torch.int32, device="cuda")
    with pytest.raises(binding.UsError):
        _run(torch, W, Xt, sc, 2, 0, 2, ws=ws)


@pytest.mark.parametrize("name,N,split,ch,kb", [
    ("ffn_down_4096x11008_s50", 8, 16, 11, 1),
    ("ffn_down_4096x11008_s50", 8, 8, 11, 2),
    ("kv_1024x4096_s50", 8, 8, 4, 2),
    ("kv_512x3584_s50", 8, 4, 4, 4),
    ("qkv_12288x4096_s50", 1, 4, 16, 1),
])
def test_full_size_single_pass(torch_cuda, name, N, split, ch, kb):
    torch = torch_cuda
    w = synth.WORKLOADS[name]
    announce(f"single pass full size {name} N={N} {split}x{ch} k_blocks={kb}")
    W = synth.weights(w)
    Xt = synth.activations(w, N)
    sc = synth.scales(w) if w.dequant else None
    nbytes = binding.workspace_size(w.M, w.K, N, split_k=split, variant=3, chunk_lts=ch, k_blocks=kb)
    ws = torch.zeros(max(1, nbytes // 4), dtype=torch.int32, device="cuda") if kb > 1 else None
    Y, Yf = _run(torch, W, Xt, sc, split, ch, kb, ws=ws)
    check(Y, Yf, W, Xt, sc)


def test_graph_capture_split_replays(torch_cuda):
    # A split across workgroups leaves its workspace zeroed, so a captured
    # call needs no clearing between replays (and records no memset). Two
    # calls on one workspace are captured once after an eager warm-up;
    # between replays the activations are rewritten in place and the
    # outputs poisoned by eager work, and every replay is checked against
    # the oracle for the inputs it saw. The same holds for the
    # no-allocation entry point, whose array is captured by address.
    torch = torch_cuda
    announce("graph capture, single pass split over 2 workgroups: M=256 K=4096 N=8 and N=3")
    M, K = 256, 4096
    W, _, sc = synth.random_problem(M, K, 8, 0.5, 61)
    dev = binding.to_device(binding.encode(W))
    nbytes = binding.workspace_size(M, K, 8, 4, binding.VARIANT_BURST, 8, 2)
    assert nbytes > 0
    ws = torch.zeros(nbytes // 4, dtype=torch.int32, device="cuda")
    xa = torch.zeros((8, K // 2), dtype=torch.uint8, device="cuda")
    xb = torch.zeros((3, K // 2), dtype=torch.uint8, device="cuda")
    ya = torch.empty((8, M), dtype=torch.int32, device="cuda")
    yfa = torch.empty((8, M), dtype=torch.float32, device="cuda")
    yb = torch.empty((3, M), dtype=torch.int32, device="cuda")
    yc = torch.empty((3, M), dtype=torch.int32, device="cuda")
    s = torch.from_numpy(sc).cuda()
    opts = dict(split_k=4, variant=binding.VARIANT_BURST, chunk_lts=8, k_blocks=2)

    def calls():
        binding.spmm(dev, xa, 8, ya, s, yfa, ws=ws, **opts)
        binding.spmm(dev, xb, 3, yb, ws=ws, **opts)
        binding.spmm_noalloc(dev, xb, 3, yc, **opts)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        calls()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        calls()
    rng = np.random.default_rng(62)
    for rep in range(4):
        XA = rng.integers(-8, 8, size=(8, K), dtype=np.int8)
        XB = rng.integers(-8, 8, size=(3, K), dtype=np.int8)
        xa.copy_(torch.from_numpy(binding.pack_int4(XA)))
        xb.copy_(torch.from_numpy(binding.pack_int4(XB)))
        for t in (ya, yb, yc):
            t.fill_(-1)
        yfa.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        check(ya.cpu().numpy().T, yfa.cpu().numpy().T, W, XA, sc)
        check(yb.cpu().numpy().T, None, W, XB)
        check(yc.cpu().numpy().T, None, W, XB)
        assert int((ws != 0).sum().item()) == 0, rep
