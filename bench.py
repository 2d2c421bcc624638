#!/usr/bin/env python3
"""Benchmark of the W4A4 IE-BME SpMM on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--N n] [--split-k S] [--reorder] [--bits 2]

One step is one us_spmm call (stream the IE-BME tiles, decode, multiply,
combine, store Y and the dequantised Y) over one copy of the encoded weight
matrix; the encoding itself is offline, as in the paper, and is not timed.
With --reorder the matrix is encoded after bitmap-aware row reordering
(Section V-B) and the kernel undoes the row permutation of every tile; with
--bits 2 the weights are 2-bit (the W2A4 setting of Section VII).
Every timed batch queues its launches behind a bounded spin kernel, so the
GPU runs them back to back and host launch cost never enters the event
timings; the weight copies rotate over at least 1 GiB so that none of them
can be served from the 256 MB Infinity Cache.

Prints one JSON line on stdout; details go to stderr.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2608_09291_amd import binding, synth  # noqa: E402

METRIC = "W4A4 SpMM µs/call, achieved HBM GB/s on encoded bytes, dense-equiv TOPS"
DEFAULT_WORKLOAD = "ffn_down_4096x11008_s50"
HBM_PEAK_GBS = 8000.0
ROTATE_BYTES = 1 << 30
ROUND_LAUNCHES = 200
KERNEL_SRCS = [os.path.join(ROOT, "paper_2608_09291_amd", "csrc", f)
               for f in ("us_spmm_kernel.h", "us_range.h", "us_spmm.hip", "us_spmm_narrow.hip", "us_spmm_perm.hip",
                         "us_spmm_w2.hip", "us_spmm_wide.hip", "us_spmm_wide8.hip", "us_spmm_burst.h", "us_spmm_burst_plain.hip",
                         "us_spmm_burst_narrow.hip", "us_spmm_burst_perm.hip", "us_spmm_burst_w2.hip")] + [
    os.path.join(ROOT, "paper_2608_09291_amd", "build.py")]      # its compiler flags shape the kernels too

# HBM traffic of one SpMM launch, read from rocprofv3 --pmc runs of this
# script (one pass for FETCH_SIZE, one for WRITE_SIZE; KiB per dispatch), each
# divided by what the same counter reads per byte copied by a copy kernel of
# known size. Both copy probes give the same factor: bench.py --copy-probe
# 268435456 copies 262144 KiB, and FETCH_SIZE reads 131082 KiB per dispatch
# with plain loads (--copy-kind plain) and 131083 KiB with the SpMM payload's
# non-temporal buffer loads straight into LDS (--copy-kind lds); WRITE_SIZE
# reads 262144 KiB for both: 0.50004 and 1.0 KiB per KiB copied. An entry
# holds only for the kernel sources whose SHA-256 (of the files in
# KERNEL_SRCS, concatenated) starts with `src`; after any change to them the
# traffic is unknown. Keyed by workload, N and row reordering.
COPY_FACTOR = {"FETCH_SIZE": 131083.0 / 262144.0, "WRITE_SIZE": 262144.0 / 262144.0}
MEASURED_TRAFFIC = {
    ("ffn_down_4096x11008_s50", 8, False): dict(src="18f3c274054a93c2", FETCH_SIZE=11374.3125, WRITE_SIZE=256.0),
}


def kernel_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for path in KERNEL_SRCS:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload: str, N: int, reordered: bool):
    """Counter-derived HBM bytes per launch, or None if not measured for this kernel source."""
    e = MEASURED_TRAFFIC.get((workload, N, reordered))
    if e is None or not kernel_source_hash().startswith(e["src"]):
        return None
    return int(round(sum(e[c] / COPY_FACTOR[c] for c in COPY_FACTOR) * 1024))


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(synth.WORKLOADS))
    ap.add_argument("--N", type=int, default=0, help="activation columns (default: the workload's first)")
    ap.add_argument("--split-k", type=int, default=0)
    ap.add_argument("--variant", type=int, default=0, choices=(0, 1, 2, 3),
                    help="us_spmm_opts.variant: 0 automatic, 1 whole / 2 ring staging, 3 single pass "
                         "(needs --split-k)")
    ap.add_argument("--chunk-lts", type=int, default=0, help="us_spmm_opts.chunk_lts (0: automatic)")
    ap.add_argument("--k-blocks", type=int, default=0,
                    help="us_spmm_opts.k_blocks: workgroups per row block with the single pass (0: one)")
    ap.add_argument("--reorder", action="store_true", help="row-reorder the LTs before encoding")
    ap.add_argument("--bits", type=int, default=4, choices=(4, 2), help="weight bits (4: W4A4, 2: W2A4)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-extras", action="store_true", help="skip the read-ceiling and dense GEMM points")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run the plain copy kernel over BYTES bytes, --steps times (the known "
                         "byte count that calibrates the FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--copy-kind", default="plain", choices=("plain", "lds"),
                    help="copy probe loads: plain vector loads, or the SpMM payload's non-temporal "
                         "buffer loads straight into LDS")
    return ap.parse_args()


class Timer:
    """GPU-side timing of back-to-back launches on the current stream."""

    def __init__(self, torch):
        self.torch = torch
        self.stream = torch.cuda.current_stream()

    def run(self, launch, count: int, per_launch_host_us: float = 20.0) -> float:
        """Total GPU milliseconds of `count` launches (launch(i) enqueues one).

        Each batch is queued behind a spin kernel that lasts twice the
        expected host enqueue time; a batch whose enqueue took longer than
        the spin (the GPU may then have idled waiting for the host) is timed
        again with a longer spin."""
        torch = self.torch
        total = 0.0
        done = 0
        retries = 0
        self.batches = []                                  # (ms, launches) per timed batch
        while done < count:
            n = min(ROUND_LAUNCHES, count - done)
            spin_ns = int(max(2e6, n * per_launch_host_us * 1e3 * 2))
            binding.probe_spin(spin_ns)
            start = torch.cuda.Event(enable_timing=True)
            end = torch.cuda.Event(enable_timing=True)
            t_host = time.perf_counter()
            start.record(self.stream)
            for i in range(n):
                launch(done + i)
            end.record(self.stream)
            t_host = time.perf_counter() - t_host
            end.synchronize()
            if t_host * 1e9 > 0.9 * spin_ns and retries < 4:
                per_launch_host_us *= 4
                retries += 1
                continue
            ms = start.elapsed_time(end)
            self.batches.append((ms, n))
            total += ms
            done += n
        return total


def spmm_bench(torch, args, w, N, timer, reorder=False, bits=4):
    W = synth.weights(w, bits)
    Xt = synth.activations(w, N)
    enc = binding.encode(W, reorder=reorder, bits=bits)
    rep = binding.pmr(enc, N)
    dev0 = binding.to_device(enc)
    enc_bytes = dev0.nbytes
    n_copies = max(2, -(-ROTATE_BYTES // enc_bytes))
    copies = [dev0] + [binding.DeviceEncoded(dev0.bitmaps.clone(), dev0.offsets.clone(),
                                             dev0.payload.clone(), dev0.M, dev0.K, dev0.n_lt,
                                             dev0.n_payload,
                                             None if dev0.perm is None else dev0.perm.clone(), dev0.bits)
                       for _ in range(n_copies - 1)]
    xp = torch.from_numpy(binding.pack_int4(Xt)).cuda()
    y = torch.empty((N, w.M), dtype=torch.int32, device="cuda")
    sc = yf = None
    if w.dequant:
        sc = torch.from_numpy(synth.scales(w)).cuda()
        yf = torch.empty((N, w.M), dtype=torch.float32, device="cuda")

    # Prebuilt C arguments: the timed loop only calls the library.
    L = binding.lib()
    structs = [c.struct() for c in copies]
    sptrs = [ctypes.byref(s) for s in structs]
    opts = binding.SpmmOpts(args.split_k, args.variant, args.chunk_lts, args.k_blocks)
    optp = ctypes.byref(opts)
    # A split across workgroups takes a zeroed reduction workspace, which
    # every call leaves zeroed again.
    ws_bytes = binding.workspace_size(w.M, w.K, N, args.split_k, args.variant, args.chunk_lts, args.k_blocks)
    ws = torch.zeros(max(1, ws_bytes // 4), dtype=torch.int32, device="cuda") if ws_bytes else None
    wsa = None if ws is None else ws.data_ptr()
    xa, ya = xp.data_ptr(), y.data_ptr()
    sca = None if sc is None else sc.data_ptr()
    yfa = None if yf is None else yf.data_ptr()
    sh = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    status = [0]

    def launch(i):
        st = L.us_spmm(sptrs[i % n_copies], xa, N, ya, sca, yfa, wsa, ws_bytes, optp, sh)
        if st:
            status[0] = st

    # Setup: every rotating copy is run once and must give copy 0's Y, so a
    # bad copy cannot go unnoticed. This also has the GPU map each copy's
    # pages before the timed calls, as the weights of a serving loop are
    # (each timed call still reads its copy from HBM: the copies together
    # are far larger than the last-level cache).
    launch(0)
    y0 = y.clone()
    for i in range(1, n_copies):
        launch(i)
        if not torch.equal(y, y0):
            raise RuntimeError(f"rotating copy {i} gives a different Y")
    torch.cuda.synchronize()
    if status[0]:
        raise binding.UsError("us_spmm", status[0])

    timer.run(launch, args.warmup)
    torch.cuda.synchronize()
    ms = timer.run(launch, args.steps)
    batches = [1e3 * b_ms / n for b_ms, n in timer.batches]   # µs per call, one value per timed batch
    if status[0]:
        raise binding.UsError("us_spmm", status[0])

    # Algorithmic bytes of one call: stored payload (zeros of active groups
    # included), bitmaps (32 B/LT), offsets (4 B/LT), row permutations (8 B/LT
    # when reordered), X, Y, and with the dequant epilogue the scales and the
    # float32 Y.
    alg = (rep["payload_stored_bytes"] + rep["bitmap_bytes"] + rep["offset_bytes"] + rep["perm_bytes"]
           + w.K * N // 2 + w.M * N * 4)
    if w.dequant:
        alg += w.M * 4 + w.M * N * 4
    return dict(W=W, Xt=Xt, enc=enc, rep=rep, ms=ms, alg_bytes=alg, enc_bytes=enc_bytes,
                n_copies=n_copies, y=y, yf=yf, batches=batches)


def read_ceiling(torch, nbytes, steps, timer):
    """Streaming-read time of HBM at the same byte count, same rotation: the
    fastest of the read probe's launch shapes. Returns (ms per read, shape)."""
    nbytes = (nbytes + 15) // 16 * 16
    n_copies = max(2, -(-ROTATE_BYTES // nbytes))
    bufs = [torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(i % 251) for i in range(n_copies)]
    sink = torch.empty(binding.probe_read_sink_words(nbytes), dtype=torch.int32, device="cuda")
    best = None
    for shape in range(binding.PROBE_READ_SHAPES):
        def launch(i, shape=shape):
            binding.probe_read(bufs[i % n_copies], nbytes, sink, shape)
        timer.run(launch, min(steps, 200))
        ms = timer.run(launch, steps) / steps
        if best is None or ms < best[0]:
            best = (ms, shape)
    del bufs
    return best


def dense_gemm(torch, w, N, steps, timer):
    """Dense INT8 GEMM of the same shape (1 byte per weight)."""
    nbytes = w.M * w.K
    n_copies = max(2, -(-ROTATE_BYTES // nbytes))
    rng = np.random.default_rng(0)
    W8 = torch.from_numpy(rng.integers(-128, 128, size=(w.M, w.K), dtype=np.int8)).cuda()
    mats = [W8] + [W8.clone() for _ in range(n_copies - 1)]
    x = torch.from_numpy(rng.integers(-128, 128, size=(N, w.K), dtype=np.int8)).cuda()
    y = torch.empty((N, w.M), dtype=torch.int32, device="cuda")
    timer.run(lambda i: binding.gemm_i8(mats[i % n_copies], x, w.M, w.K, N, y), min(steps, 200))
    ms = timer.run(lambda i: binding.gemm_i8(mats[i % n_copies], x, w.M, w.K, N, y), steps)
    del mats
    return ms / steps, nbytes + w.K * N + w.M * N * 4


def cpu_baseline(w, W, Xt, enc_bytes_alg, budget_s=12.0, bits=4):
    """The oracle's int64 masked dense product, timed on this host's cores."""
    from oracle import iebme, product
    product.build(force=False)
    threads = product.max_threads()
    t0 = time.perf_counter()
    ref = iebme.encode(W, bits=bits)
    dense = iebme.decode(ref).astype(np.int8)
    t_dec = time.perf_counter() - t0
    times = []
    t_start = time.perf_counter()
    while len(times) < 3 or (time.perf_counter() - t_start < budget_s and len(times) < 5000):
        t = time.perf_counter()
        product.matmul_c(dense, Xt)
        times.append(time.perf_counter() - t)
    med = float(np.median(times))
    # The same product on one core: a few calls, at most about 3 s.
    product.set_threads(1)
    one = []
    t_start = time.perf_counter()
    try:
        while len(one) < 1 or (time.perf_counter() - t_start < 3.0 and len(one) < 20):
            t = time.perf_counter()
            product.matmul_c(dense, Xt)
            one.append(time.perf_counter() - t)
    finally:
        product.set_threads(threads)
    med1 = float(np.median(one))
    return dict(value=round(enc_bytes_alg / med / 1e9, 4), unit="GB/s", cores=threads, kind="oracle",
                sample=(f"whole {w.M}x{w.K} matrix, N={Xt.shape[0]}: oracle int64 masked dense product "
                        f"(oracle/matmul_i64.c, OpenMP) over the oracle-decoded weights, median of "
                        f"{len(times)} calls = {med * 1e3:.1f} ms/call; on one core, median of {len(one)} "
                        f"calls = {med1 * 1e3:.1f} ms/call; oracle encode+decode (numpy) "
                        f"{t_dec:.2f} s, not included"),
                ms_per_call=round(med * 1e3, 3), single_core_ms_per_call=round(med1 * 1e3, 3),
                single_core_value=round(enc_bytes_alg / med1 / 1e9, 4))


def copy_probe(torch, args, timer):
    nbytes = (args.copy_probe + 15) // 16 * 16
    src = torch.full((nbytes,), 7, dtype=torch.uint8, device="cuda")
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    copy = binding.probe_copy_lds if args.copy_kind == "lds" else binding.probe_copy
    ms = timer.run(lambda i: copy(src, dst, nbytes), args.steps)
    torch.cuda.synchronize()
    if not bool((dst == 7).all()):
        raise RuntimeError("copy probe produced wrong bytes")
    us = ms * 1e3 / args.steps
    print(json.dumps({"probe": "copy", "kind": args.copy_kind, "bytes_read": nbytes, "bytes_written": nbytes,
                      "steps": args.steps,
                      "us_per_call": round(us, 3), "gbs": round(2 * nbytes / (us * 1e-6) / 1e9, 1)}),
          flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the library has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    binding.lib()
    if args.copy_probe:
        copy_probe(torch, args, Timer(torch))
        return
    w = synth.WORKLOADS[args.workload]
    N = args.N or w.Ns[0]
    timer = Timer(torch)

    log(f"[bench] workload {w.name} M={w.M} K={w.K} N={N} s={w.sparsity} dequant={w.dequant}")
    if args.bits == 2 and args.reorder:
        print("--reorder applies to 4-bit weights only", file=sys.stderr)
        sys.exit(2)
    r = spmm_bench(torch, args, w, N, timer, reorder=args.reorder, bits=args.bits)
    ms_step = r["ms"] / args.steps
    us = ms_step * 1e3
    gbs = r["alg_bytes"] / (ms_step * 1e-3) / 1e9
    tops = 2.0 * w.M * w.K * N / (ms_step * 1e-3) / 1e12
    log(f"[bench] us_spmm {us:.3f} us/call  {gbs:.1f} GB/s on {r['alg_bytes'] / 1e6:.2f} MB  "
        f"{tops:.1f} dense-equiv TOPS  ({r['n_copies']} rotating copies)")

    extras = {}
    if not args.no_extras:
        ceil_ms, ceil_shape = read_ceiling(torch, r["alg_bytes"], min(args.steps, 1000), timer)
        extras["read_ceiling_gbs"] = round(r["alg_bytes"] / (ceil_ms * 1e-3) / 1e9, 1)
        extras["read_ceiling_us"] = round(ceil_ms * 1e3, 3)
        extras["read_ceiling_shape"] = ceil_shape
        extras["kernel_of_read_ceiling"] = round(ceil_ms / ms_step, 3)
        g_ms, g_bytes = dense_gemm(torch, w, N, min(args.steps, 1000), timer)
        extras["dense_int8_gemm_us"] = round(g_ms * 1e3, 3)
        extras["dense_int8_gemm_gbs"] = round(g_bytes / (g_ms * 1e-3) / 1e9, 1)
        extras["speedup_vs_dense_int8"] = round(g_ms / ms_step, 3)
        # The floor of any dense INT8 kernel of this shape: the fastest plain
        # read of its bytes (weights, activations, Y), same rotation.
        d_ms, _ = read_ceiling(torch, g_bytes, min(args.steps, 1000), timer)
        extras["dense_int8_read_floor_us"] = round(d_ms * 1e3, 3)
        extras["speedup_vs_dense_int8_read_floor"] = round(d_ms / ms_step, 3)
        log(f"[bench] read ceiling {extras['read_ceiling_us']} us ({extras['read_ceiling_gbs']} GB/s); "
            f"dense int8 GEMM {extras['dense_int8_gemm_us']} us; plain read of the dense bytes "
            f"{extras['dense_int8_read_floor_us']} us")

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(w, r["W"], r["Xt"], r["alg_bytes"], bits=args.bits)
        log(f"[bench] cpu oracle {cpu['ms_per_call']} ms/call on {cpu['cores']} threads")

    rep = r["rep"]
    plan = binding.spmm_plan(w.M, w.K, N, args.split_k, args.variant, reordered=args.reorder, bits=args.bits,
                             chunk_lts=args.chunk_lts, k_blocks=args.k_blocks, full=True)
    out = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": w.name, "M": w.M, "K": w.K, "N": N, "sparsity": w.sparsity,
                   "dequant": w.dequant, "weight_bits": args.bits, "reordered": args.reorder,
                   "split_k": plan[0], "chunk_lts": plan[1], "k_blocks": plan[3],
                   "staging": {1: "whole", 2: "ring", 3: "single pass"}[plan[2]],
                   "plan": "auto" if not (args.split_k or args.variant or args.chunk_lts or args.k_blocks) else "forced",
                   "weights": f"w{args.bits}a4 IE-BME (16x64 tiles, 2x2 areas), int8 MFMA, int32 accumulate",
                   "rotating_copies": r["n_copies"]},
        "us_per_call": round(us, 3),
        "us_per_call_batches": {"batches": len(r["batches"]), "max_launches_per_batch": ROUND_LAUNCHES,
                                "median": round(float(np.median(r["batches"])), 3),
                                "min": round(min(r["batches"]), 3), "max": round(max(r["batches"]), 3)},
        "dense_equiv_tops": round(tops, 2),
        "encoded_mb": round(r["alg_bytes"] / 1e6, 3),
        "pmr": round(rep["pmr"], 4),
        "pmr_stored": round(rep["pmr_stored"], 4),
        "ci_eff_eq2": round(rep["ci_eff"], 3),
        "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4),
                     "traffic": (measured_traffic(w.name, N, args.reorder)
                                 if args.bits == 4 and not (args.split_k or args.variant or args.chunk_lts
                                                            or args.k_blocks) else None),
                     "kernel": "us_spmm_kernel",
                     "bytes_per_launch": r["alg_bytes"]},
        "cpu_baseline": cpu,
        **extras,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
