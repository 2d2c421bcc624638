"""Seeded synthetic inputs for the W4A4 sparse projections.

This module only draws random numbers. It holds none of the encoding or
product arithmetic, so both the HIP path and the CPU oracle can take their
inputs from here without sharing any of the method's code.

Recipe (every draw from numpy PCG64):
  * seed: ``SeedSequence([20261202 + config_id, variant])``, spawned into four
    independent streams: mask, weight values, activations, scales;
  * weight nonzeros: uniform over the 15 INT4 values {-8..-1, 1..7}, or for
    2-bit weights (W2A4) over the 3 values {-2, -1, 1};
  * mask: Bernoulli(keep = 1 - sparsity), i.i.d. per element; the row-skewed
    variant draws a keep rate per row from Beta(2, 3), rescales the rates to
    the requested mean and clips them to [0, 1];
  * activations: uniform over {-8..7};
  * per-output-channel scales: U(0.01, 0.1) in float32.

The weight shapes are those of LLaMA-2 7B/13B and 70B-class projections (the
paper's kernel corpus draws its shapes from such models; its exact shape list
and its pruned/quantised weights are not published, so these stand in).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

BASE_SEED = 20261202


@dataclass(frozen=True)
class Workload:
    """One weight matrix of a synthetic decode projection."""

    name: str
    config_id: int
    variant: int
    M: int
    K: int
    sparsity: float
    Ns: tuple
    dequant: bool = False
    row_skew: bool = False  # row keep-rate ~ Beta(2,3) rescaled to mean 1-sparsity
    note: str = field(default="", compare=False)


def _wl(name, cid, var, M, K, s, Ns, dequant=False, row_skew=False, note=""):
    return Workload(name, cid, var, M, K, s, tuple(Ns), dequant, row_skew, note)


#: The five workload families (variants of a family share its config id).
WORKLOADS = {
    w.name: w
    for w in [
        _wl("tiny_512x512_s50", 0, 0, 512, 512, 0.5, (8,), note="tiny SpMM"),
        _wl("qkv_12288x4096_s50", 1, 0, 12288, 4096, 0.5, (1, 8, 16, 32),
            note="LLaMA-2-7B fused QKV projection"),
        _wl("ffn_up_11008x4096_s30", 2, 0, 11008, 4096, 0.3, (8,), dequant=True),
        _wl("ffn_up_11008x4096_s50", 2, 1, 11008, 4096, 0.5, (8,), dequant=True),
        _wl("ffn_up_11008x4096_s70", 2, 2, 11008, 4096, 0.7, (8,), dequant=True),
        _wl("ffn_down_4096x11008_s30", 2, 3, 4096, 11008, 0.3, (8,), dequant=True),
        _wl("ffn_down_4096x11008_s50", 2, 4, 4096, 11008, 0.5, (8,), dequant=True,
            note="LLaMA-2-7B FFN down projection, 50% sparse"),
        _wl("ffn_down_4096x11008_s70", 2, 5, 4096, 11008, 0.7, (8,), dequant=True),
        _wl("ffn_13824x5120_skew60", 3, 0, 13824, 5120, 0.6, (4, 16), row_skew=True,
            note="LLaMA-2-13B FFN, row-skewed density"),
        _wl("ffn_28672x8192_s70", 4, 0, 28672, 8192, 0.7, (1, 32), dequant=True,
            note="70B-class FFN, whole matrix on one GPU"),
        _wl("ffn_28672x8192_s40", 4, 1, 28672, 8192, 0.4, (8,), dequant=True,
            note="the paper's 28672x8192 shape at 40% sparsity (its PMR example)"),
        _wl("prof_28672x7168_s50", 5, 0, 28672, 7168, 0.5, (8,),
            note="the paper's first profiling shape (m=28672, k=7168, batch 8)"),
        _wl("prof_12288x49152_s50", 5, 1, 12288, 49152, 0.5, (4,),
            note="the paper's second profiling shape (m=12288, k=49152, batch 4)"),
        _wl("kv_1024x4096_s50", 6, 0, 1024, 4096, 0.5, (8,),
            note="grouped-query key/value projection of an 8B model (8 KV heads of 128)"),
        _wl("kv_512x3584_s50", 6, 1, 512, 3584, 0.5, (8,),
            note="grouped-query key/value projection of a 7B model (4 KV heads of 128)"),
    ]
}

#: Activation columns drawn from the workload's own stream; narrower N take
#: the leading columns, wider N (prefill, up to N_LIMIT) append columns from
#: a second stream so that the first 32 never change.
N_DRAW = 32
N_LIMIT = 1024


def _streams(config_id: int, variant: int):
    ss = np.random.SeedSequence([BASE_SEED + config_id, variant])
    mask_ss, val_ss, x_ss, sc_ss = ss.spawn(4)
    return (np.random.Generator(np.random.PCG64(mask_ss)),
            np.random.Generator(np.random.PCG64(val_ss)),
            np.random.Generator(np.random.PCG64(x_ss)),
            np.random.Generator(np.random.PCG64(sc_ss)))


def nonzero_int4(rng: np.random.Generator, shape) -> np.ndarray:
    """Uniform draw over {-8..-1, 1..7} as int8."""
    u = rng.integers(0, 15, size=shape, dtype=np.int8)
    return np.where(u < 8, u - 8, u - 7).astype(np.int8)


def nonzero_int2(rng: np.random.Generator, shape) -> np.ndarray:
    """Uniform draw over {-2, -1, 1} as int8."""
    u = rng.integers(0, 3, size=shape, dtype=np.int8)
    return np.where(u < 2, u - 2, 1).astype(np.int8)


def _nonzero(rng, shape, bits):
    if bits == 4:
        return nonzero_int4(rng, shape)
    if bits == 2:
        return nonzero_int2(rng, shape)
    raise ValueError(f"weights are 4 or 2 bits, not {bits}")


def keep_mask(rng: np.random.Generator, M: int, K: int, sparsity: float,
              row_skew: bool = False, chunk_rows: int = 2048) -> np.ndarray:
    """Boolean keep mask, drawn in row chunks to bound peak memory."""
    keep = 1.0 - float(sparsity)
    if row_skew:
        p = rng.beta(2.0, 3.0, size=M)
        p = np.clip(p * (keep / p.mean()), 0.0, 1.0).astype(np.float32)
    else:
        p = np.full(M, keep, dtype=np.float32)
    out = np.empty((M, K), dtype=bool)
    for r0 in range(0, M, chunk_rows):
        r1 = min(M, r0 + chunk_rows)
        out[r0:r1] = rng.random((r1 - r0, K), dtype=np.float32) < p[r0:r1, None]
    return out


def weights(w: Workload, bits: int = 4) -> np.ndarray:
    """Masked INT4 (or 2-bit) weight matrix, int8 (M, K); zero means pruned."""
    mrng, vrng, _, _ = _streams(w.config_id, w.variant)
    mask = keep_mask(mrng, w.M, w.K, w.sparsity, w.row_skew)
    vals = _nonzero(vrng, (w.M, w.K), bits)
    vals[~mask] = 0
    return vals


def activations(w: Workload, N: int) -> np.ndarray:
    """INT4 activations as int8 of shape (N, K): row n is activation column n."""
    if not 1 <= N <= N_LIMIT:
        raise ValueError(f"N={N} outside [1, {N_LIMIT}]")
    _, _, xrng, _ = _streams(w.config_id, w.variant)
    xt = xrng.integers(-8, 8, size=(N_DRAW, w.K), dtype=np.int8)
    if N <= N_DRAW:
        return np.ascontiguousarray(xt[:N])
    more = np.random.Generator(np.random.PCG64(np.random.SeedSequence([BASE_SEED + w.config_id, w.variant, 1])))
    extra = more.integers(-8, 8, size=(N - N_DRAW, w.K), dtype=np.int8)
    return np.ascontiguousarray(np.concatenate([xt, extra]))


def scales(w: Workload) -> np.ndarray:
    """Per-output-channel float32 scales ~ U(0.01, 0.1)."""
    _, _, _, srng = _streams(w.config_id, w.variant)
    return srng.uniform(0.01, 0.1, size=w.M).astype(np.float32)


def random_problem(M: int, K: int, N: int, sparsity: float, seed: int,
                   row_skew: bool = False, bits: int = 4):
    """Small seeded problem (W (M,K), Xt (N,K), scales (M,)) for parity tests."""
    ss = np.random.SeedSequence([BASE_SEED, 1000 + seed])
    mrng, vrng, xrng, srng = (np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(4))
    mask = keep_mask(mrng, M, K, sparsity, row_skew)
    W = _nonzero(vrng, (M, K), bits)
    W[~mask] = 0
    Xt = xrng.integers(-8, 8, size=(N, K), dtype=np.int8)
    sc = srng.uniform(0.01, 0.1, size=M).astype(np.float32)
    return W, Xt, sc
