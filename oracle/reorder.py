"""Oracle for bitmap-aware row reordering (TEST INFRASTRUCTURE ONLY).

Plain restatement of Section V-B ("Bitmap-Aware Row Reordering"): the grouped
activity of a row group (Eq. 3), its grouped cost (Eq. 4), the grouped subset
dynamic programme (Eq. 5 and the algorithm "Bitmap-Aware Row Reordering via
Grouped Subset DP"), and the canonical permutation built partition-wise from
the optimal groups. The reordered tiles are then IE-BME-encoded by
``oracle.iebme.encode`` exactly like any other matrix. Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
this package. It shares no code with the native encoder or the HIP path.

The geometry is general here (any H_L, K_L, R_A, C_A that tile exactly), as
the section states the method for arbitrary R_A and C_A; the hot path uses
16 x 64 tiles with R_A = C_A = 2.

Readings taken where the section is silent:
  * ties in Eq. 5: for the smallest remaining row r, the candidate groups are
    the (R_A - 1)-subsets of the other remaining rows, enumerated in
    lexicographic order; a candidate replaces the current best only when it
    is strictly cheaper, so the first optimal candidate is kept, and the
    optimal groups are recovered by following these choices from the full
    row set;
  * pi[p] is the original LT row that becomes row p of the reordered LT
    (the concatenation pi = [r_{g,p} | p = 0..R_A-1, g = 0..H_L/R_A-1]), so
    reordered row p = R_A-partition a, row i of that partition, with
    p = a * H_L / R_A + i, holds the rows of group i across the partitions;
  * storage of pi: for H_L = 16, one 64-bit word per LT whose 4-bit field p
    (bits 4p .. 4p + 3) holds pi[p].
"""
from __future__ import annotations

import itertools

import numpy as np

from .iebme import Encoded, check_weights, encode, local_tiles


def tile_mask(T) -> np.ndarray:
    """M_t = I(W_t != 0), the binary nonzero mask of one LT."""
    return np.asarray(T) != 0


def grouped_activity(Mt: np.ndarray, rows, ca: int) -> np.ndarray:
    """Eq. 3: phi_t(r; j) = OR over a < R_A, c < C_A of M_t(r_a, j + c K_L / C_A).

    ``rows`` is the row group r = (r_0, ..., r_{R_A-1}); returns phi for every
    grouped column j < K_L / C_A.
    """
    kl = Mt.shape[1]
    kb = kl // ca
    phi = np.zeros(kb, dtype=bool)
    for r in rows:
        for c in range(ca):
            for j in range(kb):
                phi[j] = phi[j] or bool(Mt[r, j + c * kb])
    return phi


def grouped_cost(Mt: np.ndarray, rows, ca: int) -> int:
    """Eq. 4: c_t(r) = sum over j of phi_t(r; j), the union-mask entries the group activates."""
    return int(grouped_activity(Mt, rows, ca).sum())


def optimal_groups(Mt: np.ndarray, ra: int, ca: int):
    """Eq. 5 by memoised recursion over row subsets; returns (F(all rows), groups).

    F(S) = min over groups r of size R_A inside S that contain the smallest
    row of S of c_t(r) + F(S without r), with F(empty) = 0. The groups are
    returned in the order they are recovered from the full set.
    """
    H = Mt.shape[0]
    if H % ra:
        raise ValueError("H_L must be a multiple of R_A")
    # Grouped costs of every candidate group (first step of the algorithm).
    cost = {g: grouped_cost(Mt, g, ca) for g in itertools.combinations(range(H), ra)}
    F = {frozenset(): 0}
    choice = {}

    def solve(S: frozenset) -> int:
        if S in F:
            return F[S]
        r = min(S)
        others = sorted(S - {r})
        best, arg = None, None
        for rest in itertools.combinations(others, ra - 1):
            group = (r,) + rest
            v = cost[group] + solve(S - set(group))
            if best is None or v < best:
                best, arg = v, group
        F[S] = best
        choice[S] = arg
        return best

    full = frozenset(range(H))
    total = solve(full)
    groups, S = [], full
    while S:
        g = choice[S]
        groups.append(g)
        S = S - set(g)
    return total, groups


def canonical_permutation(groups, ra: int) -> list:
    """Sort rows inside each group, sort the groups, then concatenate partition-wise."""
    gs = sorted(tuple(sorted(g)) for g in groups)
    return [gs[g][p] for p in range(ra) for g in range(len(gs))]


def reorder_tile(T, ra: int = 2, ca: int = 2):
    """Row permutation pi*_t of one LT and its optimal union-mask size."""
    Mt = tile_mask(T)
    total, groups = optimal_groups(Mt, ra, ca)
    return canonical_permutation(groups, ra), total


def reorder(W, lt_h: int = 16, lt_w: int = 64, ra: int = 2, ca: int = 2):
    """Reorder the rows of every LT of W independently.

    Returns (W_reordered, perms, costs): perms[t] is pi*_t, costs[t] the
    optimal F of LT t. Row p of reordered LT t is row perms[t][p] of LT t.
    """
    W = check_weights(W)
    M, K = W.shape
    if M % lt_h or K % lt_w:
        raise ValueError("shape must tile exactly into LTs")
    T = local_tiles(W, lt_h, lt_w)
    perms = np.zeros((T.shape[0], lt_h), dtype=np.int64)
    costs = np.zeros(T.shape[0], dtype=np.int64)
    R = np.empty_like(T)
    for t in range(T.shape[0]):
        pi, total = reorder_tile(T[t], ra, ca)
        perms[t] = pi
        costs[t] = total
        R[t] = T[t][pi, :]
    nmb, nkb = M // lt_h, K // lt_w
    Wr = R.reshape(nmb, nkb, lt_h, lt_w).transpose(0, 2, 1, 3).reshape(M, K)
    return Wr, perms, costs


def undo_reorder(Wr, perms, lt_h: int = 16, lt_w: int = 64) -> np.ndarray:
    """Inverse of reorder: row perms[t][p] of LT t takes reordered row p."""
    Wr = np.asarray(Wr, dtype=np.int64)
    M, K = Wr.shape
    T = local_tiles(Wr, lt_h, lt_w)
    out = np.empty_like(T)
    for t in range(T.shape[0]):
        out[t][np.asarray(perms[t]), :] = T[t]
    nmb, nkb = M // lt_h, K // lt_w
    return out.reshape(nmb, nkb, lt_h, lt_w).transpose(0, 2, 1, 3).reshape(M, K)


def perm_words(perms) -> np.ndarray:
    """pi of each 16-row LT as one uint64: bits 4p .. 4p + 3 hold pi[p]."""
    perms = np.asarray(perms, dtype=np.uint64)
    if perms.ndim != 2 or perms.shape[1] != 16:
        raise ValueError("perm words hold 16-row permutations")
    shifts = (4 * np.arange(16)).astype(np.uint64)
    return np.bitwise_or.reduce(perms << shifts, axis=1).astype(np.uint64)


def encode_reordered(W, lt_h: int = 16, lt_w: int = 64, ra: int = 2, ca: int = 2, order: str = "areas"):
    """Row reordering (Section V-B) followed by IE-BME (Section V-A), with the
    values of each LT in ``order`` (see oracle.iebme).

    Returns (Encoded of the reordered matrix, perms).
    """
    Wr, perms, _ = reorder(W, lt_h, lt_w, ra, ca)
    enc: Encoded = encode(Wr, lt_h, lt_w, ra, ca, order=order)
    return enc, perms
