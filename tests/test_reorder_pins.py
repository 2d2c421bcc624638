"""Pins that tie the row-reordering oracle (Section V-B) to things other than itself.

* The subset DP of Eq. 5 must reach the true minimum: for R_A = 2 that is a
  minimum-weight perfect matching on the rows, which networkx solves with an
  unrelated (blossom) algorithm; for small tiles every row partition is
  enumerated outright.
* Costs are scored by the IE-BME encoder's own union mask (Section V-A), not
  by Eq. 3/4, so a slip in the grouped activity (a dropped column partition,
  a wrong column offset) shows up as a mismatch.
* Planted tiles have a unique optimum known by construction, which fixes the
  canonical permutation to the last index.
* The tie reading (first optimal candidate in lexicographic order) is pinned
  on tiles where every grouping costs the same.
"""
import itertools

import networkx as nx
import numpy as np
import pytest

from oracle import iebme, reorder


def _random_tile(rng, h, w, keep):
    mask = rng.random((h, w)) < keep
    vals = rng.integers(1, 8, size=(h, w)) * rng.choice([-1, 1], size=(h, w))
    return np.where(mask, vals, 0).astype(np.int64)


def _encoded_union_size(T, ra, ca):
    """P_t of one tile as the IE-BME encoder builds it (Section V-A)."""
    h, w = T.shape
    return int(iebme.encode(T, lt_h=h, lt_w=w, ra=ra, ca=ca).P[0])


def _reordered(T, pi):
    return np.asarray(T)[np.asarray(pi), :]


@pytest.mark.parametrize("keep", [0.05, 0.15, 0.3, 0.5, 0.7])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_dp_matches_min_weight_perfect_matching(keep, seed):
    rng = np.random.default_rng(100 * seed + int(keep * 100))
    T = _random_tile(rng, 16, 64, keep)
    pi, total = reorder.reorder_tile(T, ra=2, ca=2)
    # Pair weight = union-mask entries the encoder activates for the two rows
    # alone (rows 0 and 8 of a 16 x 64 tile form union row 0).
    G = nx.Graph()
    for u, v in itertools.combinations(range(16), 2):
        pair = np.zeros((16, 64), dtype=np.int64)
        pair[0], pair[8] = T[u], T[v]
        G.add_edge(u, v, weight=_encoded_union_size(pair, 2, 2))
    matching = nx.min_weight_matching(G)
    assert len(matching) == 8
    best = sum(G[u][v]["weight"] for u, v in matching)
    assert total == best
    # The permutation realises that cost in the encoder, and never loses to the identity.
    assert _encoded_union_size(_reordered(T, pi), 2, 2) == best
    assert best <= _encoded_union_size(T, 2, 2)


def _all_partitions(h, ra):
    """Every split of range(h) into groups of ra rows, from all row orders."""
    seen = set()
    for order in itertools.permutations(range(h)):
        key = frozenset(frozenset(order[k:k + ra]) for k in range(0, h, ra))
        if key not in seen:
            seen.add(key)
            yield [sorted(g) for g in key]


@pytest.mark.parametrize("ra,ca,keep", [(2, 2, 0.2), (2, 2, 0.5), (2, 1, 0.3), (4, 2, 0.1), (4, 1, 0.25)])
def test_dp_matches_brute_force_small_tiles(ra, ca, keep):
    h, w = 8, 64
    rng = np.random.default_rng(ra * 10 + ca + int(keep * 1000))
    T = _random_tile(rng, h, w, keep)
    pi, total = reorder.reorder_tile(T, ra=ra, ca=ca)
    costs = []
    for groups in _all_partitions(h, ra):
        # Partition-wise layout: group g fills row g of every row partition.
        perm = [groups[g][a] for a in range(ra) for g in range(h // ra)]
        costs.append(_encoded_union_size(_reordered(T, perm), ra, ca))
    assert len(costs) == {2: 105, 4: 35}[ra]
    assert total == min(costs)
    assert _encoded_union_size(_reordered(T, pi), ra, ca) == total


@pytest.mark.parametrize("seed", range(4))
def test_planted_pairs_have_a_unique_canonical_permutation(seed):
    """Rows come in identical pairs over disjoint grouped columns.

    Pairing the two copies activates each pair's columns once; any other
    pairing activates some pair's columns twice. The optimum is therefore
    unique and its canonical form is known.
    """
    rng = np.random.default_rng(seed)
    rows = rng.permutation(16)
    pairs = [tuple(sorted(rows[2 * k:2 * k + 2])) for k in range(8)]
    cols = rng.permutation(32)
    T = np.zeros((16, 64), dtype=np.int64)
    for k, (u, v) in enumerate(pairs):
        for j in cols[4 * k:4 * k + 4]:
            c = int(rng.integers(2))
            T[u, j + 32 * c] = T[v, j + 32 * c] = int(rng.integers(1, 8))
    pi, total = reorder.reorder_tile(T, ra=2, ca=2)
    assert total == 32
    first = sorted(pairs)
    assert pi == [g[0] for g in first] + [g[1] for g in first]


def test_ties_take_the_first_candidate():
    # Every grouping of a fully dense (or empty) tile costs the same, so the
    # first candidate of each DP state wins: groups {0,1}, {2,3}, ...
    expected = list(range(0, 16, 2)) + list(range(1, 16, 2))
    for fill in (0, 3):
        T = np.full((16, 64), fill, dtype=np.int64)
        pi, total = reorder.reorder_tile(T, ra=2, ca=2)
        assert pi == expected
        assert total == (32 * 8 if fill else 0)


def test_single_row_groups_keep_the_identity():
    # R_A = 1 leaves nothing to group: every row is its own group and the
    # union-mask size is the per-row count of active grouped columns.
    rng = np.random.default_rng(5)
    T = _random_tile(rng, 16, 64, 0.3)
    pi, total = reorder.reorder_tile(T, ra=1, ca=2)
    assert pi == list(range(16))
    assert total == _encoded_union_size(T, 1, 2)


@pytest.mark.parametrize("M,K,keep", [(32, 128, 0.5), (48, 192, 0.3), (16, 64, 0.7)])
def test_reorder_round_trip_and_invariants(M, K, keep):
    rng = np.random.default_rng(M + K)
    W = _random_tile(rng, M, K, keep)
    Wr, perms, costs = reorder.reorder(W)
    n_lt = (M // 16) * (K // 64)
    assert perms.shape == (n_lt, 16)
    for pi in perms:
        assert sorted(pi) == list(range(16))
        assert pi[0] == 0                                  # smallest row leads the first group
        assert all(pi[g] < pi[8 + g] for g in range(8))    # rows sorted inside a group
        assert all(pi[g] < pi[g + 1] for g in range(7))    # groups sorted
    assert np.array_equal(reorder.undo_reorder(Wr, perms), W)
    assert np.count_nonzero(Wr) == np.count_nonzero(W)
    enc, perms2 = reorder.encode_reordered(W)
    assert np.array_equal(perms2, perms)
    assert np.array_equal(enc.P, costs)
    assert np.array_equal(reorder.undo_reorder(iebme.decode(enc), perms), W)
    assert enc.n_payload <= iebme.encode(W).n_payload


def test_perm_words_layout():
    pi = [0, 2, 4, 6, 8, 10, 12, 14, 1, 3, 5, 7, 9, 11, 13, 15]
    w = int(reorder.perm_words(np.array([pi]))[0])
    assert w == 0xFDB97531ECA86420
    assert [(w >> (4 * p)) & 0xF for p in range(16)] == pi


def test_reordering_shrinks_iid_tiles():
    # On i.i.d. 50 % masks the optimal pairing activates fewer union-mask
    # entries than the fixed pairing of rows i and i + 8 (mean 240 = 256(1 - s^4)).
    rng = np.random.default_rng(11)
    W = _random_tile(rng, 32, 256, 0.5)
    _, _, costs = reorder.reorder(W)
    plain = iebme.encode(W).P
    assert np.all(costs <= plain)
    assert costs.mean() < plain.mean() - 5
