"""Pins of the oracle's pruning and merging realizers (Sec. 4.3, "Compatible
evidence realizers").

The paper fixes only what every realizer must give: an ordered hierarchy
whose finest level is v, with coarser levels for less cost.  The criteria are
readings (token L1 saliency; single-linkage merging on the crop's grid graph
by cosine similarity), pinned here by hand-derived answers, brute force over
all subsets, scipy's single-linkage clustering and minimum spanning tree,
scikit-learn's cosine similarity, and the partition / nesting invariants.
"""

import itertools

import numpy as np
import pytest
from scipy.cluster.hierarchy import fcluster, linkage
from scipy.sparse import csr_matrix
from scipy.sparse.csgraph import connected_components, minimum_spanning_tree
from sklearn.metrics.pairwise import cosine_similarity

from oracle import realizers as R
from oracle import views


def _partition(offs, mem):
    return {frozenset(int(m) for m in mem[offs[j]:offs[j + 1]])
            for j in range(len(offs) - 1)}


# ------------------------------------------------------------------ sizes --

@pytest.mark.parametrize("G,K", [(1, 2), (2, 3), (5, 3), (7, 4), (27, 3)])
def test_level_counts_match_the_pooling_pyramid(G, K):
    for lv in range(K):
        assert R.level_counts(G, K)[lv] == views.level_size(1, G, K, lv)


# ------------------------------------------------------------------ prune --

def test_prune_hand_example():
    # 2x2 crop, K = 2: level 0 keeps ceil(2/2)^2 = 1 token.  L1 norms by
    # hand: 1+1+2 = 4, 3+4 = 7, 7 (tie with token 1), 2.  The tie goes to the
    # lower index, so token 1 is kept.
    v = np.zeros((4, 8), np.float32)
    v[0, :3] = [1, -1, 2]
    v[1, :2] = [3, -4]
    v[2, :1] = [-7]
    v[3, 5] = 2
    keys = R.prune_keys(v, 1, 2)
    assert list(keys) == [4.0, 7.0, 7.0, 2.0]
    levels, maps = R.build_views(v, 1, 2, 2, R.PRUNE)
    assert list(maps[0][0]) == [0, 1] and list(maps[0][1]) == [1]
    assert np.array_equal(levels[0], v[1:2])
    assert list(maps[1][1]) == [0, 1, 2, 3]
    assert levels[1] is v


def test_prune_keeps_the_best_subset_brute_force():
    rng = np.random.default_rng(3)
    C, G, K = 2, 3, 3
    v = rng.standard_normal((C * G * G, 16)).astype(np.float32)
    keys = R.prune_keys(v, C, G)
    maps = R.prune_index_maps(keys, C, G, K)
    for lv, n in enumerate(R.level_counts(G, K)):
        mem = maps[lv][1]
        for c in range(C):
            kept = {int(m) - c * 9 for m in mem if c * 9 <= m < (c + 1) * 9}
            best = max(itertools.combinations(range(9), n),
                       key=lambda s: sum(keys[c * 9 + i] for i in s))
            assert kept == set(best)


def test_prune_sets_are_nested_ordered_and_copied():
    rng = np.random.default_rng(4)
    C, G, K = 3, 7, 4
    v = rng.standard_normal((C * G * G, 24)).astype(np.float32)
    levels, maps = R.build_views(v, C, G, K, R.PRUNE)
    prev = None
    for lv in range(K):
        offs, mem = maps[lv]
        assert list(offs) == list(range(len(mem) + 1))
        assert len(mem) == C * R.level_counts(G, K)[lv]
        assert list(mem) == sorted(mem)             # original order
        if prev is not None:
            assert set(prev) <= set(mem)            # nested
        prev = mem
        if lv < K - 1:
            assert np.array_equal(levels[lv], v[mem])


def test_prune_ties_nan_and_signed_zero():
    # all keys equal: the first n tokens in order; NaN ranks last; -0 == +0
    keys = np.array([0.0, -0.0, np.nan, 0.0, 1.0, 0.0, 0.0, -0.0, 0.0])
    maps = R.prune_index_maps(keys, 1, 3, 2)
    assert list(maps[0][1]) == [0, 1, 3, 4]
    keys2 = np.array([np.nan, -np.inf, 0.0, np.nan])
    maps2 = R.prune_index_maps(keys2, 1, 2, 2)
    assert list(maps2[0][1]) == [2]
    # NaN and -inf tie: lower index first
    assert R._ranked(list(keys2)) == [2, 0, 1, 3]


# ------------------------------------------------------------------ merge --

def test_edge_numbering():
    assert R.grid_edges(2) == [(0, 1), (2, 3), (0, 2), (1, 3)]
    e = R.grid_edges(5)
    assert len(e) == 2 * 5 * 4 and len(set(e)) == len(e)
    assert all(b - a in (1, 5) for a, b in e)


def test_cosine_special_cases():
    a = np.array([1.0, 2.0, -2.0])
    assert R.cosine(a, a) == pytest.approx(1.0, abs=1e-15)
    assert R.cosine(a, 3.5 * a) == pytest.approx(1.0, abs=1e-15)
    assert R.cosine(a, -a) == pytest.approx(-1.0, abs=1e-15)
    assert R.cosine(a, np.array([2.0, -1.0, 0.0])) == 0.0
    assert R.cosine(a, np.zeros(3)) == 0.0


def test_merge_keys_match_sklearn():
    rng = np.random.default_rng(5)
    C, G = 2, 4
    v = rng.standard_normal((C * G * G, 32)).astype(np.float32)
    keys = R.merge_keys(v, C, G)
    S = cosine_similarity(v.astype(np.float64))
    ref = [S[c * 16 + a, c * 16 + b] for c in range(C)
           for a, b in R.grid_edges(G)]
    np.testing.assert_allclose(keys, ref, rtol=0, atol=1e-13)


def test_merge_hand_example():
    # 3x3 crop with four unit vectors
    #     a a b
    #     a a b
    #     c c d
    # similarity 1 inside a colour, 0 across.  Level 1 (4 groups) = the four
    # colours; level 0 (1 group) = everything.
    e = np.eye(8, dtype=np.float32)
    a, b, c, d = e[0], e[1], e[2], e[3]
    v = np.stack([a, a, b, a, a, b, c, c, d])
    keys = R.merge_keys(v, 1, 3)
    assert sorted(set(keys.tolist())) == [0.0, 1.0]
    levels, maps = R.build_views(v, 1, 3, 3, R.MERGE)
    assert list(maps[1][0]) == [0, 4, 6, 8, 9]
    assert list(maps[1][1]) == [0, 1, 3, 4, 2, 5, 6, 7, 8]
    assert np.array_equal(levels[1], np.stack([a, b, c, d]))
    assert list(maps[0][0]) == [0, 9]
    np.testing.assert_array_equal(levels[0], v.astype(np.float64).mean(0)
                                  .astype(np.float32)[None])


@pytest.mark.parametrize("G,K,seed", [(5, 3, 0), (6, 4, 1), (4, 2, 2)])
def test_merge_matches_scipy_single_linkage(G, K, seed):
    rng = np.random.default_rng(seed)
    v = rng.standard_normal((G * G, 12))
    keys = R.merge_keys(v, 1, G)
    # distance 1 - cos on grid edges, a larger constant elsewhere: single
    # linkage then merges along grid edges in decreasing similarity
    N = G * G
    D = np.full((N, N), 10.0)
    for k, (a, b) in zip(keys, R.grid_edges(G)):
        D[a, b] = D[b, a] = 1.0 - k
    np.fill_diagonal(D, 0.0)
    iu = np.triu_indices(N, 1)
    Z = linkage(D[iu], method="single")
    maps = R.merge_index_maps(keys, 1, G, K)
    for lv in range(K - 1):
        n = R.level_counts(G, K)[lv]
        lab = fcluster(Z, t=n, criterion="maxclust")
        ref = {frozenset(np.nonzero(lab == x)[0].tolist()) for x in set(lab)}
        assert _partition(*maps[lv]) == ref


def test_merge_levels_are_components_of_the_maximum_spanning_tree():
    # single linkage = the heaviest N - n_l edges of the maximum spanning tree;
    # the tree comes from scipy (minimum tree of 2 - similarity) and the
    # components from scipy's connected_components
    rng = np.random.default_rng(7)
    G, K = 6, 4
    N = G * G
    v = rng.standard_normal((N, 10))
    keys = R.merge_keys(v, 1, G)
    edges = R.grid_edges(G)
    rows = [a for a, _ in edges]
    cols = [b for _, b in edges]
    W = csr_matrix((2.0 - keys, (rows, cols)), shape=(N, N))
    mst = minimum_spanning_tree(W).tocoo()
    assert mst.nnz == N - 1
    order = np.argsort(mst.data, kind="stable")        # heaviest similarity first
    maps = R.merge_index_maps(keys, 1, G, K)
    for lv in range(K - 1):
        take = order[:N - R.level_counts(G, K)[lv]]
        F = csr_matrix((np.ones(len(take)), (mst.row[take], mst.col[take])),
                       shape=(N, N))
        nc, lab = connected_components(F, directed=False)
        ref = {frozenset(np.nonzero(lab == x)[0].tolist()) for x in range(nc)}
        assert _partition(*maps[lv]) == ref


def _connected(group, G):
    group = set(group)
    start = next(iter(group))
    seen, todo = {start}, [start]
    while todo:
        x = todo.pop()
        r, s = divmod(x, G)
        for y in ((r - 1) * G + s if r else None, (r + 1) * G + s if r + 1 < G
                  else None, x - 1 if s else None, x + 1 if s + 1 < G else None):
            if y is not None and y in group and y not in seen:
                seen.add(y)
                todo.append(y)
    return seen == group


def test_merge_levels_are_nested_connected_partitions():
    rng = np.random.default_rng(8)
    C, G, K = 2, 7, 4
    v = rng.standard_normal((C * G * G, 16)).astype(np.float32)
    levels, maps = R.build_views(v, C, G, K, R.MERGE)
    N = G * G
    finer = None
    for lv in range(K - 1, -1, -1):
        offs, mem = maps[lv]
        part = _partition(offs, mem)
        assert len(part) == C * R.level_counts(G, K)[lv]
        assert sorted(mem) == list(range(C * N))            # a partition
        firsts = [int(mem[offs[j]]) for j in range(len(offs) - 1)]
        assert firsts == sorted(firsts)                     # by smallest member
        for j in range(len(offs) - 1):
            grp = [int(m) for m in mem[offs[j]:offs[j + 1]]]
            assert grp == sorted(grp)
            assert len({m // N for m in grp}) == 1          # inside one crop
            assert _connected([m % N for m in grp], G)
        if finer is not None:                               # whole groups
            assert all(any(f <= g for g in part) for f in finer)
        finer = part


def test_level_values_are_brute_force_means():
    rng = np.random.default_rng(9)
    C, G, K = 2, 5, 3
    v = rng.standard_normal((C * G * G, 16)).astype(np.float32)
    for rz in (R.PRUNE, R.MERGE):
        levels, maps = R.build_views(v, C, G, K, rz)
        for lv in range(K - 1):
            offs, mem = maps[lv]
            for j in range(len(offs) - 1):
                rows = v[mem[offs[j]:offs[j + 1]]].astype(np.float64)
                np.testing.assert_array_equal(
                    levels[lv][j], rows.mean(0).astype(np.float32))


def test_decisions_follow_given_keys():
    # replacing the keys changes only the decisions: reversed saliency keeps
    # the lowest-norm tokens
    rng = np.random.default_rng(10)
    v = rng.standard_normal((16, 8)).astype(np.float32)
    keys = R.prune_keys(v, 1, 4)
    _, maps = R.build_views(v, 1, 4, 2, R.PRUNE, keys_=-keys)
    assert set(maps[0][1]) == set(np.argsort(keys, kind="stable")[:4])


def test_merge_equal_similarities_in_edge_order():
    # identical tokens: every edge has similarity 1, so edges are taken in
    # index order: horizontal (0,1), (1,2), (3,4), (4,5), (6,7) give the 4
    # groups of level 0 for a 3x3 crop with K = 2
    v = np.ones((9, 8), np.float32)
    keys = R.merge_keys(v, 1, 3)
    assert np.all(keys == 1.0)
    maps = R.merge_index_maps(keys, 1, 3, 2)
    assert list(maps[0][0]) == [0, 3, 6, 8, 9]
    assert list(maps[0][1]) == [0, 1, 2, 3, 4, 5, 6, 7, 8]
    # a lower key on edge (6,7) defers it: (7,8) joins instead
    keys2 = keys.copy()
    keys2[4] = 0.5
    maps2 = R.merge_index_maps(keys2, 1, 3, 2)
    assert list(maps2[0][0]) == [0, 3, 6, 7, 9]
    assert list(maps2[0][1]) == [0, 1, 2, 3, 4, 5, 6, 7, 8]
