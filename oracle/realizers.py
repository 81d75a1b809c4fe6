"""Pruning and merging evidence realizers (Sec. 4.3, "Compatible evidence
realizers"; Sec. 5.3 and its realizer table).  TEST INFRASTRUCTURE ONLY.

The paper says that any construction with an ordered evidence-cost hierarchy
can serve as the realizer: pruning varies how many tokens are retained,
merging varies how strongly tokens are aggregated, and the allocation policy
is unchanged.  It fixes neither criterion.  Readings used here:

Level sizes.  Both realizers keep the token count of the pooling pyramid at
every level, per crop n_l = ceil(G / 2^(K-1-l))^2, so a level costs the same
under all three realizers; level K-1 is v itself (identity map).

Order of keys.  Larger key first; equal keys by lower index; NaN counts as
-inf and -0 as +0.

Prune (nested visual-token pruning).  The saliency of a token is its L1 norm,
the float64 sum of |v_ij| over its features.  Per crop, level l keeps the n_l
tokens of highest saliency, listed in their original order, each a
one-member window (the token unchanged).  Every level ranks by the same key,
so the retained sets are nested.

Merge (hierarchical similarity merging).  Per crop, the tokens are the nodes
of the 4-neighbour grid graph; an edge weighs the cosine similarity of its
two tokens (float64, dot / sqrt(|a|^2 |b|^2); 0 when either norm is 0).
Edges are visited in key order and each edge that joins two different groups
merges them (single linkage, i.e. Kruskal's order), until n_l groups remain
for level l, taken from l = K-2 down to 0; coarser levels therefore merge
whole groups of finer ones.  Groups are listed by their smallest member,
members ascending; a level token is the mean of its members (float64 sum in
member order, rounded once to the view dtype).  Edge numbering per crop:
horizontal edges (r, s)-(r, s+1) first, index r*(G-1) + s, then vertical
edges (r, s)-(r+1, s), index G*(G-1) + r*G + s.

Index maps use the pooling realizer's CSR form: token j of level l is the
mean of rows ``members[offsets[j]:offsets[j+1]]`` of v (global row ids
c*G*G + r*G + s), crops concatenated in order.
"""

import math

import numpy as np

from .views import _round_f64_to_bf16

POOL, PRUNE, MERGE = 0, 1, 2


def level_counts(grid: int, K: int):
    """Tokens per crop of each level: the pooling pyramid's counts."""
    return [(-(-grid // (1 << (K - 1 - lv)))) ** 2 for lv in range(K)]


def _key(x: float) -> float:
    x = float(x)
    if math.isnan(x):
        return -math.inf
    return x + 0.0          # -0.0 -> +0.0


def _ranked(keys):
    """Indices of ``keys`` in key order (larger first, ties by index)."""
    return sorted(range(len(keys)), key=lambda i: (-_key(keys[i]), i))


# ------------------------------------------------------------------- prune --

def prune_keys(v: np.ndarray, n_crops: int, grid: int) -> np.ndarray:
    """Saliency of every token of v: the float64 L1 norm of its row."""
    if v.shape[0] != n_crops * grid * grid:
        raise ValueError("v rows != n_crops * grid * grid")
    return np.sum(np.abs(np.asarray(v, dtype=np.float64)), axis=1)


def prune_index_maps(keys, n_crops: int, grid: int, K: int):
    """CSR maps of all K levels from the per-token saliency keys."""
    N = grid * grid
    counts = level_counts(grid, K)
    maps = []
    for lv in range(K):
        members = []
        for c in range(n_crops):
            order = _ranked(list(keys[c * N:(c + 1) * N]))
            kept = sorted(order[:counts[lv]])
            members.extend(c * N + i for i in kept)
        offsets = list(range(len(members) + 1))
        maps.append((np.asarray(offsets, np.int32),
                     np.asarray(members, np.int32)))
    return maps


# ------------------------------------------------------------------- merge --

def grid_edges(grid: int):
    """(a, b) token pairs of one crop's edges, in edge-index order."""
    out = []
    for r in range(grid):
        for s in range(grid - 1):
            out.append((r * grid + s, r * grid + s + 1))
    for r in range(grid - 1):
        for s in range(grid):
            out.append((r * grid + s, (r + 1) * grid + s))
    return out


def cosine(a: np.ndarray, b: np.ndarray) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    dot = float(np.dot(a, b))
    na = float(np.dot(a, a))
    nb = float(np.dot(b, b))
    if na == 0.0 or nb == 0.0:
        return 0.0
    return dot / math.sqrt(na * nb)


def merge_keys(v: np.ndarray, n_crops: int, grid: int) -> np.ndarray:
    """Cosine similarity of every grid edge, crop by crop."""
    if v.shape[0] != n_crops * grid * grid:
        raise ValueError("v rows != n_crops * grid * grid")
    N = grid * grid
    out = []
    for c in range(n_crops):
        for a, b in grid_edges(grid):
            out.append(cosine(v[c * N + a], v[c * N + b]))
    return np.asarray(out, dtype=np.float64)


def merge_partitions(keys, grid: int, K: int):
    """Group label (smallest member) of every token of one crop at each
    level l < K-1, by single-linkage merging in key order."""
    N = grid * grid
    edges = grid_edges(grid)
    parent = list(range(N))

    def find(x):
        while parent[x] != x:
            x = parent[x]
        return x

    counts = level_counts(grid, K)
    labels = [None] * K
    groups = N
    order = _ranked(list(keys))
    pos = 0
    for lv in range(K - 2, -1, -1):
        while groups > counts[lv]:
            a, b = edges[order[pos]]
            pos += 1
            ra, rb = find(a), find(b)
            if ra != rb:
                parent[max(ra, rb)] = min(ra, rb)
                groups -= 1
        labels[lv] = [find(i) for i in range(N)]
    labels[K - 1] = list(range(N))
    return labels


def merge_index_maps(keys, n_crops: int, grid: int, K: int):
    """CSR maps of all K levels from the per-edge similarity keys."""
    N = grid * grid
    E = 2 * grid * (grid - 1)
    per_crop = [merge_partitions(keys[c * E:(c + 1) * E], grid, K)
                for c in range(n_crops)]
    maps = []
    for lv in range(K):
        offsets, members = [0], []
        for c in range(n_crops):
            lab = per_crop[c][lv]
            for root in sorted(set(lab)):
                members.extend(c * N + i for i in range(N) if lab[i] == root)
                offsets.append(len(members))
        maps.append((np.asarray(offsets, np.int32),
                     np.asarray(members, np.int32)))
    return maps


# ----------------------------------------------------------------- levels --

def pool_by_map(v: np.ndarray, offsets, members, out_dtype: str = "f32"):
    """Token j = float64 sum of rows members[offsets[j]:offsets[j+1]] of v in
    that order, divided by the member count, rounded once to the dtype."""
    v64 = np.asarray(v, dtype=np.float64)
    n = len(offsets) - 1
    out = np.empty((n, v.shape[1]), dtype=np.float64)
    for t in range(n):
        acc = np.zeros(v.shape[1], dtype=np.float64)
        for m in members[offsets[t]:offsets[t + 1]]:
            acc = acc + v64[m]
        out[t] = acc / float(offsets[t + 1] - offsets[t])
    if out_dtype == "bf16":
        return _round_f64_to_bf16(out)
    if out_dtype == "f16":
        return out.astype(np.float16).astype(np.float32)
    return out.astype(np.float32)


def keys(v: np.ndarray, n_crops: int, grid: int, realizer: int):
    if realizer == PRUNE:
        return prune_keys(v, n_crops, grid)
    if realizer == MERGE:
        return merge_keys(v, n_crops, grid)
    raise ValueError("keys exist for the prune and merge realizers only")


def index_maps(keys_, n_crops: int, grid: int, K: int, realizer: int):
    if realizer == PRUNE:
        return prune_index_maps(keys_, n_crops, grid, K)
    if realizer == MERGE:
        return merge_index_maps(keys_, n_crops, grid, K)
    raise ValueError("maps from keys exist for the prune and merge realizers")


def build_views(v: np.ndarray, n_crops: int, grid: int, K: int,
                realizer: int, out_dtype: str = "f32", keys_=None):
    """All K levels (level K-1 is v itself) and their index maps.  ``keys_``
    replaces the keys computed from v (to test the decisions alone)."""
    if v.shape[0] != n_crops * grid * grid:
        raise ValueError("v rows != n_crops * grid * grid")
    k = keys(v, n_crops, grid, realizer) if keys_ is None else keys_
    maps = index_maps(k, n_crops, grid, K, realizer)
    levels = [pool_by_map(v, o, m, out_dtype) for o, m in maps[:-1]]
    levels.append(v)
    return levels, maps
