"""Evidence hierarchy by pooling (Sec. 4.3, "Ordered evidence hierarchy").

The realizer builds K views ordered by granularity with the finest one equal
to the encoding itself (v^(K) = v; a budget of 1 leaves v unchanged, Sec. 3.2).
The coarser views use structured pooling.  Reading used here (the paper does
not fix the pooling arithmetic): per crop of a G x G grid, level l in
{0..K-1} pools non-overlapping windows of side f = 2^(K-1-l); windows at the
grid edge keep only their in-bounds members (ceil padding) and the value is
the plain mean over those members.  Crops are pooled independently and
concatenated crop-major.  Level K-1 (f = 1) is v with the identity map.

Index map of a level (CSR): ``offsets[n_l + 1]`` and ``members[C*G*G]``;
token j of the level is the mean of rows ``members[offsets[j]:offsets[j+1]]``
of v, listed row-major inside its window.  Member ids are global:
``c*G*G + r*G + s``.

Mixed view (Sec. 4.3: the middle view augments the pooled representation
with a fixed subset of unpooled tokens; K = 3).  The paper does not say which
tokens; reading used here: with a stride S >= 2, the raw tokens on the
lattice r = o, o+S, ... and s = o, o+S, ... of every crop, o = S // 2 (one
token per S x S cell, near its centre).  Per crop the mixed level lists the
coarse (level 0) tokens, then the lattice tokens row-major; each lattice
token is a one-member "window", i.e. the raw token itself.
"""

import numpy as np


def level_window(K: int, level: int) -> int:
    if not (0 <= level < K):
        raise ValueError("level out of range")
    return 1 << (K - 1 - level)


def level_size(n_crops: int, grid: int, K: int, level: int) -> int:
    f = level_window(K, level)
    w = -(-grid // f)
    return n_crops * w * w


def index_map(n_crops: int, grid: int, K: int, level: int):
    """CSR index map of one level, built by enumerating windows."""
    f = level_window(K, level)
    w = -(-grid // f)
    offsets = [0]
    members = []
    for c in range(n_crops):
        for i in range(w):
            for j in range(w):
                for r in range(i * f, min((i + 1) * f, grid)):
                    for s in range(j * f, min((j + 1) * f, grid)):
                        members.append(c * grid * grid + r * grid + s)
                offsets.append(len(members))
    return np.asarray(offsets, dtype=np.int32), np.asarray(members, np.int32)


def _round_f64_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (ties to even), in a single
    rounding step, returned as float32.  Valid for normal-range values."""
    b = np.ascontiguousarray(x, dtype=np.float64).view(np.uint64)
    # bf16 keeps 7 explicit mantissa bits of the 52 of a double: drop 45.
    lsb = (b >> np.uint64(45)) & np.uint64(1)
    b = (b + np.uint64((1 << 44) - 1) + lsb) & ~np.uint64((1 << 45) - 1)
    return b.view(np.float64).astype(np.float32)


def pool_level(v: np.ndarray, n_crops: int, grid: int, K: int, level: int,
               out_dtype: str = "f32") -> np.ndarray:
    """Level ``level`` of the hierarchy: each token is the float64 sum of its
    members (taken in index-map order) divided by the member count, rounded
    once to the output precision (fp32, bf16 or fp16, as the encoding)."""
    offs, mem = index_map(n_crops, grid, K, level)
    v64 = np.asarray(v, dtype=np.float64)
    n = len(offs) - 1
    out = np.empty((n, v.shape[1]), dtype=np.float64)
    for t in range(n):
        acc = np.zeros(v.shape[1], dtype=np.float64)
        for m in mem[offs[t]:offs[t + 1]]:
            acc = acc + v64[m]
        out[t] = acc / float(offs[t + 1] - offs[t])
    if out_dtype == "bf16":
        return _round_f64_to_bf16(out)
    if out_dtype == "f16":
        # numpy converts float64 to binary16 directly (one rounding, ties to
        # even, subnormals included)
        return out.astype(np.float16).astype(np.float32)
    return out.astype(np.float32)


def lattice(grid: int, stride: int):
    """Row and column indices of the mixed view's raw tokens in one crop."""
    if stride < 2:
        raise ValueError("mixed stride must be >= 2")
    return list(range(stride // 2, grid, stride))


def mixed_index_map(n_crops: int, grid: int, stride: int):
    """CSR map of the mixed level: per crop the coarse windows (side 4), then
    the lattice tokens as single members."""
    coarse_offs, coarse_mem = index_map(1, grid, 3, 0)
    lat = lattice(grid, stride)
    offsets = [0]
    members = []
    for c in range(n_crops):
        base = c * grid * grid
        for t in range(len(coarse_offs) - 1):
            for m in coarse_mem[coarse_offs[t]:coarse_offs[t + 1]]:
                members.append(base + int(m))
            offsets.append(len(members))
        for r in lat:
            for q in lat:
                members.append(base + r * grid + q)
                offsets.append(len(members))
    return np.asarray(offsets, dtype=np.int32), np.asarray(members, np.int32)


def mixed_level(v: np.ndarray, n_crops: int, grid: int, stride: int,
                out_dtype: str = "f32") -> np.ndarray:
    """Mixed level: every token is the float64 mean of its members rounded
    once (a single raw member is returned unchanged)."""
    offs, mem = mixed_index_map(n_crops, grid, stride)
    v64 = np.asarray(v, dtype=np.float64)
    out = np.empty((len(offs) - 1, v.shape[1]), dtype=np.float64)
    for t in range(len(offs) - 1):
        acc = np.zeros(v.shape[1], dtype=np.float64)
        for m in mem[offs[t]:offs[t + 1]]:
            acc = acc + v64[m]
        out[t] = acc / float(offs[t + 1] - offs[t])
    if out_dtype == "bf16":
        return _round_f64_to_bf16(out)
    if out_dtype == "f16":
        return out.astype(np.float16).astype(np.float32)
    return out.astype(np.float32)


def build_views(v: np.ndarray, n_crops: int, grid: int, K: int = 3,
                out_dtype: str = "f32", mixed_stride: int = 0):
    """All K levels (level K-1 is v itself) and their index maps; with
    ``mixed_stride`` (K = 3 only) the middle level is the mixed view."""
    if v.shape[0] != n_crops * grid * grid:
        raise ValueError("v rows != n_crops * grid * grid")
    if mixed_stride and K != 3:
        raise ValueError("the mixed view needs K = 3")
    levels, maps = [], []
    for lv in range(K):
        if mixed_stride and lv == 1:
            maps.append(mixed_index_map(n_crops, grid, mixed_stride))
            levels.append(mixed_level(v, n_crops, grid, mixed_stride,
                                      out_dtype))
            continue
        maps.append(index_map(n_crops, grid, K, lv))
        if lv == K - 1:
            levels.append(v)
        else:
            levels.append(pool_level(v, n_crops, grid, K, lv, out_dtype))
    return levels, maps
