"""Pins of the oracle's evidence hierarchy (Sec. 4.3, v^(K) = v; Sec. 3.2).

Each pooled token is checked against a brute-force window mean computed by
slicing the 2-D grid, against torch's ceil-mode average pooling (a library
routine whose edge windows divide by their in-bounds count), and the index
maps against partition and size properties.
"""

from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import views


@pytest.mark.parametrize("C,G,sizes", [
    (1, 12, (9, 36, 144)),          # tiny config: 144 -> 36 -> 9
    (1, 27, (49, 196, 729)),        # one 27x27 crop
    (5, 27, (245, 980, 3645)),      # five crops
    (4, 27, (196, 784, 2916)),      # four crops
])
def test_level_sizes(C, G, sizes):
    assert tuple(views.level_size(C, G, 3, lv) for lv in range(3)) == sizes
    for lv in range(3):
        offs, mem = views.index_map(C, G, 3, lv)
        assert len(offs) == sizes[lv] + 1


@pytest.mark.parametrize("C,G,K", [(1, 12, 3), (2, 27, 3), (3, 5, 3),
                                   (1, 9, 4), (2, 1, 3), (1, 7, 1)])
def test_index_map_partitions(C, G, K):
    for lv in range(K):
        offs, mem = views.index_map(C, G, K, lv)
        assert offs[0] == 0 and offs[-1] == C * G * G
        assert np.all(np.diff(offs) >= 1)
        assert sorted(mem.tolist()) == list(range(C * G * G))
        f = views.level_window(K, lv)
        assert np.diff(offs).max() <= f * f
    offs, mem = views.index_map(C, G, K, K - 1)
    assert np.array_equal(mem, np.arange(C * G * G))
    assert np.array_equal(offs, np.arange(C * G * G + 1))


def _brute(v, C, G, f):
    d = v.shape[1]
    w = -(-G // f)
    grid = v.astype(np.float64).reshape(C, G, G, d)
    out = []
    for c in range(C):
        for i in range(w):
            for j in range(w):
                blk = grid[c, i * f:(i + 1) * f, j * f:(j + 1) * f]
                out.append(blk.reshape(-1, d).mean(axis=0))
    return np.asarray(out)


@pytest.mark.parametrize("C,G", [(1, 12), (2, 27), (1, 5)])
def test_pool_brute_force(C, G):
    rng = np.random.default_rng(7)
    v = rng.standard_normal((C * G * G, 16)).astype(np.float32)
    levels, maps = views.build_views(v, C, G, 3, "f32")
    assert levels[2] is v                      # v^(K) = v, no copy
    for lv, f in ((0, 4), (1, 2)):
        ref = _brute(v, C, G, f)
        np.testing.assert_allclose(levels[lv], ref, rtol=1e-6, atol=1e-7)
        # each token is the mean of the members its own map lists
        offs, mem = maps[lv]
        for t in range(len(offs) - 1):
            m = v[mem[offs[t]:offs[t + 1]]].astype(np.float64).mean(axis=0)
            np.testing.assert_allclose(levels[lv][t], m, rtol=1e-6,
                                       atol=1e-7)


@pytest.mark.parametrize("C,G", [(1, 12), (1, 27), (3, 27)])
def test_pool_matches_torch_ceil_avg_pool(C, G):
    rng = np.random.default_rng(11)
    d = 8
    v = rng.standard_normal((C * G * G, d)).astype(np.float32)
    levels, _ = views.build_views(v, C, G, 3, "f32")
    x = torch.from_numpy(v.astype(np.float64)).reshape(C, G, G, d) \
        .permute(0, 3, 1, 2)
    for lv, f in ((0, 4), (1, 2)):
        y = torch.nn.functional.avg_pool2d(x, f, f, ceil_mode=True)
        y = y.permute(0, 2, 3, 1).reshape(-1, d).numpy()
        np.testing.assert_allclose(levels[lv], y, rtol=1e-6, atol=1e-7)


def test_cascade_equals_direct_on_even_grid():
    # 12x12: two 2x2 poolings equal one 4x4 pooling (textbook special case)
    rng = np.random.default_rng(3)
    v = rng.standard_normal((144, 4)).astype(np.float32)
    l1 = views.pool_level(v, 1, 12, 3, 1)
    l0 = views.pool_level(v, 1, 12, 3, 0)
    l1_as_grid = l1.reshape(6, 6, 4)
    casc = views.pool_level(l1_as_grid.reshape(36, 4), 1, 6, 2, 0)
    np.testing.assert_allclose(l0, casc, rtol=1e-6)


def _nearest_bf16(x: float) -> float:
    """Nearest bfloat16 to x by exact rational comparison, ties to even."""
    f = np.float32(x)
    bits = int(np.array([f]).view(np.uint32)[0])
    lo_bits = bits & 0xFFFF0000
    cands = []
    for b in (lo_bits - 0x10000, lo_bits, lo_bits + 0x10000):
        val = np.array([b & 0xFFFFFFFF], dtype=np.uint32).view(np.float32)[0]
        cands.append((abs(Fraction(float(val)) - Fraction(x)),
                      (b >> 16) & 1, float(val)))
    cands.sort()
    return cands[0][2]


def test_bf16_single_rounding_from_double():
    rng = np.random.default_rng(5)
    xs = rng.standard_normal(2000) * np.exp(rng.uniform(-5, 5, 2000))
    # plant exact ties and values just off ties
    xs = np.concatenate([xs, [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8,
                              1.0 + 2 ** -8 + 2 ** -40, -(1.0 + 2 ** -8)]])
    got = views._round_f64_to_bf16(xs)
    exp = np.array([_nearest_bf16(float(x)) for x in xs], dtype=np.float32)
    np.testing.assert_array_equal(got, exp)


def _nearest_f16(x: float) -> float:
    """Nearest binary16 to x by exact rational comparison, ties to even."""
    h = np.float16(np.float32(x))       # a neighbour within one step
    bits = int(np.array([h]).view(np.uint16)[0])
    cands = []
    for b in (bits - 1, bits, bits + 1):
        if not 0 <= b <= 0xFFFF:
            continue
        val = np.array([b], dtype=np.uint16).view(np.float16)[0]
        if not np.isfinite(val):
            continue
        cands.append((abs(Fraction(float(val)) - Fraction(x)), b & 1,
                      float(val)))
    cands.sort()
    return cands[0][2]


def test_f16_single_rounding_from_double():
    """fp16 views: float64 means round once to binary16 (subnormals too)."""
    rng = np.random.default_rng(6)
    xs = rng.standard_normal(3000) * np.exp(rng.uniform(-14, 6, 3000))
    ties = [1.0 + 2 ** -11, 1.0 + 3 * 2 ** -11, 2.0 ** -20 + 2.0 ** -25,
            1.0 + 2 ** -11 + 2 ** -40, -(1.0 + 2 ** -11)]
    xs = np.concatenate([xs, ties])
    # one-token windows (grid 1, K = 1): each "mean" is the value itself
    got = views.pool_level(xs.reshape(-1, 1), len(xs), 1, 1, 0, "f16")[:, 0]
    exp = np.array([_nearest_f16(float(x)) for x in xs], dtype=np.float32)
    np.testing.assert_array_equal(got, exp)


@pytest.mark.parametrize("C,G,S", [(1, 27, 2), (2, 27, 3), (1, 12, 4),
                                   (3, 5, 2), (1, 1, 2), (2, 7, 5)])
def test_mixed_view(C, G, S):
    """Mixed view (Sec. 4.3): the coarse tokens of each crop, unchanged, then
    the raw lattice tokens bit-for-bit; the map lists exactly those members."""
    rng = np.random.default_rng(G * 10 + S)
    d = 8
    v = rng.standard_normal((C * G * G, d)).astype(np.float32)
    levels, maps = views.build_views(v, C, G, 3, "f32", mixed_stride=S)
    coarse = levels[0]
    n0 = (-(-G // 4)) ** 2
    lat = [(r, q) for r in range(S // 2, G, S) for q in range(S // 2, G, S)]
    # lattice from its definition with numpy index arithmetic
    rr, qq = np.meshgrid(np.arange(G), np.arange(G), indexing="ij")
    on = ((rr % S) == S // 2) & ((qq % S) == S // 2)
    assert sorted(zip(rr[on].tolist(), qq[on].tolist())) == lat
    mix = levels[1]
    assert mix.shape[0] == C * (n0 + len(lat))
    offs, mem = maps[1]
    assert offs[-1] == C * (G * G + len(lat)) == len(mem)
    per = n0 + len(lat)
    for c in range(C):
        blk = mix[c * per:(c + 1) * per]
        np.testing.assert_array_equal(blk[:n0], coarse[c * n0:(c + 1) * n0])
        raw = np.asarray([v[c * G * G + r * G + q] for r, q in lat],
                         np.float32).reshape(-1, d)
        np.testing.assert_array_equal(blk[n0:], raw)
        # pooled part of the map covers the crop once; singletons are the
        # lattice tokens in row-major order
        t0 = c * per
        pooled = mem[offs[t0]:offs[t0 + n0]]
        assert sorted(pooled.tolist()) == list(range(c * G * G,
                                                     (c + 1) * G * G))
        singles = [mem[offs[t0 + n0 + k]:offs[t0 + n0 + k + 1]].tolist()
                   for k in range(len(lat))]
        assert singles == [[c * G * G + r * G + q] for r, q in lat]


def test_mixed_view_needs_three_levels():
    v = np.zeros((16, 8), np.float32)
    with pytest.raises(ValueError):
        views.build_views(v, 1, 4, 4, "f32", mixed_stride=2)
    with pytest.raises(ValueError):
        views.build_views(v, 1, 4, 3, "f32", mixed_stride=1)
