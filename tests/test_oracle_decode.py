"""Pins of decoding, commitment and the risk signals (Eq. 2; Sec. 4.2; Sec.
5.1: confidence ranking at temperature 0)."""

import math

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

from oracle import decode, stats


def test_argmax_conf_against_torch_softmax():
    rng = np.random.default_rng(0)
    V, mask = 50, 49
    lg = rng.standard_normal((6, V)) * 3
    lg[2, mask] = 100.0                    # [MASK] never wins
    am, cf = decode.argmax_conf(lg, mask)
    t = torch.from_numpy(np.delete(lg, mask, axis=1))
    p = torch.softmax(t, dim=1)
    assert np.array_equal(am, torch.argmax(p, dim=1).numpy())
    np.testing.assert_allclose(cf, p.max(dim=1).values.numpy(), rtol=1e-13)
    assert am[2] != mask


def test_argmax_ties_lowest_id():
    lg = np.zeros((2, 8))
    lg[0, [3, 5]] = 2.0
    lg[1, [0, 7]] = 1.0                    # 7 is the mask id: excluded
    am, cf = decode.argmax_conf(lg, 7)
    assert am.tolist() == [3, 0]
    assert cf[0] == pytest.approx(math.e ** 2 / (2 * math.e ** 2 + 5))


def _check_selection(conf, masked, k, sel):
    """Properties that determine the commitment set uniquely."""
    M = [i for i in range(len(masked)) if masked[i]]
    assert len(sel) == min(k, len(M))
    assert set(sel) <= set(M)
    key = [decode.rank_key(float(c)) for c in conf]
    rest = [i for i in M if i not in sel]
    for i in sel:
        for j in rest:
            assert key[i] > key[j] or (key[i] == key[j] and i < j)


@settings(max_examples=300, deadline=None)
@given(data=st.data(), L=st.integers(0, 40), k=st.integers(1, 8))
def test_select_properties(data, L, k):
    vals = st.sampled_from([0.1, 0.5, 0.5, 0.9, -math.inf, math.nan, 1.0])
    conf = data.draw(st.lists(vals, min_size=L, max_size=L))
    masked = data.draw(st.lists(st.integers(0, 1), min_size=L, max_size=L))
    sel = decode.select(conf, masked, k)
    _check_selection(conf, masked, k, sel)


def test_select_brute_force_small():
    # enumerate every k-subset: the chosen one maximises the sorted key
    # vector, then prefers lower positions
    import itertools
    rng = np.random.default_rng(1)
    for _ in range(200):
        L = int(rng.integers(1, 8))
        conf = rng.choice([0.2, 0.4, 0.4, 0.7, math.nan], size=L)
        masked = rng.integers(0, 2, size=L)
        k = int(rng.integers(1, 4))
        M = [i for i in range(L) if masked[i]]
        kk = min(k, len(M))
        best = None
        for sub in itertools.combinations(M, kk):
            keys = sorted(((-decode.rank_key(conf[i]), i) for i in sub))
            if best is None or keys < best[0]:
                best = (keys, sorted(sub))
        exp = best[1] if best else []
        assert decode.select(conf, masked, k) == exp


def test_commit_is_eq2():
    ids = np.array([9, 4, 9, 9], np.int32)
    m = np.array([1, 0, 1, 1], np.uint8)
    am = np.array([1, 2, 3, 5], np.int32)
    ids2, m2 = decode.commit(ids, m, am, [2])
    assert ids2.tolist() == [9, 4, 3, 9]       # committed one; others kept
    assert m2.tolist() == [1, 0, 0, 1]


def test_stats_hand_traces():
    masked = [1, 0, 1, 1]
    assert stats.mean_conf([0.5, 0.9, 0.5, 0.5], masked) == 0.5
    assert stats.mean_conf([0.1, 0.9, 0.2, 0.3], masked) == \
        pytest.approx(0.2)
    assert stats.churn([1, 2, 3, 4], [1, 9, 3, 4], masked, False) == 0.0
    assert stats.churn([1, 2, 3, 4], [0, 2, 0, 0], masked, False) == 1.0
    assert stats.churn([1, 2, 3, 4], [0, 2, 3, 0], masked, False) == 2 / 3
    assert stats.churn([1, 2, 3, 4], None, masked, True) == 0.0   # chi_1 = 0
    assert stats.mean_conf([0.3], [0]) == 0.0 and \
        stats.churn([1], [2], [0], False) == 0.0
