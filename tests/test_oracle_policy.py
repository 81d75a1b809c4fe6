"""Pins of the oracle's allocation policy (Sec. 4.2, Eqs. 6-9; App. A).

Expected values here are derived by hand from the equations (closed forms
worked out in the comments) or printed in the paper (golden fixtures), never
produced by the oracle itself.
"""

import json
import math
import os

import pytest
from hypothesis import given, settings, strategies as st

from oracle import policy

LLADA = dict(T=16, early=True, B=0.75, rho=0.20, alpha=1.0)
LAVIDA = dict(T=32, early=False, B=0.45, rho=0.20, alpha=0.5)


def levels_at_constant_risk(cfg, demand, r):
    lo, up = policy.envelope(cfg["T"], cfg["early"], cfg["B"], cfg["rho"],
                             demand)
    return [policy.quantize(policy.allocate(lo[t], up[t], r))
            for t in range(cfg["T"])]


def test_phase_profile_closed_form():
    # early: p_t = 1 - (t - 1/2)/T = (2T - 2t + 1)/(2T); late: (2t - 1)/(2T)
    p = policy.phase_profile(16, True)
    assert p == [(33 - 2 * t) / 32 for t in range(1, 17)]
    q = policy.phase_profile(32, False)
    assert q == [(2 * t - 1) / 64 for t in range(1, 33)]
    # symmetric, no zero endpoints (Sec. 4.2)
    assert min(p) > 0 and min(q) > 0
    # the two orientations mirror each other
    assert policy.phase_profile(16, False)[::-1] == p


def test_llada_upper_is_dyadic_closed_form():
    # d = 1: beta = (1 - .2 + .2) * .75 = .75, T*beta = 12.  With s = 2 the
    # entries t <= 8 exceed 1 and clip; the rest sum to (15+13+...+1)/32 = 2,
    # so s = (12 - 8)/2 = 2 and upper_t = min(1, (33 - 2t)/16) exactly.
    _, up = policy.envelope(16, True, 0.75, 0.20, 1.0)
    assert up == [min(1.0, (33 - 2 * t) / 16) for t in range(1, 17)]


def test_llada_lower_closed_form():
    # beta = .6, T*beta = 9.6.  Clipping 3 entries leaves t = 4..16 with
    # sum (25+23+...+1)/32 = 169/32 = 5.28125, s = 6.6/5.28125 and
    # s * p_4 = .976 <= 1; clipping only 2 would need s*p_3 = 1.047 > 1.
    lo, _ = policy.envelope(16, True, 0.75, 0.20, 1.0)
    s = 6.6 / 5.28125
    exp = [1.0] * 3 + [s * (33 - 2 * t) / 32 for t in range(4, 17)]
    for a, b in zip(lo, exp):
        assert a == pytest.approx(b, rel=1e-14, abs=1e-15)


@pytest.mark.parametrize("r,expect", [
    (1.0, "2222222222211000"),   # b = upper
    (0.5, "2222222221111000"),   # midpoint of the envelope
    (0.0, "2222222111110000"),   # b = lower
])
def test_llada_levels_hand_derived(r, expect):
    got = "".join(str(x) for x in levels_at_constant_risk(LLADA, 1.0, r))
    assert got == expect


def test_lavida_no_clip_closed_form():
    # late, T=32, d=1: mean p = 1/2, so upper = .9 p and lower = .72 p with
    # max .9 * 63/64 < 1: nothing clips.
    lo, up = policy.envelope(32, False, 0.45, 0.20, 1.0)
    p = [(2 * t - 1) / 64 for t in range(1, 33)]
    for a, b in zip(up, p):
        assert a == pytest.approx(0.9 * b, rel=1e-14)
    for a, b in zip(lo, p):
        assert a == pytest.approx(0.72 * b, rel=1e-14)
    hi1 = levels_at_constant_risk(LAVIDA, 1.0, 1.0)
    assert [hi1.count(i) for i in range(3)] == [12, 12, 8]
    hi0 = levels_at_constant_risk(LAVIDA, 1.0, 0.0)
    assert [hi0.count(i) for i in range(3)] == [15, 15, 2]


def test_table_a_prior(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "table_a_demand_prior.json")))
    assert list(policy.DEMAND_PRIOR) == g["demand"]


def _n_high(cfg, demand, r):
    return levels_at_constant_risk(cfg, demand, r).count(2)


def test_table_d_high_counts_within_reading(golden_dir):
    """Table D: the printed average number of high steps must be reachable:
    r ranges over [1 - alpha, 1] (c, chi in [0, 1]) and the high count is
    monotone in r, so it lies between the counts at the two ends."""
    g = json.load(open(os.path.join(golden_dir, "table_d_high_steps.json")))
    for row in g["rows"]:
        cfg = g["backbones"][row["backbone"]]
        rmin = 1.0 - cfg["alpha"]
        if row["demand"] == "uniform":
            lo_d = hi_d = 1.0
        else:
            lo_d, hi_d = min(policy.DEMAND_PRIOR), max(policy.DEMAND_PRIOR)
        lo = _n_high(cfg, lo_d, rmin)
        hi = _n_high(cfg, hi_d, 1.0)
        assert lo <= row["high"] <= hi, (row, lo, hi)


def test_table_d_rejects_other_normalisations(golden_dir):
    """The same table rules out the two other readings of the normaliser,
    which shows the pin above discriminates."""
    g = json.load(open(os.path.join(golden_dir, "table_d_high_steps.json")))
    # clip once: min(1, p * beta / mean(p)); LLaDA-V uniform d=1 at r=1
    T = 16
    p = [(33 - 2 * t) / 32 for t in range(1, T + 1)]
    once = [min(1.0, x * 0.75 / 0.5) for x in p]
    max_high_once = sum(1 for x in once if x >= 2 / 3)
    uni = [r["high"] for r in g["rows"]
           if r["backbone"] == "LLaDA-V" and r["demand"] == "uniform"]
    assert max_high_once < min(uni)
    # additive shift + clip: LaViDa lower trajectory (r = 0) alone already
    # gives more high steps than the default-demand average
    T = 32
    p = [(2 * t - 1) / 64 for t in range(1, T + 1)]
    shift = [min(1.0, max(0.0, x + (0.36 - 0.5))) for x in p]
    min_high_shift = sum(1 for x in shift if x >= 2 / 3)
    dflt = [r["high"] for r in g["rows"]
            if r["backbone"] == "LaViDa" and r["demand"] == "default"]
    assert min_high_shift > max(dflt)


def test_risk_and_allocation_special_cases():
    assert policy.risk(1, 1.0, 0.9, 0.1) == 1.0          # r_1 = 1
    assert policy.risk(5, 0.0, 0.9, 0.1) == 1.0          # alpha = 0
    assert policy.risk(5, 1.0, 1.0, 0.0) == 0.0          # confident, stable
    assert policy.risk(5, 1.0, 1.0, 1.0) == 1.0          # full churn
    assert policy.allocate(0.2, 0.7, 0.0) == 0.2         # r = 0 -> lower
    assert policy.allocate(0.2, 0.7, 1.0) == 0.7         # r = 1 -> upper


def test_quantize_thresholds():
    third = 1.0 / 3.0
    assert policy.quantize(0.0) == 0
    assert policy.quantize(math.nextafter(third, 0)) == 0
    assert policy.quantize(third) == 1
    assert policy.quantize(math.nextafter(2.0 / 3.0, 0)) == 1
    assert policy.quantize(2.0 / 3.0) == 2
    assert policy.quantize(1.0) == 2
    assert [policy.quantize(b, 4) for b in (0.1, 0.25, 0.5, 0.75)] == \
        [0, 1, 2, 3]
    assert policy.quantize(0.99, 1) == 0


def test_normalize_edges():
    p = policy.phase_profile(8, True)
    assert policy.normalize(p, 1.0) == [1.0] * 8
    assert policy.normalize(p, 1.5) == [1.0] * 8
    assert policy.normalize(p, 0.0) == [0.0] * 8
    assert policy.normalize(p, -0.1) == [0.0] * 8


@settings(max_examples=200, deadline=None)
@given(T=st.integers(1, 128), early=st.booleans(),
       beta=st.floats(0.001, 0.999))
def test_normalize_invariants(T, early, beta):
    p = policy.phase_profile(T, early)
    n = policy.normalize(p, beta)
    assert all(0.0 <= x <= 1.0 + 1e-15 for x in n)
    assert sum(n) / T == pytest.approx(beta, rel=1e-12, abs=1e-12)
    # phase ordering is preserved
    for i in range(T):
        for j in range(T):
            if p[i] > p[j]:
                assert n[i] >= n[j]


@settings(max_examples=200, deadline=None)
@given(T=st.integers(1, 64), early=st.booleans(), B=st.floats(0.05, 1.0),
       rho=st.floats(0.0, 1.0), d=st.floats(0.0, 1.0),
       cbar=st.floats(0.0, 1.0), chi=st.floats(0.0, 1.0),
       alpha=st.floats(0.0, 1.0))
def test_envelope_invariants(T, early, B, rho, d, cbar, chi, alpha):
    lo, up = policy.envelope(T, early, B, rho, d)
    assert sum(up) / T <= B + 1e-12                     # mean(upper) <= B
    for t in range(T):
        assert lo[t] <= up[t] + 1e-15
        r = policy.risk(t + 1, alpha, cbar, chi)
        b = policy.allocate(lo[t], up[t], r)
        assert lo[t] - 1e-15 <= b <= up[t] + 1e-15
    # widening d never reorders phases: upper keeps the order of p
    p = policy.phase_profile(T, early)
    for i in range(T - 1):
        if p[i] > p[i + 1]:
            assert up[i] >= up[i + 1]


@settings(max_examples=100, deadline=None)
@given(T=st.integers(2, 48), early=st.booleans(), B1=st.floats(0.05, 1.0),
       B2=st.floats(0.05, 1.0), r=st.floats(0.0, 1.0))
def test_level_monotone_in_budget(T, early, B1, B2, r):
    """Latency rises with B (App. D): for a fixed risk trace the level of
    every step is weakly monotone in B."""
    lo_B, hi_B = min(B1, B2), max(B1, B2)
    l1, u1 = policy.envelope(T, early, lo_B, 0.2, 0.8)
    l2, u2 = policy.envelope(T, early, hi_B, 0.2, 0.8)
    for t in range(T):
        a = policy.quantize(policy.allocate(l1[t], u1[t], r))
        b = policy.quantize(policy.allocate(l2[t], u2[t], r))
        assert a <= b
