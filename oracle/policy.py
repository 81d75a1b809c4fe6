"""Denoising-aware allocation policy (Sec. 4.2, Eqs. 6-9; Appendix A).

All arithmetic is IEEE double, evaluated left to right exactly as the
equations print it, with no fused multiply-add (Python floats never fuse).
"""

import math
from typing import List, Sequence

# Demand prior d(o) per operation category (Appendix A, Table A), in the
# category order: lexical readout, numerical reasoning, entity grounding,
# binary decision, general understanding.
DEMAND_PRIOR = (1.000, 0.941, 0.824, 0.647, 0.529)


def phase_profile(T: int, early: bool) -> List[float]:
    """Two-orientation phase family (Sec. 4.2): early grounding
    p_t = 1 - (t - 0.5)/T, late verification p_t = (t - 0.5)/T, t = 1..T."""
    if T <= 0:
        raise ValueError("T must be positive")
    out = []
    for t in range(1, T + 1):
        x = (t - 0.5) / T
        out.append(1.0 - x if early else x)
    return out


def normalize(p: Sequence[float], beta: float) -> List[float]:
    """N(p; beta): rescale the profile and clip to [0, 1] so its mean is beta
    (Sec. 4.2).  Reading: min(1, s * p_t) with the scale s solved exactly.
    Entries are clipped from the largest p down (ties by lower index); for j
    clipped entries s_j = (T*beta - j) / (sum of the unclipped p_t, ascending
    t), and the first j whose largest unclipped entry satisfies
    s_j * p <= 1 is used.  beta >= 1 gives all ones, beta <= 0 all zeros."""
    T = len(p)
    if beta >= 1.0:
        return [1.0] * T
    if beta <= 0.0:
        return [0.0] * T
    order = sorted(range(T), key=lambda i: (-p[i], i))
    clipped = [False] * T
    target = T * beta
    s = None
    for j in range(T):
        denom = 0.0
        for t in range(T):
            if not clipped[t]:
                denom = denom + p[t]
        sj = (target - j) / denom
        if sj * p[order[j]] <= 1.0:
            s = sj
            break
        clipped[order[j]] = True
    if s is None:              # only reachable through rounding at beta ~ 1
        return [1.0] * T
    return [1.0 if clipped[t] else s * p[t] for t in range(T)]


def envelope(T: int, early: bool, B: float, rho: float, demand: float):
    """Evidence envelope, Eq. (6): lower = N(p; (1-rho)B),
    upper = N(p; [1 - rho + rho d(o)] B)."""
    p = phase_profile(T, early)
    lower = normalize(p, (1.0 - rho) * B)
    upper = normalize(p, ((1.0 - rho) + rho * demand) * B)
    return lower, upper


def risk(t: int, alpha: float, cbar_prev: float, churn_prev: float) -> float:
    """Trajectory risk, Eq. (7): r_1 = 1; r_t = 1 - alpha c_{t-1} (1 - chi_{t-1})."""
    if t == 1:
        return 1.0
    return 1.0 - ((alpha * cbar_prev) * (1.0 - churn_prev))


def allocate(lower_t: float, upper_t: float, r_t: float) -> float:
    """Envelope allocation, Eq. (8): b_t = lower_t + r_t (upper_t - lower_t)."""
    return lower_t + r_t * (upper_t - lower_t)


def quantize(b: float, K: int = 3) -> int:
    """K-level quantisation, Eq. (9) (canonical thirds for K = 3): the level
    is the number of thresholds j/K, j = 1..K-1, that are <= b."""
    lv = 0
    for j in range(1, K):
        if (j / K) <= b:
            lv += 1
    return lv


def step(t: int, lower, upper, alpha: float, cbar_prev: float,
         churn_prev: float, K: int = 3):
    """(b_t, level_t, r_t) for step t (1-based)."""
    r = risk(t, alpha, cbar_prev, churn_prev)
    b = allocate(lower[t - 1], upper[t - 1], r)
    return b, quantize(b, K), r


def is_finite_budget(b: float) -> bool:
    return math.isfinite(b)
