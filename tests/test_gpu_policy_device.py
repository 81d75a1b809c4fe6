"""The closed-loop policy step on the GPU (Sec. 4.2: signals c̄ and χ after a
commitment, then Eqs. 7-9 for the next step) against the oracle
(oracle.policy.envelope, oracle.stats.mean_conf / churn, oracle.policy.step)
and against the library's host functions davet_step_stats +
davet_policy_step, bit for bit, on seeded inputs chosen so that any change
of summation order or any fused multiply-add would show: confidences
spanning many binades, empty masked sets, unchanged and changed
predictions, budgets near the Eq. 9 thresholds, and K = 1..4."""

import numpy as np
import pytest
import torch

import paper_2608_01821_amd as dv
from oracle import policy as opol
from oracle import stats as ostats

pytestmark = pytest.mark.gpu


def _policies(rng, n, K):
    out = []
    for _ in range(n):
        out.append(dv.Policy(float(rng.uniform(0.2, 0.9)),
                             float(rng.uniform(0.0, 1.0)),
                             float(rng.uniform(0.0, 1.0)),
                             float(rng.choice([1.0, 0.941, 0.824, 0.647,
                                               0.529])),
                             int(rng.integers(0, 2)), K))
    return out


@pytest.mark.parametrize("n,L,K,T,seed", [
    (1, 128, 3, 64, 0),
    (5, 24, 3, 4, 1),
    (16, 128, 3, 64, 2),
    (64, 256, 4, 32, 3),
    (7, 1024, 2, 8, 4),
    (3, 1, 3, 5, 5),
    (9, 37, 1, 6, 6),
])
def test_device_policy_step_matches_host(n, L, K, T, seed):
    rng = np.random.default_rng(seed)
    pols = _policies(rng, n, K)
    lower = np.empty(n * T)
    upper = np.empty(n * T)
    for s, p in enumerate(pols):
        lo, up = opol.envelope(T, bool(p.early), p.B, p.rho, p.demand)
        assert (lo, up) == tuple(dv.davet_policy_envelope(p, T))
        lower[s * T:(s + 1) * T] = lo
        upper[s * T:(s + 1) * T] = up
    for t in sorted({1, min(2, T - 1), T - 1}):
        if t < 1:
            continue
        # confidences over many binades; masked sets of every size incl. 0
        conf = (rng.random(n * L) ** 8).astype(np.float32)
        conf[rng.random(n * L) < 0.1] = 1.0
        masked = (rng.random(n * L) < rng.random(n).repeat(L)).astype(np.uint8)
        masked[:L] = 0 if n > 1 else masked[:L]          # an empty set
        am = rng.integers(0, 50, n * L).astype(np.int32)
        prev = np.where(rng.random(n * L) < 0.6, am,
                        rng.integers(0, 50, n * L)).astype(np.int32)
        d_conf = torch.from_numpy(conf).cuda()
        d_am = torch.from_numpy(am).cuda()
        d_prev = None if t == 1 else torch.from_numpy(prev).cuda()
        d_mask = torch.from_numpy(masked).cuda()
        lv = torch.full((n,), -1, dtype=torch.int32, device="cuda")
        bu = torch.full((n,), np.nan, dtype=torch.float64, device="cuda")
        rr = torch.full((n,), np.nan, dtype=torch.float64, device="cuda")
        dv.davet_policy_step_device(pols, t, T, lower, upper, d_conf, d_am,
                                    d_prev, d_mask, lv, bu, rr)
        torch.cuda.synchronize()
        g_lv, g_bu, g_r = lv.cpu().numpy(), bu.cpu().numpy(), rr.cpu().numpy()
        for s in range(n):
            o = slice(s * L, (s + 1) * L)
            lo_s = lower[s * T:(s + 1) * T].tolist()
            up_s = upper[s * T:(s + 1) * T].tolist()
            # the oracle's signals and next-step allocation
            ocb = ostats.mean_conf(conf[o], masked[o])
            och = ostats.churn(am[o], prev[o], masked[o], t == 1)
            ob, olv, orr = opol.step(t + 1, lo_s, up_s, pols[s].alpha, ocb,
                                     och, K)
            assert g_bu[s] == ob and g_r[s] == orr, (t, s, g_bu[s], ob)
            assert g_lv[s] == olv
            # and the library's host policy, on the same signals
            cb, ch = dv.davet_step_stats(conf[o], am[o],
                                         None if t == 1 else prev[o],
                                         masked[o])
            assert (cb, ch) == (ocb, och)
            b, l_, r = dv.davet_policy_step(pols[s], t + 1, T, lo_s, up_s,
                                            cb, ch)
            assert (b, l_, r) == (ob, olv, orr)


def test_device_policy_step_argument_checks():
    pols = [dv.Policy(0.5, 0.5, 1.0, 1.0, 1, 3)]
    lo, up = dv.davet_policy_envelope(pols[0], 4)
    x = torch.zeros(8, device="cuda")
    i = torch.zeros(8, dtype=torch.int32, device="cuda")
    m = torch.zeros(8, dtype=torch.uint8, device="cuda")
    o = torch.zeros(1, dtype=torch.int32, device="cuda")
    b = torch.zeros(1, dtype=torch.float64, device="cuda")
    with pytest.raises(dv.DavetError):            # t = T has no next step
        dv.davet_policy_step_device(pols, 4, 4, lo, up, x, i, i, m, o, b)
    with pytest.raises(dv.DavetError):            # t = 1 has no previous step
        dv.davet_policy_step_device(pols, 1, 4, lo, up, x, i, i, m, o, b)
    with pytest.raises(dv.DavetError):            # t > 1 needs one
        dv.davet_policy_step_device(pols, 2, 4, lo, up, x, i, None, m, o, b)
