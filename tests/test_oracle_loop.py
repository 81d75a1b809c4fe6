"""Invariants of the oracle's full loop (Sec. 3.1, Eq. 2; Sec. 4) on the tiny
fp32 workload: flags only go from masked to committed, exactly min(k, |M_t|)
positions are revealed per step, committed tokens never change, every
position is revealed after T steps when k T = L, levels follow the schedule
or the policy, and the policy sees the signals of the previous step."""

import numpy as np
import pytest

import synth
from oracle import loop, policy


def _weights(cfg):
    return dict(embed=synth.gen_embed(cfg), head=synth.gen_head(cfg),
                layers=[synth.gen_layer_weights(cfg, i)
                        for i in range(cfg.n_layers)])


@pytest.fixture(scope="module")
def c1():
    cfg = synth.get_config(1)
    return cfg, _weights(cfg), synth.gen_sample(cfg)


def _check_trajectory(cfg, res, k):
    tr = res["trace"]
    L = cfg.resp_len
    masked = np.ones(L, np.uint8)
    ids = np.full(L, cfg.mask_id)
    for t in range(len(tr["levels"])):
        sel = tr["selected"][t]
        assert len(sel) == min(k, int(masked.sum()))
        assert all(masked[i] for i in sel)
        # confidences exist exactly at masked positions
        assert np.all(np.isfinite(tr["conf"][t][masked == 1]))
        assert np.all(tr["conf"][t][masked == 0] == -np.inf)
        for i in sel:
            masked[i] = 0
            ids[i] = tr["argmax"][t][i]
    assert np.array_equal(masked, res["masked"])
    assert np.array_equal(ids, res["ids"])
    assert np.all(res["ids"][res["masked"] == 0] != cfg.mask_id)


def test_fixed_schedule_loop(c1):
    cfg, w, s = c1
    res = loop.run_sequence(cfg, w, s["visual"][0], 1, s["prompts"][0],
                            cfg.steps, cfg.k, fixed_levels=cfg.fixed_levels)
    assert res["trace"]["levels"] == list(cfg.fixed_levels)
    assert cfg.k * cfg.steps == cfg.resp_len
    assert res["masked"].sum() == 0
    _check_trajectory(cfg, res, cfg.k)


def test_policy_loop_uses_previous_signals(c1):
    cfg, w, s = c1
    pol = dict(early=True, B=0.75, rho=0.2, alpha=1.0)
    res = loop.run_sequence(cfg, w, s["visual"][0], 1, s["prompts"][0],
                            cfg.steps, 3, pol=pol, demand=0.824)
    tr = res["trace"]
    lo, up = policy.envelope(cfg.steps, True, 0.75, 0.2, 0.824)
    assert tr["risks"][0] == 1.0
    for t in range(1, cfg.steps):
        r = 1.0 - ((1.0 * tr["cbar"][t - 1]) * (1.0 - tr["chi"][t - 1]))
        assert tr["risks"][t] == r
        assert lo[t] <= tr["budgets"][t] <= up[t]
        assert tr["levels"][t] == policy.quantize(tr["budgets"][t])
    assert tr["chi"][0] == 0.0
    _check_trajectory(cfg, res, 3)
    assert res["masked"].sum() == cfg.resp_len - 3 * cfg.steps


def test_k_larger_than_remaining(c1):
    cfg, w, s = c1
    res = loop.run_sequence(cfg, w, s["visual"][0], 1, s["prompts"][0],
                            3, 15, fixed_levels=(0, 0, 0))
    # 15 + 15 + 2 = 32: the last step reveals only what is left
    assert [len(x) for x in res["trace"]["selected"]] == [15, 15, 2]
    _check_trajectory(cfg, res, 15)
