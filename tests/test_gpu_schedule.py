"""The whole loop on the GPU (Sec. 3.1 with Sec. 4).

1. Teacher-forced along the oracle's own trajectory: at every step the GPU
   gets the oracle's state (ids, flags, level) and its denoiser output is
   compared with the oracle's; the commitment kernel gets the oracle's
   confidences (rounded to float32, the kernel's precision) and must select
   exactly what the oracle selects from the same float32 values.
2. Free-running ``davet_run_schedule`` (fixed schedule and policy mode):
   schedule, per-step reveal counts and flag monotonicity hold exactly; at
   every step the policy's levels/budgets equal what the oracle's policy
   (oracle.stats + oracle.policy) gives for the run's own confidence trace;
   step 1 (identical inputs on both sides)
   matches the oracle; and later steps match it for as long as the two
   trajectories coincide.
"""

import numpy as np
import pytest
import torch

import paper_2608_01821_amd as dv
import synth
from gpu_util import (TOL, Model, Sample, compare, dev_tensor, model_cfg,
                      oracle_step, run_gpu_step, to_mode, view_geom,
                      workspace)
from oracle import decode, loop
from oracle import policy as opol
from oracle import stats as ostats

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cid", [1, 11])
def test_teacher_forced_loop(cid):
    cfg = synth.get_any_config(cid)
    mdl = Model(cfg)
    s = synth.gen_sample(cfg)
    sample = Sample(cfg, s["n_crops"][0], s["visual"][0], s["prompts"][0])
    ref = loop.run_sequence(cfg, mdl.host, sample.visual, s["n_crops"][0],
                            s["prompts"][0], cfg.steps, cfg.k,
                            fixed_levels=cfg.fixed_levels,
                            out_dtype=mdl.mode)
    tr = ref["trace"]
    L = cfg.resp_len
    ids = np.full(L, cfg.mask_id, np.int32)
    masked = np.ones(L, np.uint8)
    for t in range(cfg.steps):
        lv = tr["levels"][t]
        g_conf, g_am, g_lg = run_gpu_step(cfg, mdl, [sample], [lv], ids,
                                          masked)
        pos, lg, am, cf = oracle_step(cfg, mdl, sample, lv, ids, masked)
        compare(cfg, TOL[mdl.mode], masked, g_conf[0], g_am[0], g_lg[0], pos,
                lg, am, cf)
        # commitment on the oracle's confidences at float32
        c32 = tr["conf"][t].astype(np.float32)
        d_ids = torch.from_numpy(ids.copy()).cuda()
        d_m = torch.from_numpy(masked.copy()).cuda()
        sel = torch.empty(cfg.k, dtype=torch.int32, device="cuda")
        dv.davet_unmask(1, L, cfg.k, torch.from_numpy(c32).cuda(),
                        torch.from_numpy(tr["argmax"][t]).cuda(), d_ids, d_m,
                        sel)
        exp_sel = decode.select(c32, masked, cfg.k)
        got = sel.cpu().numpy()
        assert sorted(got[got >= 0].tolist()) == exp_sel
        ids, masked = decode.commit(ids, masked, tr["argmax"][t], exp_sel)
        assert np.array_equal(d_ids.cpu().numpy(), ids)
        assert np.array_equal(d_m.cpu().numpy(), masked)


def _run_schedule(cfg, mdl, s, pols=None, fixed=None, weights=None,
                  mailbox=None):
    n = cfg.n_seqs
    L, T = cfg.resp_len, cfg.steps
    mode = mdl.mode
    geoms = [view_geom(cfg, c, mode) for c in s["n_crops"]]
    sizes = [dv.davet_view_sizes(g) for g in geoms]
    tdt = torch.float32 if mode == "f32" else torch.int16
    visual = [dev_tensor(v, mode) for v in s["visual"]]
    bufs = [torch.empty((sz[l], cfg.d), dtype=tdt, device="cuda")
            for sz in sizes for l in range(cfg.K - 1)]
    prompt = torch.from_numpy(np.concatenate(s["prompts"])).cuda()
    cu = np.concatenate([[0], np.cumsum([len(p) for p in s["prompts"]])])
    total = sum(sz[-1] for sz in sizes) + int(cu[-1]) + n * L
    ws = workspace(cfg, total, n, L, mode)
    ids = torch.full((n * L,), cfg.mask_id, dtype=torch.int32, device="cuda")
    msk = torch.ones((n * L,), dtype=torch.uint8, device="cuda")
    ctr = torch.empty((T, n * L), device="cuda")
    atr = torch.empty((T, n * L), dtype=torch.int32, device="cuda")
    levels, budgets = dv.davet_run_schedule(
        model_cfg(cfg, mode), weights or mdl.weights, geoms, visual, bufs,
        prompt, cu, L, T,
        cfg.k, pols, fixed, ids, msk, ws, ctr, atr, mailbox=mailbox)
    torch.cuda.synchronize()
    return (np.array(levels).reshape(n, T), np.array(budgets).reshape(n, T),
            ctr.cpu().numpy().reshape(T, n, L),
            atr.cpu().numpy().reshape(T, n, L),
            ids.cpu().numpy().reshape(n, L), msk.cpu().numpy().reshape(n, L))


def _check_invariants(cfg, conf_tr, am_tr, ids, msk):
    """Reveal counts, flag monotonicity, committed tokens never change."""
    T, n, L = conf_tr.shape
    for s in range(n):
        live = np.ones(L, bool)
        for t in range(T):
            fin = np.isfinite(conf_tr[t, s])
            assert np.array_equal(fin, live), "conf finite exactly at masked"
            nxt = np.isfinite(conf_tr[t + 1, s]) if t + 1 < T else \
                msk[s].astype(bool)
            assert not np.any(nxt & ~live), "a committed position re-masked"
            revealed = live & ~nxt
            assert revealed.sum() == min(cfg.k, live.sum())
            assert np.array_equal(ids[s][revealed], am_tr[t, s][revealed])
            live = nxt
        assert np.all(ids[s][~msk[s].astype(bool)] != cfg.mask_id)


def _gpu_states(cfg, conf_tr, am_tr, final_masked, s):
    """(live set, ids) before every step, rebuilt from the run's traces."""
    T, _, L = conf_tr.shape
    ids = np.full(L, cfg.mask_id, np.int32)
    live = np.ones(L, bool)
    out = []
    for t in range(T):
        out.append((live.copy(), ids.copy()))
        nxt = np.isfinite(conf_tr[t + 1, s]) if t + 1 < T else \
            final_masked[s].astype(bool)
        rev = live & ~nxt
        ids[rev] = am_tr[t, s][rev]
        live = nxt
    return out


def _oracle_states(cfg, tr):
    L = cfg.resp_len
    ids = np.full(L, cfg.mask_id, np.int32)
    live = np.ones(L, bool)
    out = []
    for t in range(len(tr["levels"])):
        out.append((live.copy(), ids.copy()))
        for i in tr["selected"][t]:
            ids[i] = tr["argmax"][t][i]
            live[i] = False
    return out


# The free-running loop stores no logits, so the per-row confidence bound of
# the teacher-forced checks (derived from the logit error) is not available
# here; along the shared prefix of the two trajectories a coarse relative
# tolerance is used instead (the tight checks are the teacher-forced ones).
TRAJ_CONF_RTOL = {"f32": 1e-4, "bf16": 5e-2}


def _trajectory_prefix_match(cfg, ref_tr, conf_tr, am_tr, final_masked, s):
    """Steps compared while the GPU and oracle states coincide; returns the
    number of steps compared."""
    gs = _gpu_states(cfg, conf_tr, am_tr, final_masked, s)
    os_ = _oracle_states(cfg, ref_tr)
    n_ok = 0
    for t, ((gl, gi), (ol, oi)) in enumerate(zip(gs, os_)):
        if not (np.array_equal(gl, ol) and np.array_equal(gi, oi)):
            break
        c = conf_tr[t, s][gl]
        r = ref_tr["conf"][t][ol]
        err = np.abs(c - r) / r
        assert err.max() <= TRAJ_CONF_RTOL[cfg.dtype], (t, err.max())
        n_ok += 1
    return n_ok


def _check_policy_trace(cfg, pols, lv, bu, ctr, atr, msk):
    """Every step's level and budget of every sequence equal the oracle's
    allocation (oracle.policy) from the signals (oracle.stats) of the run's
    own previous step: its confidence and prediction traces."""
    T = cfg.steps
    for i, pol in enumerate(pols):
        lo, up = opol.envelope(T, bool(pol.early), pol.B, pol.rho, pol.demand)
        cb, ch = 0.0, 0.0
        for t in range(1, T + 1):
            b, l_, _ = opol.step(t, lo, up, pol.alpha, cb, ch, cfg.K)
            assert b == bu[i, t - 1] and l_ == lv[i, t - 1], (i, t)
            after = np.isfinite(ctr[t, i]) if t < T else msk[i].astype(bool)
            cb = ostats.mean_conf(ctr[t - 1, i], after)
            ch = ostats.churn(atr[t - 1, i], None if t == 1 else
                              atr[t - 2, i], after, t == 1)


def test_run_schedule_fixed_tiny():
    cfg = synth.get_config(1)
    mdl = Model(cfg)
    s = synth.gen_sample(cfg)
    lv, bu, ctr, atr, ids, msk = _run_schedule(cfg, mdl, s,
                                               fixed=s["schedule"])
    assert np.array_equal(lv[0], np.array(cfg.fixed_levels))
    assert np.all(np.isnan(bu))
    assert msk.sum() == 0
    _check_invariants(cfg, ctr, atr, ids, msk)
    ref = loop.run_sequence(cfg, mdl.host, s["visual"][0], 1, s["prompts"][0],
                            cfg.steps, cfg.k, fixed_levels=cfg.fixed_levels,
                            out_dtype="f32")
    assert _trajectory_prefix_match(cfg, ref["trace"], ctr, atr, msk, 0) >= 1


@pytest.mark.parametrize("cid", [12, 13])
def test_run_schedule_policy_ragged(cid):
    cfg = synth.get_any_config(cid)
    mdl = Model(cfg)
    s = synth.gen_sample(cfg)
    p = cfg.policy
    pols = [dv.Policy(p["B"], p["rho"], p["alpha"], dv.davet_demand_prior(c),
                      1 if p["early"] else 0, cfg.K) for c in s["categories"]]
    lv, bu, ctr, atr, ids, msk = _run_schedule(cfg, mdl, s, pols=pols)
    _check_invariants(cfg, ctr, atr, ids, msk)
    T, L = cfg.steps, cfg.resp_len
    _check_policy_trace(cfg, pols, lv, bu, ctr, atr, msk)
    for i, pol in enumerate(pols):
        ref = loop.run_sequence(cfg, mdl.host,
                                to_mode(s["visual"][i], mdl.mode)[1],
                                s["n_crops"][i], s["prompts"][i], T, cfg.k,
                                pol=p, demand=dv.davet_demand_prior(
                                    s["categories"][i]), out_dtype=mdl.mode)
        assert ref["trace"]["levels"][0] == lv[i, 0]
        assert ref["trace"]["budgets"][0] == bu[i, 0]
        assert _trajectory_prefix_match(cfg, ref["trace"], ctr, atr, msk,
                                        i) >= 1


def test_run_schedule_head_over_several_row_tiles():
    """Five sequences of 100 response positions: the vocabulary head sees up
    to 500 masked rows, so the schedule sizes its grid for several 128-row
    tiles per vocabulary slab; every sequence still matches the oracle."""
    import dataclasses
    cfg = dataclasses.replace(synth.get_any_config(12), resp_len=100, k=40,
                              steps=3)
    mdl = Model(cfg)
    s = synth.gen_sample(cfg)
    p = cfg.policy
    pols = [dv.Policy(p["B"], p["rho"], p["alpha"], dv.davet_demand_prior(c),
                      1 if p["early"] else 0, cfg.K) for c in s["categories"]]
    lv, bu, ctr, atr, ids, msk = _run_schedule(cfg, mdl, s, pols=pols)
    _check_invariants(cfg, ctr, atr, ids, msk)
    _check_policy_trace(cfg, pols, lv, bu, ctr, atr, msk)
    assert cfg.n_seqs * cfg.resp_len > 3 * 128
    for i, pol in enumerate(pols):
        ref = loop.run_sequence(cfg, mdl.host,
                                to_mode(s["visual"][i], mdl.mode)[1],
                                s["n_crops"][i], s["prompts"][i], cfg.steps,
                                cfg.k, pol=p, demand=dv.davet_demand_prior(
                                    s["categories"][i]), out_dtype=mdl.mode)
        assert ref["trace"]["levels"][0] == lv[i, 0]
        assert _trajectory_prefix_match(cfg, ref["trace"], ctr, atr, msk,
                                        i) >= 1


def test_run_schedule_tiled_head():
    """The loop as the benchmark runs it, with the head packed by
    davet_pack_head: 500, 300 and 100 masked rows over three steps (the head's
    256 x 256 tile, then its 128 x 256 tile over three and one row slots).
    Step 1 sees identical inputs in both layouts: the same argmaxes and
    confidences up to the regrouping of the softmax sum; the tiled run keeps
    every invariant and matches the oracle as the row-major run does."""
    import dataclasses
    from gpu_util import assert_conf_regrouped
    cfg = dataclasses.replace(synth.get_any_config(12), resp_len=100, k=40,
                              steps=3)
    mdl = Model(cfg)
    tiled = torch.empty(dv.davet_head_tiled_elems(cfg.vocab, cfg.d),
                        dtype=torch.int16, device="cuda")
    dv.davet_pack_head(mdl.dev_head, tiled, cfg.vocab, cfg.d,
                       dv.DAVET_F16 if mdl.mode == "f16" else dv.DAVET_BF16)
    w_tiled = dv.Weights(mdl.dev_embed, tiled, mdl.dev_layers,
                         head_layout=dv.DAVET_HEAD_TILED)
    s = synth.gen_sample(cfg)
    p = cfg.policy
    pols = [dv.Policy(p["B"], p["rho"], p["alpha"], dv.davet_demand_prior(c),
                      1 if p["early"] else 0, cfg.K) for c in s["categories"]]
    lv_r, _, ctr_r, atr_r, _, _ = _run_schedule(cfg, mdl, s, pols=pols)
    lv, bu, ctr, atr, ids, msk = _run_schedule(cfg, mdl, s, pols=pols,
                                               weights=w_tiled)
    _check_invariants(cfg, ctr, atr, ids, msk)
    _check_policy_trace(cfg, pols, lv, bu, ctr, atr, msk)
    assert np.array_equal(lv[:, 0], lv_r[:, 0])
    assert np.array_equal(atr[0], atr_r[0])
    assert_conf_regrouped(ctr[0], ctr_r[0])
    for i, pol in enumerate(pols):
        ref = loop.run_sequence(cfg, mdl.host,
                                to_mode(s["visual"][i], mdl.mode)[1],
                                s["n_crops"][i], s["prompts"][i], cfg.steps,
                                cfg.k, pol=p, demand=dv.davet_demand_prior(
                                    s["categories"][i]), out_dtype=mdl.mode)
        assert ref["trace"]["levels"][0] == lv[i, 0]
        assert _trajectory_prefix_match(cfg, ref["trace"], ctr, atr, msk,
                                        i) >= 1


def test_run_schedule_64_sequences():
    """The policy loop over 64 sequences, the most the C ABI takes (the
    device policy step serves four per wavefront, the pinned mailbox holds
    64 levels): every invariant on every sequence, and three sequences
    against the oracle's own trajectory."""
    import dataclasses
    cfg = dataclasses.replace(synth.get_any_config(12), n_seqs=64,
                              resp_len=32, k=8, steps=3)
    mdl = Model(cfg)
    s = synth.gen_sample(cfg)
    p = cfg.policy
    pols = [dv.Policy(p["B"], p["rho"], p["alpha"], dv.davet_demand_prior(c),
                      1 if p["early"] else 0, cfg.K) for c in s["categories"]]
    lv, bu, ctr, atr, ids, msk = _run_schedule(cfg, mdl, s, pols=pols)
    _check_invariants(cfg, ctr, atr, ids, msk)
    _check_policy_trace(cfg, pols, lv, bu, ctr, atr, msk)
    for i in (0, 31, 63):
        ref = loop.run_sequence(cfg, mdl.host,
                                to_mode(s["visual"][i], mdl.mode)[1],
                                s["n_crops"][i], s["prompts"][i], cfg.steps,
                                cfg.k, pol=p, demand=dv.davet_demand_prior(
                                    s["categories"][i]), out_dtype=mdl.mode)
        assert ref["trace"]["levels"][0] == lv[i, 0]
        assert _trajectory_prefix_match(cfg, ref["trace"], ctr, atr, msk,
                                        i) >= 1


def test_run_schedule_wait_limit_and_mailbox_reuse():
    """The host's wait for a step's published levels is bounded: with a
    limit far below one step's duration (one 8B-shaped layer, ~0.5 ms per
    step) the call returns DAVET_EHIP while the stream keeps running, and
    after the stream drains the same mailbox serves a normal call whose
    levels and budgets equal those of a call on a fresh mailbox (each call
    takes stamps no earlier call on that mailbox used)."""
    import dataclasses
    cfg = dataclasses.replace(synth.get_config(2), steps=3, schedule="policy",
                              fixed_levels=None)
    mdl = Model(cfg, keep_host=False)
    s = synth.gen_sample(cfg)
    p = cfg.policy
    pols = [dv.Policy(p["B"], p["rho"], p["alpha"], dv.davet_demand_prior(0),
                      1 if p["early"] else 0, cfg.K)]
    mb = dv.Mailbox()
    try:
        dv.davet_set_wait_limit(1e-6)
        with pytest.raises(dv.DavetError) as e:
            _run_schedule(cfg, mdl, s, pols=pols, mailbox=mb)
        assert e.value.status == -5 and "no levels published" in str(e.value)
    finally:
        torch.cuda.synchronize()          # the failed call's steps drain
        dv.davet_set_wait_limit(120.0)
    lv_a, bu_a = _run_schedule(cfg, mdl, s, pols=pols, mailbox=mb)[:2]
    mb2 = dv.Mailbox()
    lv_b, bu_b = _run_schedule(cfg, mdl, s, pols=pols, mailbox=mb2)[:2]
    mb.close()
    mb2.close()
    assert np.array_equal(lv_a, lv_b) and np.array_equal(bu_a, bu_b)
    assert np.all(np.isfinite(bu_a))
