"""The DAVET denoising loop (Sec. 3.1 with Sec. 4; the procedure of Fig. 2).

Once per sample: build the K evidence views from the single encoding and,
in policy mode, the evidence envelope.  Then for t = 1..T: choose the level
(fixed schedule, or Eqs. 7-9 from the previous step's signals), run the
denoiser over [view | prompt | response] (Eq. 1), decode, commit (Eq. 2),
and record the signals for the next step's risk.  Samples of a batch are
independent (their attention never mixes), so they run one after another.
"""

import math

import numpy as np

from . import decode, model, policy, stats, views


def run_sequence(cfg, weights, visual, n_crops, prompt_ids, T, k,
                 fixed_levels=None, pol=None, demand=1.0, out_dtype=None):
    """One sample.  ``pol`` = dict(early, B, rho, alpha) selects policy mode.
    Returns a dict with final ids, masked flags and the per-step trace."""
    out_dtype = out_dtype or cfg.dtype
    levels, maps = views.build_views(visual, n_crops, cfg.grid, cfg.K,
                                     out_dtype)
    L = cfg.resp_len
    resp = np.full(L, cfg.mask_id, dtype=np.int32)
    masked = np.ones(L, dtype=np.uint8)
    if pol is not None:
        lower, upper = policy.envelope(T, pol["early"], pol["B"], pol["rho"],
                                       demand)
    cbar, chi = 0.0, 0.0
    prev_am = None
    trace = dict(levels=[], budgets=[], risks=[], cbar=[], chi=[],
                 selected=[], conf=[], argmax=[])
    for t in range(1, T + 1):
        if pol is not None:
            b, lv, r = policy.step(t, lower, upper, pol["alpha"], cbar, chi,
                                   cfg.K)
        else:
            lv, b, r = int(fixed_levels[t - 1]), math.nan, math.nan
        pos, lg = model.step_logits(cfg, levels[lv], prompt_ids, resp,
                                    masked, weights)
        am, cf = decode.argmax_conf(lg, cfg.mask_id)
        conf_full = np.full(L, -np.inf, dtype=np.float64)
        am_full = np.full(L, -1, dtype=np.int32)
        conf_full[pos] = cf
        am_full[pos] = am
        sel = decode.select(conf_full, masked, k)
        resp, masked = decode.commit(resp, masked, am_full, sel)
        cbar = stats.mean_conf(conf_full, masked)
        chi = stats.churn(am_full, prev_am, masked, t == 1)
        prev_am = am_full
        for key, val in (("levels", lv), ("budgets", b), ("risks", r),
                         ("cbar", cbar), ("chi", chi), ("selected", sel),
                         ("conf", conf_full), ("argmax", am_full)):
            trace[key].append(val)
    return dict(ids=resp, masked=masked, trace=trace, views=levels,
                maps=maps)
