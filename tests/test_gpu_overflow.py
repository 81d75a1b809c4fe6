"""The fp16 overflow counter (davet_fp16_overflow_count).

It counts the non-finite 16-bit values a step stored as projection outputs:
the rotated Q/K/V columns and the SwiGLU product.  The expected count comes
from the oracle's values of those two tensors (oracle.model.layer_parts).

To push a chosen share of them past the fp16 range, both sides scale one
weight matrix by a power of two.  The fp16 scaling is exact, so the oracle
sees exactly the weights the device holds.  fp16 rounds to nearest even, so
a value overflows when its magnitude is at least 65520.  The GPU computes
these values from fp16 operands with fp32 accumulation, within a few 1e-3
of the oracle.  So the count must lie between the oracle's counts at
65520 * 1.03 and at 65520 / 1.03.

Two shapes cover both store paths.  At d = 256 each projection runs in one
K pass, and the GEMM epilogue stores (and counts) its outputs.  At d = ffn =
2048 the row counts here are small, so the Q/K/V and gate/up projections
split K in two, and the reduce kernels store and count instead.  The
profiler's launch classes confirm which path ran.
"""

import dataclasses

import numpy as np
import pytest
import torch

import synth
import paper_2608_01821_amd as dv
from gpu_util import Model, Sample, model_cfg, random_state, view_geom, \
    workspace
from oracle import model as omodel

pytestmark = pytest.mark.gpu

OVERFLOW_AT = 65520.0
MARGIN = 1.03
LEVEL = 2            # the raw view: the schedule and the single steps share it
SHARE = 0.03         # aimed-for share of overflowing elements


def _cfg(kind):
    base = synth.get_any_config(11)
    if kind == "direct":
        return dataclasses.replace(base, n_layers=1)
    return dataclasses.replace(base, n_layers=1, d=2048, n_heads=16,
                               ffn=2048)


@pytest.fixture(scope="module", params=["direct", "splitk"])
def setup(request):
    cfg = _cfg(request.param)
    mdl = Model(cfg, "f16")
    s = synth.gen_sample(cfg)
    smp = Sample(cfg, s["n_crops"][0], s["visual"][0], s["prompts"][0], "f16")
    rng = np.random.default_rng(3)
    ids, masked = random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab, 0.7)
    return request.param, cfg, mdl, smp, ids, masked


def _scaled(mdl, name, k):
    """(device weights, oracle layer dict) with layer 0's `name` matrix
    multiplied by 2**k on both sides."""
    lw = dict(mdl.dev_layers[0])
    w16 = lw[name].view(torch.float16)
    assert float(w16.abs().max()) * 2.0 ** k < 65504.0
    lw[name] = (w16 * 2.0 ** k).view(torch.int16)
    host = dict(mdl.host["layers"][0])
    host[name] = host[name] * np.float32(2.0 ** k)
    return dv.Weights(mdl.dev_embed, mdl.dev_head, [lw]), host


def _parts(cfg, mdl, smp, host_layer, ids, masked):
    x = omodel.embed_sequence(smp.ref_levels[LEVEL], smp.prompt, ids, masked,
                              mdl.host["embed"], cfg.mask_id)
    ang = omodel.rope_angles(x.shape[0], cfg.head_dim, cfg.rope_theta)
    _, qkv, hdn = omodel.layer_parts(x, host_layer, cfg.n_heads, cfg.head_dim,
                                     cfg.rms_eps, ang)
    return qkv, hdn


def _exponent(vals):
    """The power of two that lifts about SHARE of |vals| past 65520."""
    q = np.quantile(np.abs(vals), 1.0 - SHARE)
    return int(np.round(np.log2(OVERFLOW_AT / q)))


def _bracket(vals):
    a = np.abs(vals)
    return (int(np.count_nonzero(a >= OVERFLOW_AT * MARGIN)),
            int(np.count_nonzero(a >= OVERFLOW_AT / MARGIN)))


def _step(cfg, weights, smp, ids, masked, ws=None, mode="f16"):
    L = cfg.resp_len
    nv = smp.sizes[LEVEL]
    if ws is None:
        ws = workspace(cfg, nv + len(smp.prompt) + L, 1, L, mode)
        ws.fill_(0xAB)      # the step must clear the counter itself
    conf = torch.empty(L, device="cuda")
    am = torch.empty(L, dtype=torch.int32, device="cuda")
    dv.davet_denoise_step(
        model_cfg(cfg, mode), weights, [smp.dev_levels[LEVEL]], [nv],
        smp.dev_prompt, [0, len(smp.prompt)],
        torch.from_numpy(np.ascontiguousarray(ids, np.int32)).cuda(),
        torch.from_numpy(np.ascontiguousarray(masked, np.uint8)).cuda(), L,
        conf, am, None, ws)
    return dv.davet_fp16_overflow_count(ws), ws


def test_normal_step_counts_zero(setup):
    kind, cfg, mdl, smp, ids, masked = setup
    dv.prof_enable(256)
    try:
        dv.prof_reset()
        cnt, _ = _step(cfg, mdl.weights, smp, ids, masked)
        torch.cuda.synchronize()
        launches = dv.prof_read()
    finally:
        dv.prof_enable(0)
    assert cnt == 0
    # in the 16-bit path the "rope" class is the split-K Q/K/V reduction
    assert (launches["rope"][0] > 0) == (kind == "splitk")


def test_swiglu_overflow_count(setup):
    """Only the SwiGLU product leaves the fp16 range (up projection scaled):
    the count brackets the oracle's, and the next ordinary step on the same
    workspace reads 0."""
    kind, cfg, mdl, smp, ids, masked = setup
    _, hdn1 = _parts(cfg, mdl, smp, mdl.host["layers"][0], ids, masked)
    k = _exponent(hdn1)
    weights, host = _scaled(mdl, "wu", k)
    qkv, hdn = _parts(cfg, mdl, smp, host, ids, masked)
    assert _bracket(qkv)[1] == 0
    lo, hi = _bracket(hdn)
    assert lo > 0
    cnt, ws = _step(cfg, weights, smp, ids, masked)
    print("%s swiglu overflow: 2^%d, count %d in [%d, %d] of %d"
          % (kind, k, cnt, lo, hi, hdn.size))
    assert lo <= cnt <= hi
    cnt2, _ = _step(cfg, mdl.weights, smp, ids, masked, ws)
    assert cnt2 == 0


def test_qkv_overflow_counted(setup):
    """Q/K/V leave the fp16 range (Q/K/V projection scaled).  Every later
    16-bit store of the sequence may turn non-finite as well, so the count is
    at least the oracle's Q/K/V count and at most that plus every element of
    the SwiGLU product."""
    kind, cfg, mdl, smp, ids, masked = setup
    qkv1, _ = _parts(cfg, mdl, smp, mdl.host["layers"][0], ids, masked)
    k = _exponent(qkv1)
    weights, host = _scaled(mdl, "wqkv", k)
    qkv = qkv1 * 2.0 ** k               # the projection is linear in wqkv
    lo, hi = _bracket(qkv)
    assert lo > 0
    cnt, _ = _step(cfg, weights, smp, ids, masked)
    n_hdn = qkv.shape[0] * cfg.ffn
    print("%s qkv overflow: 2^%d, count %d, q/k/v bracket [%d, %d]"
          % (kind, k, cnt, lo, hi))
    assert lo <= cnt <= hi + n_hdn


def test_f32_model_counts_zero():
    cfg = synth.get_any_config(1)
    mdl = Model(cfg, "f32", keep_host=False)
    s = synth.gen_sample(cfg)
    smp = Sample(cfg, s["n_crops"][0], s["visual"][0], s["prompts"][0], "f32")
    ids = np.full(cfg.resp_len, cfg.mask_id, np.int32)
    cnt, _ = _step(cfg, mdl.weights, smp, ids, np.ones(cfg.resp_len, np.uint8),
                   mode="f32")
    assert cnt == 0


def test_schedule_counts_over_all_steps(setup):
    """davet_run_schedule clears the counter once and counts every step: two
    fixed-level steps read the sum of the same two steps run one by one."""
    kind, cfg, mdl, smp, _, _ = setup
    L, T = cfg.resp_len, 2
    ids0 = np.full(L, cfg.mask_id, np.int32)
    m0 = np.ones(L, np.uint8)
    _, hdn1 = _parts(cfg, mdl, smp, mdl.host["layers"][0], ids0, m0)
    weights, _ = _scaled(mdl, "wu", _exponent(hdn1))

    geom = view_geom(cfg, smp.n_crops, "f16")
    bufs = [torch.empty((smp.sizes[l], cfg.d), dtype=torch.int16,
                        device="cuda") for l in range(cfg.K - 1)]
    ws = workspace(cfg, smp.sizes[-1] + len(smp.prompt) + L, 1, L, "f16")
    ws.fill_(0xAB)
    ids = torch.from_numpy(ids0.copy()).cuda()
    msk = torch.from_numpy(m0.copy()).cuda()
    ctr = torch.empty((T, L), device="cuda")
    atr = torch.empty((T, L), dtype=torch.int32, device="cuda")
    dv.davet_run_schedule(model_cfg(cfg, "f16"), weights, [geom], [smp.dev_v],
                          bufs, smp.dev_prompt, [0, len(smp.prompt)], L, T,
                          cfg.k, None, [LEVEL] * T, ids, msk, ws, ctr, atr)
    sched = dv.davet_fp16_overflow_count(ws)
    conf_tr, am_tr = ctr.cpu().numpy(), atr.cpu().numpy()
    # the state before step 2 from the traces: committed positions read -inf
    # (a masked row whose values overflowed may read NaN, still masked)
    live2 = conf_tr[1] != -np.inf
    ids1 = ids0.copy()
    ids1[~live2] = am_tr[0][~live2]
    c1, _ = _step(cfg, weights, smp, ids0, m0)
    c2, _ = _step(cfg, weights, smp, ids1, live2.astype(np.uint8))
    print("%s schedule overflow: steps %d + %d, schedule %d"
          % (kind, c1, c2, sched))
    assert c1 > 0 and c2 > 0 and sched == c1 + c2
