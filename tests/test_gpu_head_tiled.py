"""The tiled vocabulary-head layout: the packing kernel against its defining
index formula (written out in numpy), and a denoising step with the tiled
head against the row-major one (logits and argmaxes bit-identical,
confidences up to the regrouping of the softmax sum) and against the
oracle."""

import numpy as np
import pytest
import torch

import paper_2608_01821_amd as dv
import synth
from gpu_util import (TOL, Model, Sample, assert_conf_regrouped, compare,
                      model_cfg, oracle_step, random_state, workspace)

pytestmark = pytest.mark.gpu


def _tiled_reference(head, vocab, d):
    """tiled[((c*S + s)*128 + r)*64 + j] = head[(128 s + r)*d + 64 c + j],
    zero past the vocabulary."""
    S = -(-vocab // 128)
    pad = np.zeros((S * 128, d), head.dtype)
    pad[:vocab] = head
    t = pad.reshape(S, 128, d // 64, 64).transpose(2, 0, 1, 3)
    return np.ascontiguousarray(t).reshape(-1)


@pytest.mark.parametrize("vocab,d", [(1000, 256), (128, 64), (1, 128),
                                     (126464, 4096)])
def test_pack_head_matches_formula(vocab, d):
    rng = np.random.default_rng(vocab + d)
    head = rng.integers(-2 ** 15, 2 ** 15, (vocab, d), dtype=np.int16)
    src = torch.from_numpy(head).cuda()
    n = dv.davet_head_tiled_elems(vocab, d)
    assert n == -(-vocab // 128) * 128 * d
    dst = torch.full((n,), 77, dtype=torch.int16, device="cuda")
    dv.davet_pack_head(src, dst, vocab, d, dv.DAVET_F16)
    torch.cuda.synchronize()
    exp = _tiled_reference(head, vocab, d)
    assert np.array_equal(dst.cpu().numpy(), exp)


# (config, sequences, response length, masked fraction): the last three pack
# 200, 300 and 500 response rows, so the head runs its 256 x 256 tile over one
# and two row slots and its 128 x 256 tile over three
@pytest.mark.parametrize("cid,n_seqs,L,frac,mode", [
    (11, 3, None, 0.6, "f16"), (12, 3, None, 0.6, "f16"),
    (12, 5, 40, 1.0, "f16"), (12, 6, 50, 0.9, "f16"),
    (12, 5, 100, 0.8, "f16"), (12, 5, 100, 0.8, "bf16")])
def test_tiled_head_step(cid, n_seqs, L, frac, mode):
    import dataclasses
    cfg = synth.get_any_config(cid)
    if L is not None:
        cfg = dataclasses.replace(cfg, resp_len=L, n_seqs=n_seqs)
    mdl = Model(cfg, mode)
    s = synth.gen_sample(cfg)
    n_seqs = min(cfg.n_seqs, n_seqs)
    samples = [Sample(cfg, s["n_crops"][i], s["visual"][i], s["prompts"][i],
                      mode) for i in range(n_seqs)]
    tiled = torch.empty(dv.davet_head_tiled_elems(cfg.vocab, cfg.d),
                        dtype=torch.int16, device="cuda")
    dv.davet_pack_head(mdl.dev_head, tiled, cfg.vocab, cfg.d,
                       dv.DAVET_F16 if mode == "f16" else dv.DAVET_BF16)
    w_tiled = dv.Weights(mdl.dev_embed, tiled, mdl.dev_layers,
                         head_layout=dv.DAVET_HEAD_TILED)
    rng = np.random.default_rng(cid)
    st = [random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab, frac)
          for _ in samples]
    ids = np.stack([a for a, _ in st])
    masked = np.stack([b for _, b in st])
    levels = [i % cfg.K for i in range(n_seqs)]
    L = cfg.resp_len
    prompt = torch.cat([x.dev_prompt for x in samples])
    cu = np.concatenate([[0], np.cumsum([len(x.prompt) for x in samples])])
    views_ = [x.dev_levels[lv] for x, lv in zip(samples, levels)]
    nview = [x.sizes[lv] for x, lv in zip(samples, levels)]
    total = sum(nview) + int(cu[-1]) + n_seqs * L
    outs = []
    for w in (mdl.weights, w_tiled):
        ws = workspace(cfg, total, n_seqs, L, mode)
        d_ids = torch.from_numpy(ids.astype(np.int32)).cuda()
        d_m = torch.from_numpy(masked.astype(np.uint8)).cuda()
        conf = torch.empty(n_seqs * L, device="cuda")
        am = torch.empty(n_seqs * L, dtype=torch.int32, device="cuda")
        lg = torch.full((n_seqs * L, cfg.vocab), 55.0, device="cuda")
        dv.davet_denoise_step(model_cfg(cfg, mode), w, views_, nview, prompt,
                              cu, d_ids, d_m, L, conf, am, lg, ws)
        torch.cuda.synchronize()
        outs.append((conf.cpu().numpy(), am.cpu().numpy(), lg.cpu().numpy()))
    (c0, a0, l0), (c1, a1, l1) = outs
    assert np.array_equal(a0, a1)
    assert_conf_regrouped(c1, c0)
    assert np.array_equal(l0.view(np.uint32), l1.view(np.uint32))
    # and the tiled run against the oracle, sequence by sequence
    for i in range(n_seqs):
        pos, rl, ra, rc = oracle_step(cfg, mdl, samples[i], levels[i], ids[i],
                                      masked[i])
        sl = slice(i * L, (i + 1) * L)
        compare(cfg, TOL[mdl.mode], masked[i], c1[sl], a1[sl],
                l1[sl].reshape(L, cfg.vocab), pos, rl, ra, rc)


def test_tiled_head_rejected_for_fp32():
    cfg = synth.get_any_config(13)
    mdl = Model(cfg)
    w = dv.Weights(mdl.dev_embed, mdl.dev_head, mdl.dev_layers,
                   head_layout=dv.DAVET_HEAD_TILED)
    s = synth.gen_sample(cfg)
    smp = Sample(cfg, s["n_crops"][0], s["visual"][0], s["prompts"][0])
    L = cfg.resp_len
    ws = workspace(cfg, smp.sizes[-1] + len(smp.prompt) + L, 1, L)
    d_ids = torch.full((L,), cfg.mask_id, dtype=torch.int32, device="cuda")
    d_m = torch.ones(L, dtype=torch.uint8, device="cuda")
    conf = torch.empty(L, device="cuda")
    am = torch.empty(L, dtype=torch.int32, device="cuda")
    with pytest.raises(dv.DavetError):
        dv.davet_denoise_step(model_cfg(cfg), w, [smp.dev_levels[-1]],
                              [smp.sizes[-1]], smp.dev_prompt,
                              [0, len(smp.prompt)], d_ids, d_m, L, conf, am,
                              None, ws)


@pytest.mark.parametrize("n_seqs,L", [(64, 16), (1, 1024), (64, 1024)])
def test_step_at_maximum_shapes(n_seqs, L):
    """The packed step at the limits the C ABI accepts (64 sequences, 1024
    response positions each, 65536 response rows at most): the first, a
    middle and the last sequence against the oracle, and the tiled head
    (256 x 256 tiles over up to 256 row slots) against the row-major one."""
    import dataclasses
    cfg = dataclasses.replace(synth.get_any_config(12), resp_len=L,
                              n_seqs=n_seqs)
    mdl = Model(cfg)
    s = synth.gen_sample(cfg)
    samples = [Sample(cfg, s["n_crops"][i], s["visual"][i], s["prompts"][i])
               for i in range(n_seqs)]
    tiled = torch.empty(dv.davet_head_tiled_elems(cfg.vocab, cfg.d),
                        dtype=torch.int16, device="cuda")
    dv.davet_pack_head(mdl.dev_head, tiled, cfg.vocab, cfg.d, dv.DAVET_F16)
    w_tiled = dv.Weights(mdl.dev_embed, tiled, mdl.dev_layers,
                         head_layout=dv.DAVET_HEAD_TILED)
    rng = np.random.default_rng(n_seqs + L)
    st = [random_state(rng, L, cfg.mask_id, cfg.vocab, 0.9) for _ in samples]
    ids = np.stack([a for a, _ in st])
    masked = np.stack([b for _, b in st])
    levels = [i % cfg.K for i in range(n_seqs)]
    prompt = torch.cat([x.dev_prompt for x in samples])
    cu = np.concatenate([[0], np.cumsum([len(x.prompt) for x in samples])])
    views_ = [x.dev_levels[lv] for x, lv in zip(samples, levels)]
    nview = [x.sizes[lv] for x, lv in zip(samples, levels)]
    total = sum(nview) + int(cu[-1]) + n_seqs * L
    ws = workspace(cfg, total, n_seqs, L)
    outs = []
    for w in (mdl.weights, w_tiled):
        d_ids = torch.from_numpy(ids.astype(np.int32)).cuda()
        d_m = torch.from_numpy(masked.astype(np.uint8)).cuda()
        conf = torch.empty(n_seqs * L, device="cuda")
        am = torch.empty(n_seqs * L, dtype=torch.int32, device="cuda")
        lg = torch.full((n_seqs * L, cfg.vocab), 55.0, device="cuda")
        dv.davet_denoise_step(model_cfg(cfg), w, views_, nview, prompt, cu,
                              d_ids, d_m, L, conf, am, lg, ws)
        torch.cuda.synchronize()
        outs.append((conf.cpu().numpy(), am.cpu().numpy(), lg))
    (c0, a0, l0), (c1, a1, l1) = outs
    assert np.array_equal(a0, a1)
    assert_conf_regrouped(c1, c0)
    assert bool(torch.equal(l0, l1))
    l0 = l0.cpu().numpy()
    for i in sorted({0, n_seqs // 2, n_seqs - 1}):
        pos, rl, ra, rc = oracle_step(cfg, mdl, samples[i], levels[i], ids[i],
                                      masked[i])
        sl = slice(i * L, (i + 1) * L)
        compare(cfg, TOL[mdl.mode], masked[i], c0[sl], a0[sl],
                l0[sl].reshape(L, cfg.vocab), pos, rl, ra, rc)
