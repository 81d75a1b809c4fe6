"""GPU parity of one denoising step (Sec. 3.1, Eq. 1 + decoding) against the
oracle, teacher-forced: both sides get the same weights, encoding, prompt,
partially denoised answer and view level, and are compared per call.

Tolerances: fp32 path logits rel-RMS <= 1e-5; bf16 path <= 1e-2 against the
oracle fed the same bf16 values (the kernels also round activations to bf16
at every matrix-core operand, which the float64 oracle does not).
"""

import numpy as np
import pytest
import torch

import paper_2608_01821_amd as dv
import synth
from gpu_util import (TOL, Model, Sample, compare, oracle_step, random_state,
                      rel_rms,
                      run_gpu_step)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", params=[(1, "f32"), (11, "f16"),
                                        (11, "bf16")])
def small(request):
    cid, mode = request.param
    cfg = synth.get_any_config(cid)
    mdl = Model(cfg, mode)
    s = synth.gen_sample(cfg)
    sample = Sample(cfg, s["n_crops"][0], s["visual"][0], s["prompts"][0],
                    mode)
    return cfg, mdl, sample


@pytest.mark.parametrize("level", [0, 1, 2])
@pytest.mark.parametrize("frac", [1.0, 0.5, 0.05])
def test_step_teacher_forced_small(small, level, frac):
    cfg, mdl, sample = small
    rng = np.random.default_rng(int(frac * 100) + 10 * level)
    ids, masked = random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab, frac)
    g_conf, g_am, g_lg = run_gpu_step(cfg, mdl, [sample], [level], ids, masked)
    pos, lg, am, cf = oracle_step(cfg, mdl, sample, level, ids, masked)
    compare(cfg, TOL[mdl.mode], masked, g_conf[0], g_am[0], g_lg[0], pos, lg,
            am, cf)


def test_step_deterministic(small):
    cfg, mdl, sample = small
    rng = np.random.default_rng(5)
    ids, masked = random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab, 0.6)
    a = run_gpu_step(cfg, mdl, [sample], [2], ids, masked)
    b = run_gpu_step(cfg, mdl, [sample], [2], ids, masked)
    for x, y in zip(a, b):
        assert np.array_equal(x, y, equal_nan=True)


@pytest.mark.parametrize("cid,mode,split", [(12, "f16", 0), (12, "bf16", 0),
                                            (13, "f32", 0), (12, "f16", 3),
                                            (12, "bf16", 8)])
def test_ragged_batch_step(cid, mode, split):
    """Packed batch of sequences with different view levels and prompt
    lengths in one call; each sequence must equal its own oracle run (the
    attention of one sequence never sees another's tokens).  Also with the
    keys of every query tile split 3 or 8 ways (forced), so that pieces and
    their merge map onto the right sequence and tile across a ragged batch,
    including empty pieces of short sequences."""
    if split:
        dv.davet_set_attention_split(split)
    try:
        _ragged_batch_step(cid, mode)
    finally:
        dv.davet_set_attention_split(0)


def _ragged_batch_step(cid, mode):
    cfg = synth.get_any_config(cid)
    mdl = Model(cfg, mode)
    s = synth.gen_sample(cfg)
    samples = [Sample(cfg, c, v, p, mode) for c, v, p in
               zip(s["n_crops"], s["visual"], s["prompts"])]
    rng = np.random.default_rng(cid)
    levels = [int(x) for x in rng.integers(0, cfg.K, len(samples))]
    ids, masked = zip(*[random_state(rng, cfg.resp_len, cfg.mask_id,
                                     cfg.vocab, 0.6) for _ in samples])
    ids, masked = np.stack(ids), np.stack(masked)
    g_conf, g_am, g_lg = run_gpu_step(cfg, mdl, samples, levels, ids, masked)
    for i, smp in enumerate(samples):
        pos, lg, am, cf = oracle_step(cfg, mdl, smp, levels[i], ids[i],
                                      masked[i])
        compare(cfg, TOL[mode], masked[i], g_conf[i], g_am[i], g_lg[i],
                pos, lg, am, cf)


@pytest.mark.parametrize("cid,mode", [(11, "f16"), (11, "bf16"), (1, "f32")])
def test_step_without_layers(cid, mode):
    """No transformer layers: the step is the final norm of the embedded
    masked rows and the vocabulary head, so the final norm and gather run on
    their own (there is no last-layer split-K reduction to carry them)."""
    import dataclasses
    cfg = dataclasses.replace(synth.get_any_config(cid), n_layers=0)
    mdl = Model(cfg, mode)
    s = synth.gen_sample(cfg)
    sample = Sample(cfg, s["n_crops"][0], s["visual"][0], s["prompts"][0],
                    mode)
    rng = np.random.default_rng(21)
    ids, masked = random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab, 0.6)
    g_conf, g_am, g_lg = run_gpu_step(cfg, mdl, [sample], [1], ids, masked)
    pos, lg, am, cf = oracle_step(cfg, mdl, sample, 1, ids, masked)
    compare(cfg, TOL[mdl.mode], masked, g_conf[0], g_am[0], g_lg[0], pos, lg,
            am, cf)


@pytest.mark.parametrize("split", [0, 4])
def test_step_edge_inputs(split):
    """Edge inputs in one packed call: a sequence with neither view tokens
    nor prompt (only its response), one with a view but no prompt, one with
    every position already committed (conf -inf, argmax -1, logit rows
    untouched), next to an ordinary one; each against its own oracle run.
    Also with attention's keys split 4 ways (forced)."""
    if split:
        dv.davet_set_attention_split(split)
    try:
        _step_edge_inputs()
    finally:
        dv.davet_set_attention_split(0)


def _step_edge_inputs():
    import copy
    cfg = synth.get_any_config(12)
    mdl = Model(cfg)
    s = synth.gen_sample(cfg)
    base = [Sample(cfg, s["n_crops"][i], s["visual"][i], s["prompts"][i])
            for i in range(4)]
    L = cfg.resp_len
    empty_prompt = np.zeros(0, np.int32)

    def without(smp, view=False, prompt=False):
        x = copy.copy(smp)
        if view:
            x.sizes = [0] + list(smp.sizes[1:])
            x.dev_levels = [smp.dev_levels[0][:0]] + list(smp.dev_levels[1:])
            x.ref_levels = [smp.ref_levels[0][:0]] + list(smp.ref_levels[1:])
        if prompt:
            x.prompt = empty_prompt
            x.dev_prompt = torch.from_numpy(empty_prompt).cuda()
        return x
    samples = [without(base[0], view=True, prompt=True),
               without(base[1], prompt=True), base[2], base[3]]
    levels = [0, 1, 2, 0]
    rng = np.random.default_rng(77)
    st = [random_state(rng, L, cfg.mask_id, cfg.vocab, 0.7) for _ in range(4)]
    ids = np.stack([a for a, _ in st])
    masked = np.stack([b for _, b in st])
    masked[2] = 0                              # nothing left to denoise
    ids[2] = rng.integers(0, cfg.vocab - 1, L)
    g_conf, g_am, g_lg = run_gpu_step(cfg, mdl, samples, levels, ids, masked)
    assert np.all(g_conf[2] == -np.inf) and np.all(g_am[2] == -1)
    assert np.all(g_lg[2] == 55.0)
    for i in (0, 1, 3):
        pos, lg, am, cf = oracle_step(cfg, mdl, samples[i], levels[i], ids[i],
                                      masked[i])
        compare(cfg, TOL[mdl.mode], masked[i], g_conf[i], g_am[i], g_lg[i],
                pos, lg, am, cf)


SPLIT_RTOL = {"f16": 1e-3, "bf16": 1e-2}


@pytest.mark.parametrize("mode", ["f16", "bf16"])
def test_key_split_attention(mode):
    """Attention with every query tile's keys split among 2, 3 or 8
    workgroups (davet_set_attention_split), merged by the merge kernel.  One
    27x27 crop: 779 tokens at the full view (13 key tiles: pieces of 7, 5
    and 2 tiles), 246 at the middle one (4 key tiles: with 8 pieces half of
    them are empty).  Each run matches the oracle, and its logits stay close
    to the unsplit launch's: only the fp32 summation order of the attention
    differs, which moves the 16-bit rounding of some attention outputs by one
    unit (fp16 2^-11, bf16 2^-8 relative), so rel-RMS within 1e-3 (fp16) or
    1e-2 (bf16)."""
    import dataclasses
    cfg = dataclasses.replace(synth.get_any_config(11), n_layers=1, grid=27,
                              n_crops=1)
    mdl = Model(cfg, mode)
    s = synth.gen_sample(cfg)
    sample = Sample(cfg, s["n_crops"][0], s["visual"][0], s["prompts"][0],
                    mode)
    rng = np.random.default_rng(31)
    ids, masked = random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab, 0.8)
    m = masked.astype(bool)
    try:
        for level in (2, 1):
            pos, lg, am, cf = oracle_step(cfg, mdl, sample, level, ids, masked)
            dv.davet_set_attention_split(1)
            _, _, u_lg = run_gpu_step(cfg, mdl, [sample], [level], ids, masked)
            for split in (2, 3, 8):
                dv.davet_set_attention_split(split)
                g_conf, g_am, g_lg = run_gpu_step(cfg, mdl, [sample], [level],
                                                  ids, masked)
                compare(cfg, TOL[mode], masked, g_conf[0], g_am[0], g_lg[0],
                        pos, lg, am, cf)
                assert rel_rms(g_lg[0][m], u_lg[0][m]) <= SPLIT_RTOL[mode]
    finally:
        dv.davet_set_attention_split(0)
