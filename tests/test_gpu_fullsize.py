"""GPU parity at the full workload sizes, in the launch configuration the
bench times (same packed batch, same kernels), on sampled outputs the oracle
computes one by one: the oracle runs the whole layer stack for the sampled
sequence (attention needs every position) but projects only sampled masked
rows on the vocabulary.  Teacher-forced; the bf16 model runs in the fp16
operand mode (its bf16 weights rounded to fp16, exact for |w| >= 2^-17) and
must reach logits rel-RMS <= 1e-2 against the oracle fed the model's own
bf16-rounded weights and encodings (so the conversion and the fp16 views sit
inside the measured error).
"""

import sys

import numpy as np
import pytest
import torch

import paper_2608_01821_amd as dv
import synth
from gpu_util import (TOL, Model, Sample, assert_conf_regrouped, check_decode,
                      model_cfg, oracle_step, random_state, rel_rms,
                      workspace)

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def gpu_step(cfg, mdl, samples, levels, ids, masked):
    n = len(samples)
    L = cfg.resp_len
    prompt = torch.cat([s.dev_prompt for s in samples])
    cu = np.concatenate([[0], np.cumsum([len(s.prompt) for s in samples])])
    views_ = [s.dev_levels[lv] for s, lv in zip(samples, levels)]
    nview = [s.sizes[lv] for s, lv in zip(samples, levels)]
    total = sum(nview) + int(cu[-1]) + n * L
    ws = workspace(cfg, total, n, L, mdl.mode)
    d_ids = torch.from_numpy(np.ascontiguousarray(ids, np.int32)).cuda()
    d_m = torch.from_numpy(np.ascontiguousarray(masked, np.uint8)).cuda()
    conf = torch.empty(n * L, device="cuda")
    am = torch.empty(n * L, dtype=torch.int32, device="cuda")
    logits = torch.full((n * L, cfg.vocab), 55.0, device="cuda")
    say("  gpu step: %d seqs, %d tokens" % (n, total))
    dv.davet_denoise_step(model_cfg(cfg, mdl.mode), mdl.weights, views_,
                          nview, prompt, cu, d_ids, d_m, L, conf, am, logits,
                          ws)
    torch.cuda.synchronize()
    return (conf.cpu().numpy().reshape(n, L), am.cpu().numpy().reshape(n, L),
            logits.reshape(n, L, cfg.vocab))


def check_sampled(cfg, mdl, sample, level, ids, masked, g_conf, g_am,
                  g_logits_dev, n_rows, seed):
    rng = np.random.default_rng(seed)
    mpos = np.nonzero(masked)[0]
    rows = np.sort(rng.choice(mpos, size=min(n_rows, len(mpos)),
                              replace=False))
    say("  oracle: level %d, %d tokens, rows %s" %
        (level, sample.sizes[level] + len(sample.prompt) + cfg.resp_len,
         rows.tolist()[:8]))
    pos, lg, am, cf = oracle_step(cfg, mdl, sample, level, ids, masked,
                                  rows=rows)
    g_lg = np.full((cfg.resp_len, cfg.vocab), np.nan, dtype=np.float32)
    g_lg[rows] = g_logits_dev[torch.from_numpy(rows).cuda()].cpu().numpy()
    # unmasked rows must be untouched (checked on device, cheaply)
    um = torch.from_numpy(np.nonzero(masked == 0)[0]).cuda()
    if len(um):
        assert bool((g_logits_dev[um] == 55.0).all())
    m = masked.astype(bool)
    assert np.all(g_conf[~m] == -np.inf) and np.all(g_am[~m] == -1)
    err = rel_rms(g_lg[pos], lg)
    tol = TOL[mdl.mode]
    assert err <= tol["logits"], ("logits rel-RMS", err)
    gap = 6.0 * err * float(np.sqrt(np.mean(lg ** 2)))
    check_decode(g_am[pos], g_conf[pos], lg, am, cf, cfg.mask_id, gap,
                 g_lg[pos])
    say("  rel-RMS %.3e" % err)
    return err


@pytest.fixture(scope="module", params=[2, 3])
def one_layer(request):
    cfg = synth.get_config(request.param)
    say("generating config %d" % cfg.cid)
    mdl = Model(cfg, oracle_values="model")
    s = synth.gen_sample(cfg)
    sample = Sample(cfg, s["n_crops"][0], s["visual"][0], s["prompts"][0],
                    oracle_values="model")
    return cfg, mdl, sample


@pytest.mark.parametrize("level,frac", [(0, 1.0), (2, 1.0), (1, 0.3)])
def test_one_layer_full_size(one_layer, level, frac):
    cfg, mdl, sample = one_layer
    rng = np.random.default_rng(level * 7 + int(frac * 10))
    ids, masked = random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab, frac)
    if frac == 1.0:
        ids[:] = cfg.mask_id
        masked[:] = 1
    g_conf, g_am, g_lg = gpu_step(cfg, mdl, [sample], [level], ids[None],
                                  masked[None])
    check_sampled(cfg, mdl, sample, level, ids, masked, g_conf[0], g_am[0],
                  g_lg[0], 12, level)


# Packed batches of copies of the workload's sample whose total token count
# lies in the GEMM planner's edge ranges (row counts just past a multiple of a
# tile height, which take a plan of their own instead of the nearest sample
# point's): config -> [(levels of the packed sequences, total tokens)].
EDGE_BATCHES = {
    2: [([1, 1, 0, 0, 0, 0], 1548),   # QKV 128x128, out/down 256x256 2 splits
        ([2, 2, 1], 2134),            # out 192x128, gate/up 192x128, down 3 splits
        ([1, 0, 0, 0], 983),          # gate/up 256x256 (4 x 4 waves)
        ([2, 2, 2, 2, 1, 0], 4121),   # down 256x256, 2 splits
        ([0, 0, 1], 774)],            # down 256x256, 4 splits
    3: [([1, 0], 1865),               # out 128x128 without a split
        ([1, 0, 0], 2430)],           # gate/up 256x256 (4 x 4 waves)
}


def test_edge_plans_full_size(one_layer):
    """The planner's edge-range plans in the packed step at the 8B shape: the
    last sequence of each batch against the oracle (each sequence's result
    depends on its own tokens only)."""
    cfg, mdl, sample = one_layer
    extra = len(sample.prompt) + cfg.resp_len
    for k, (levels, total) in enumerate(EDGE_BATCHES[cfg.cid]):
        assert sum(sample.sizes[lv] + extra for lv in levels) == total
        rng = np.random.default_rng(70 + k)
        st = [random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab, 0.8)
              for _ in levels]
        ids = np.stack([a for a, _ in st])
        masked = np.stack([m for _, m in st])
        g_conf, g_am, g_lg = gpu_step(cfg, mdl, [sample] * len(levels),
                                      levels, ids, masked)
        i = len(levels) - 1
        check_sampled(cfg, mdl, sample, levels[i], ids[i], masked[i],
                      g_conf[i], g_am[i], g_lg[i], 4, 200 + k)


def test_attention_split_matches_unsplit(one_layer):
    """The key-range split of attention at the 8B shape, against the same
    call with the split off (davet_set_attention_split(1)): logits of the
    masked rows within 1e-3 rel-RMS (only the fp32 summation order differs).
    A four-crop sequence of 24 full query tiles and a ragged one per head
    (3092 or 3188 tokens): automatically, the ragged tiles' keys split 8
    ways behind one full round of 768 workgroups.  The workload's own coarse
    view (356 or 1300 tokens) with every tile split 4 ways (forced)."""
    cfg, mdl, sample = one_layer
    c4 = synth.get_config(4)
    s4 = synth.gen_sample(c4)
    plen = 48 if cfg.resp_len == 128 else 16
    four = Sample(cfg, 4, s4["visual"][0], s4["prompts"][0][:plen],
                  oracle_values="model")
    rng = np.random.default_rng(8)
    ids, masked = random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab, 0.9)
    rows = torch.from_numpy(np.nonzero(masked)[0]).cuda()
    try:
        for smp, level, split in ((four, 2, 0), (sample, 0, 4)):
            dv.davet_set_attention_split(split)
            a = gpu_step(cfg, mdl, [smp], [level], ids[None], masked[None])
            dv.davet_set_attention_split(1)
            b = gpu_step(cfg, mdl, [smp], [level], ids[None], masked[None])
            err = rel_rms(a[2][0][rows].cpu().numpy(),
                          b[2][0][rows].cpu().numpy())
            say("  split %d vs unsplit, level %d: rel-RMS %.2e"
                % (split, level, err))
            assert err <= 1e-3
    finally:
        dv.davet_set_attention_split(0)


def test_ragged16_full_size():
    """The 16-sequence ragged batch in one packed call; four sequences are
    checked against the oracle, each on its own.  Then the same call with the
    tiled head (davet_pack_head, as the benchmark runs it: over ~1600 masked
    rows its 256 x 256 tile) gives the same argmaxes and logits bit for bit
    and the same confidences up to the regrouping of the softmax sum."""
    cfg = synth.get_config(5)
    say("generating config 5")
    mdl = Model(cfg, oracle_values="model")
    s = synth.gen_sample(cfg)
    samples = [Sample(cfg, c, v, p, oracle_values="model") for c, v, p in
               zip(s["n_crops"], s["visual"], s["prompts"])]
    rng = np.random.default_rng(55)
    levels = [int(x) for x in rng.integers(0, cfg.K, len(samples))]
    st = [random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab, 0.8)
          for _ in samples]
    ids = np.stack([a for a, _ in st])
    masked = np.stack([b for _, b in st])
    g_conf, g_am, g_lg = gpu_step(cfg, mdl, samples, levels, ids, masked)
    for i in (0, 5, 10, 15):
        check_sampled(cfg, mdl, samples[i], levels[i], ids[i], masked[i],
                      g_conf[i], g_am[i], g_lg[i], 6, 100 + i)
    tiled = torch.empty(dv.davet_head_tiled_elems(cfg.vocab, cfg.d),
                        dtype=torch.int16, device="cuda")
    dv.davet_pack_head(mdl.dev_head, tiled, cfg.vocab, cfg.d,
                       dv.DAVET_F16 if mdl.mode == "f16" else dv.DAVET_BF16)
    row_w = mdl.weights
    mdl.weights = dv.Weights(mdl.dev_embed, tiled, mdl.dev_layers,
                             head_layout=dv.DAVET_HEAD_TILED)
    try:
        t_conf, t_am, t_lg = gpu_step(cfg, mdl, samples, levels, ids, masked)
    finally:
        mdl.weights = row_w
    assert np.array_equal(t_am, g_am)
    assert_conf_regrouped(t_conf, g_conf)
    assert bool(torch.equal(t_lg, g_lg))


@pytest.fixture(scope="module")
def stack32():
    """The 32-layer 8B-shaped stack on the device (fp16 operands, ~16 GB),
    built once for the three view levels; the oracle regenerates each
    layer's bf16 weights as it reaches it."""
    cfg = synth.get_config(4)
    say("generating config 4 (32 layers)")
    mdl = Model(cfg, stream_host=True, oracle_values="model")
    gen = mdl.host["layers"]

    def layer_with_progress(i):
        if i % 4 == 0:
            say("  oracle layer %d / %d" % (i, cfg.n_layers))
        return gen(i)
    mdl.host["layers"] = layer_with_progress
    s = synth.gen_sample(cfg)
    sample = Sample(cfg, s["n_crops"][0], s["visual"][0], s["prompts"][0],
                    oracle_values="model")
    return cfg, mdl, sample


@pytest.mark.timeout(600)
@pytest.mark.parametrize("level", [0, 1, 2])
def test_stack32_full_size(stack32, level):
    """The 32-layer 8B-shaped stack at each view level (372, 960 and 3092
    tokens): the first step of the loop (all positions masked) at the coarse
    view, a partly committed answer at the middle and full views.  The error
    of 32 layers of 16-bit operands stays inside the tolerance at the
    longest sequence, where the projections run their 256 x 256 tiles
    without a K split."""
    cfg, mdl, sample = stack32
    rng = np.random.default_rng(40 + level)
    if level == 0:
        ids = np.full(cfg.resp_len, cfg.mask_id, np.int32)
        masked = np.ones(cfg.resp_len, np.uint8)
    else:
        ids, masked = random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab,
                                   0.5 if level == 1 else 0.9)
    g_conf, g_am, g_lg = gpu_step(cfg, mdl, [sample], [level], ids[None],
                                  masked[None])
    check_sampled(cfg, mdl, sample, level, ids, masked, g_conf[0], g_am[0],
                  g_lg[0], 8, 4 + level)


def test_tiled_head_full_size_bit_identical(one_layer):
    """The tiled vocabulary head (davet_pack_head) gives the very same
    argmaxes and logits as the row-major head at full size, and the same
    confidences up to the regrouping of the softmax sum (256- against
    128-column vocabulary slabs)."""
    cfg, mdl, sample = one_layer
    n = dv.davet_head_tiled_elems(cfg.vocab, cfg.d)
    tiled = torch.empty(n, dtype=torch.int16, device="cuda")
    dv.davet_pack_head(mdl.dev_head, tiled, cfg.vocab, cfg.d,
                       dv.DAVET_F16 if mdl.mode == "f16" else dv.DAVET_BF16)
    row_w = mdl.weights
    mdl.weights = dv.Weights(mdl.dev_embed, tiled, mdl.dev_layers,
                             head_layout=dv.DAVET_HEAD_TILED)
    try:
        rng = np.random.default_rng(3)
        ids, masked = random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab,
                                   0.7)
        t_conf, t_am, t_lg = gpu_step(cfg, mdl, [sample], [1], ids[None],
                                      masked[None])
    finally:
        mdl.weights = row_w
    r_conf, r_am, r_lg = gpu_step(cfg, mdl, [sample], [1], ids[None],
                                  masked[None])
    assert np.array_equal(t_am, r_am)
    assert_conf_regrouped(t_conf, r_conf)
    assert bool(torch.equal(t_lg, r_lg))
