"""The pruning and merging realizers on the GPU (Sec. 4.3, "Compatible
evidence realizers") against the oracle.

Three layers, as for the commitment kernel: the keys (L1 saliency, bit-exact
for fp16 encodings where float64 sums of fp16 values are exact; cosine
similarities to 1e-12), the decisions on identical seeded keys (index maps
bit-exact, ties, NaN and signed zeros included), and the whole build (maps
bit-exact, level rows bit-exact) on seeded encodings whose deciding key gaps
are checked to lie far outside the keys' tolerance, so the exact answer is
unique.  A denoising step on each realizer's levels and the schedule loop
building them from its own workspace close the path."""

import numpy as np
import pytest
import torch

import paper_2608_01821_amd as dv
import synth
from oracle import realizers as R
from gpu_util import (DTYPE, TOL, Model, Sample, compare, model_cfg,
                      oracle_step, random_state, run_gpu_step, to_mode,
                      view_geom, workspace)

pytestmark = pytest.mark.gpu

RZ = {"prune": dv.DAVET_REALIZER_PRUNE, "merge": dv.DAVET_REALIZER_MERGE}
KEY_TOL = 1e-12


def _encoding(rng, C, G, d, dtype):
    v = rng.standard_normal((C * G * G, d)).astype(np.float32)
    if dtype == "bf16":
        v = synth.round_to_bf16(v)
    return to_mode(v, dtype)


def _levels_to_f32(t, dtype):
    a = t.cpu().numpy()
    if dtype == "bf16":
        return synth.bf16_bits_to_f32(a.view(np.uint16))
    if dtype == "f16":
        return a.view(np.float16).astype(np.float32)
    return a


def _alloc_maps(geom, C, G):
    K = geom.K
    sizes = dv.davet_view_sizes(geom)
    msz = dv.davet_view_map_sizes(geom)
    offs = [torch.full((sizes[l] + 1,), -1, dtype=torch.int32, device="cuda")
            for l in range(K)]
    mems = [torch.full((msz[l],), -1, dtype=torch.int32, device="cuda")
            for l in range(K)]
    return offs, mems


KEY_CASES = [
    ("f32", 1, 12, 256),
    ("f16", 1, 27, 4096),         # one 27x27 crop of the 8B-shaped encoding
    ("bf16", 5, 27, 4096),        # five crops
    ("f16", 2, 7, 64),
    ("bf16", 3, 5, 16),
    ("f32", 1, 1, 8),             # one token: no edge
    ("f16", 1, 64, 64),           # the largest grid
]


@pytest.mark.parametrize("name", ["prune", "merge"])
@pytest.mark.parametrize("dtype,C,G,d", KEY_CASES)
def test_keys_match_oracle(name, dtype, C, G, d):
    rng = np.random.default_rng(7 * G + C + d)
    dev, host = _encoding(rng, C, G, d, dtype)
    geom = dv.ViewGeom(C, G, d, 3, DTYPE[dtype], 0, RZ[name])
    n = dv.davet_realizer_key_count(geom)
    ref = R.keys(host, C, G, RZ[name])
    assert n == len(ref)
    keys = torch.full((max(n, 1),), np.nan, dtype=torch.float64, device="cuda")
    dv.davet_realizer_keys(geom, torch.from_numpy(dev).cuda(), keys)
    torch.cuda.synchronize()
    got = keys.cpu().numpy()[:n]
    if name == "prune":
        if dtype == "f16":
            assert np.array_equal(got, ref)       # exact float64 sums
        else:
            np.testing.assert_allclose(got, ref, rtol=KEY_TOL, atol=0)
    else:
        np.testing.assert_allclose(got, ref, rtol=0, atol=KEY_TOL)


def _seeded_keys(rng, n):
    """Keys with many exact ties, NaN, +-inf and signed zeros."""
    special = np.array([0.0, -0.0, 0.5, 0.5, np.nan, np.inf, -np.inf, -0.25])
    k = rng.standard_normal(n)
    pick = rng.random(n) < 0.4
    k[pick] = rng.choice(special, pick.sum())
    return k


MAP_CASES = [(1, 27, 3), (5, 27, 3), (2, 7, 4), (3, 5, 2), (1, 1, 3),
             (2, 13, 1), (1, 64, 4), (2, 64, 3), (4, 2, 3)]


@pytest.mark.parametrize("name", ["prune", "merge"])
@pytest.mark.parametrize("C,G,K", MAP_CASES)
def test_maps_from_given_keys_bit_exact(name, C, G, K):
    rng = np.random.default_rng(1000 + 31 * G + 7 * C + K)
    geom = dv.ViewGeom(C, G, 8, K, dv.DAVET_F32, 0, RZ[name])
    n = dv.davet_realizer_key_count(geom)
    keys = _seeded_keys(rng, n)
    dk = torch.from_numpy(keys if n else np.zeros(1)).cuda()
    offs, mems = _alloc_maps(geom, C, G)
    dv.davet_realizer_maps(geom, dk, offs, mems)
    torch.cuda.synchronize()
    ref = R.index_maps(keys, C, G, K, RZ[name])
    for l in range(K):
        assert np.array_equal(offs[l].cpu().numpy(), ref[l][0]), (l, "offsets")
        assert np.array_equal(mems[l].cpu().numpy(), ref[l][1]), (l, "members")


def test_maps_skip_null_levels():
    # a NULL entry leaves that level's buffers untouched
    C, G, K = 2, 9, 3
    rng = np.random.default_rng(5)
    for name in ("prune", "merge"):
        geom = dv.ViewGeom(C, G, 8, K, dv.DAVET_F32, 0, RZ[name])
        keys = torch.from_numpy(rng.standard_normal(
            dv.davet_realizer_key_count(geom))).cuda()
        offs, mems = _alloc_maps(geom, C, G)
        dv.davet_realizer_maps(geom, keys, [offs[0], None, offs[2]],
                               [None, mems[1], mems[2]])
        torch.cuda.synchronize()
        assert torch.all(offs[1] == -1) and torch.all(mems[0] == -1)
        ref = R.index_maps(keys.cpu().numpy(), C, G, K, RZ[name])
        assert np.array_equal(offs[0].cpu().numpy(), ref[0][0])
        assert np.array_equal(mems[1].cpu().numpy(), ref[1][1])


def _decisions_are_unique(keys, C, G, K, name):
    """True when every decision the oracle takes from ``keys`` is separated
    by more than the keys' tolerance, so keys within it decide the same."""
    counts = R.level_counts(G, K)
    if name == "prune":
        N = G * G
        for c in range(C):
            k = np.sort(keys[c * N:(c + 1) * N])[::-1]
            for n in counts[:-1]:
                if n < N and abs(k[n - 1] - k[n]) <= 10 * KEY_TOL * max(
                        1.0, abs(k[n])):
                    return False
        return True
    E = 2 * G * (G - 1)
    for c in range(C):
        k = np.sort(keys[c * E:(c + 1) * E])
        if E > 1 and np.min(np.diff(k)) <= 10 * KEY_TOL:
            return False
    return True


VIEW_CASES = [
    ("f32", 1, 12, 3, 256),
    ("f16", 1, 27, 3, 4096),
    ("bf16", 5, 27, 3, 4096),
    ("f16", 4, 27, 3, 4096),
    ("f32", 2, 7, 4, 64),
    ("bf16", 3, 5, 2, 16),
    ("f32", 1, 1, 3, 8),
    ("bf16", 2, 13, 1, 24),
    ("f16", 1, 64, 3, 64),
]


@pytest.mark.parametrize("name", ["prune", "merge"])
@pytest.mark.parametrize("dtype,C,G,K,d", VIEW_CASES)
def test_views_match_oracle(name, dtype, C, G, K, d):
    rng = np.random.default_rng(300 + 11 * G + C + K + d)
    dev, host = _encoding(rng, C, G, d, dtype)
    geom = dv.ViewGeom(C, G, d, K, DTYPE[dtype], 0, RZ[name])
    ref_keys = R.keys(host, C, G, RZ[name])
    assert _decisions_are_unique(ref_keys, C, G, K, name)
    sizes = dv.davet_view_sizes(geom)
    tdt = torch.float32 if dtype == "f32" else torch.int16
    levels = [torch.full((sizes[l], d), -7, dtype=tdt, device="cuda")
              for l in range(K - 1)]
    offs, mems = _alloc_maps(geom, C, G)
    scratch = torch.empty(max(1, dv.davet_views_scratch_bytes(geom)),
                          dtype=torch.uint8, device="cuda")
    dv.davet_build_views(geom, torch.from_numpy(dev).cuda(), levels, offs,
                         mems, scratch=scratch)
    torch.cuda.synchronize()
    ref_levels, ref_maps = R.build_views(host, C, G, K, RZ[name], dtype)
    for l in range(K):
        assert np.array_equal(offs[l].cpu().numpy(), ref_maps[l][0])
        assert np.array_equal(mems[l].cpu().numpy(), ref_maps[l][1])
    for l in range(K - 1):
        got = _levels_to_f32(levels[l], dtype)
        ref = ref_levels[l]
        if dtype == "f32":
            rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
            assert rel <= 1e-6
        assert np.array_equal(got, ref)   # same float64 sums, same order


def test_prune_ties_end_to_end():
    # repeated tokens: equal L1 norms (exact for fp16), kept by lower index
    C, G, K, d = 2, 9, 3, 64
    rng = np.random.default_rng(12)
    base = rng.standard_normal((5, d)).astype(np.float32)
    v = base[rng.integers(0, 5, C * G * G)]
    dev, host = to_mode(v, "f16")
    geom = dv.ViewGeom(C, G, d, K, dv.DAVET_F16, 0, dv.DAVET_REALIZER_PRUNE)
    sizes = dv.davet_view_sizes(geom)
    levels = [torch.empty((sizes[l], d), dtype=torch.int16, device="cuda")
              for l in range(K - 1)]
    offs, mems = _alloc_maps(geom, C, G)
    dv.davet_build_views(geom, torch.from_numpy(dev).cuda(), levels, offs,
                         mems)
    torch.cuda.synchronize()
    ref_levels, ref_maps = R.build_views(host, C, G, K, R.PRUNE, "f16")
    for l in range(K):
        assert np.array_equal(mems[l].cpu().numpy(), ref_maps[l][1])
    for l in range(K - 1):
        assert np.array_equal(_levels_to_f32(levels[l], "f16"), ref_levels[l])


def test_scratch_reuse_and_smaller_second_call():
    # the same scratch serves a large and then a smaller geometry
    rng = np.random.default_rng(21)
    scratch = None
    for C, G in ((3, 27), (1, 6)):
        dev, host = _encoding(rng, C, G, 128, "f16")
        geom = dv.ViewGeom(C, G, 128, 3, dv.DAVET_F16, 0,
                           dv.DAVET_REALIZER_MERGE)
        if scratch is None:
            scratch = torch.empty(dv.davet_views_scratch_bytes(geom),
                                  dtype=torch.uint8, device="cuda")
        sizes = dv.davet_view_sizes(geom)
        levels = [torch.empty((sizes[l], 128), dtype=torch.int16,
                              device="cuda") for l in range(2)]
        dv.davet_build_views(geom, torch.from_numpy(dev).cuda(), levels,
                             scratch=scratch)
        torch.cuda.synchronize()
        ref_levels, _ = R.build_views(host, C, G, 3, R.MERGE, "f16")
        for l in range(2):
            assert np.array_equal(_levels_to_f32(levels[l], "f16"),
                                  ref_levels[l])


@pytest.mark.parametrize("name", ["prune", "merge"])
@pytest.mark.parametrize("cid", [11, 12])
def test_step_on_realizer_views(name, cid):
    """Teacher-forced denoising steps on the realizer's levels 0 and 1 match
    the oracle fed the oracle's own levels."""
    cfg = synth.get_any_config(cid)
    mdl = Model(cfg)
    s = synth.gen_sample(cfg)
    n = min(cfg.n_seqs, 3)
    samples = [Sample(cfg, s["n_crops"][i], s["visual"][i], s["prompts"][i],
                      realizer=RZ[name]) for i in range(n)]
    rng = np.random.default_rng(60 + cid)
    st = [random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab, 0.7)
          for _ in samples]
    ids = np.stack([a for a, _ in st])
    masked = np.stack([b for _, b in st])
    levels = [i % 2 for i in range(n)]
    g_conf, g_am, g_lg = run_gpu_step(cfg, mdl, samples, levels, ids, masked)
    for i in range(n):
        pos, rl, ra, rc = oracle_step(cfg, mdl, samples[i], levels[i], ids[i],
                                      masked[i])
        compare(cfg, TOL[mdl.mode], masked[i], g_conf[i], g_am[i], g_lg[i],
                pos, rl, ra, rc)


@pytest.mark.parametrize("name", ["prune", "merge"])
def test_run_schedule_builds_realizer_views(name):
    """davet_run_schedule builds prune / merge levels in its own workspace;
    the level buffers it leaves match the oracle's levels."""
    cfg = synth.get_any_config(12)
    mdl = Model(cfg)
    s = synth.gen_sample(cfg)
    n, L, T, mode = cfg.n_seqs, cfg.resp_len, 2, mdl.mode
    geoms = [view_geom(cfg, c, mode, realizer=RZ[name]) for c in s["n_crops"]]
    sizes = [dv.davet_view_sizes(g) for g in geoms]
    tdt = torch.float32 if mode == "f32" else torch.int16
    visual = [torch.from_numpy(to_mode(v, mode)[0]).cuda() for v in s["visual"]]
    bufs = [torch.full((sz[l], cfg.d), -7, dtype=tdt, device="cuda")
            for sz in sizes for l in range(cfg.K - 1)]
    prompt = torch.from_numpy(np.concatenate(s["prompts"])).cuda()
    cu = np.concatenate([[0], np.cumsum([len(p) for p in s["prompts"]])])
    total = sum(sz[-1] for sz in sizes) + int(cu[-1]) + n * L
    ws = workspace(cfg, total, n, L, mode)
    ids = torch.full((n * L,), cfg.mask_id, dtype=torch.int32, device="cuda")
    msk = torch.ones((n * L,), dtype=torch.uint8, device="cuda")
    fixed = [0] * (n * T)
    dv.davet_run_schedule(model_cfg(cfg, mode), mdl.weights, geoms, visual,
                          bufs, prompt, cu, L, T, cfg.k, None, fixed, ids, msk,
                          ws)
    torch.cuda.synchronize()
    for i in range(n):
        host = to_mode(s["visual"][i], mode)[1]
        ref, _ = R.build_views(host, s["n_crops"][i], cfg.grid, cfg.K,
                               RZ[name], mode)
        for l in range(cfg.K - 1):
            got = _levels_to_f32(bufs[i * (cfg.K - 1) + l], mode)
            assert np.array_equal(got, ref[l]), (i, l)
    assert int(msk.sum()) == n * (L - min(L, T * cfg.k))
