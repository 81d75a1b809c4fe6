"""The mixed view on the GPU (Sec. 4.3: the pooled view plus a fixed subset
of unpooled tokens) against the oracle: token values bit for bit (the lattice
tokens are copies of v, the coarse tokens single-rounded means), the CSR
index maps exactly, and a denoising step conditioned on the mixed level."""

import numpy as np
import pytest
import torch

import paper_2608_01821_amd as dv
import synth
from oracle import views
from gpu_util import (DTYPE, TOL, Model, Sample, compare, dev_tensor,
                      oracle_step, random_state, run_gpu_step, to_mode)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,C,G,S,d", [
    ("f16", 1, 27, 2, 4096),     # one crop: 49 coarse + 169 lattice tokens
    ("bf16", 5, 27, 3, 256),     # five crops, stride 3
    ("f32", 2, 12, 4, 64),
    ("f16", 3, 7, 2, 64),        # ragged coarse windows
    ("bf16", 1, 1, 2, 16),       # a one-token grid: no lattice token
    ("f32", 2, 9, 5, 32),
])
def test_mixed_view_matches_oracle(dtype, C, G, S, d):
    rng = np.random.default_rng(G * 100 + S * 7 + C)
    v = rng.standard_normal((C * G * G, d)).astype(np.float32)
    if dtype == "bf16":
        v = synth.round_to_bf16(v)
    v = to_mode(v, dtype)[1]
    vd = dev_tensor(v, dtype)
    geom = dv.ViewGeom(C, G, d, 3, DTYPE[dtype], S)
    sizes = dv.davet_view_sizes(geom)
    msz = dv.davet_view_map_sizes(geom)
    tdt = torch.float32 if dtype == "f32" else torch.int16
    levels = [torch.full((sizes[l], d), -7, dtype=tdt, device="cuda")
              for l in range(2)]
    offs = [torch.full((sizes[l] + 1,), -1, dtype=torch.int32, device="cuda")
            for l in range(3)]
    mems = [torch.full((msz[l],), -1, dtype=torch.int32, device="cuda")
            for l in range(3)]
    dv.davet_build_views(geom, vd, levels, offs, mems)
    torch.cuda.synchronize()
    ref_levels, ref_maps = views.build_views(v, C, G, 3, dtype,
                                             mixed_stride=S)
    for l in range(3):
        assert np.array_equal(offs[l].cpu().numpy(), ref_maps[l][0]), l
        assert np.array_equal(mems[l].cpu().numpy(), ref_maps[l][1]), l
    for l in range(2):
        got = levels[l].cpu().numpy()
        if dtype == "bf16":
            got = synth.bf16_bits_to_f32(got.view(np.uint16))
        elif dtype == "f16":
            got = got.view(np.float16).astype(np.float32)
        assert np.array_equal(got, ref_levels[l]), l


@pytest.mark.parametrize("cid", [11, 12])
def test_step_on_mixed_view(cid):
    """A teacher-forced denoising step whose sequences use the mixed level
    (level 1) matches the oracle fed the oracle's own mixed view."""
    cfg = synth.get_any_config(cid)
    mdl = Model(cfg)
    s = synth.gen_sample(cfg)
    n = min(cfg.n_seqs, 3)
    samples = [Sample(cfg, s["n_crops"][i], s["visual"][i], s["prompts"][i],
                      mixed_stride=2) for i in range(n)]
    rng = np.random.default_rng(40 + cid)
    st = [random_state(rng, cfg.resp_len, cfg.mask_id, cfg.vocab, 0.7)
          for _ in samples]
    ids = np.stack([a for a, _ in st])
    masked = np.stack([b for _, b in st])
    levels = [1] * n
    g_conf, g_am, g_lg = run_gpu_step(cfg, mdl, samples, levels, ids, masked)
    for i in range(n):
        pos, rl, ra, rc = oracle_step(cfg, mdl, samples[i], 1, ids[i],
                                      masked[i])
        compare(cfg, TOL[mdl.mode], masked[i], g_conf[i], g_am[i], g_lg[i],
                pos, rl, ra, rc)
