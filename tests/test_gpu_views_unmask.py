"""GPU parity of the evidence hierarchy and of the commitment kernel against
the oracle: bit-exact index maps, selections and bf16 views; fp32 views to
1e-6 relative (the float64 accumulation makes them equal in practice)."""

import numpy as np
import pytest
import torch

import paper_2608_01821_amd as dv
import synth
from oracle import decode, views
from gpu_util import DTYPE, dev_tensor, to_mode

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,C,G,K,d", [
    ("f32", 1, 12, 3, 256),       # tiny config: 144 -> 36 -> 9
    ("bf16", 1, 27, 3, 4096),     # one 27x27 crop: 729 -> 196 -> 49
    ("bf16", 5, 27, 3, 4096),     # five crops: 3645 -> 980 -> 245
    ("f32", 2, 7, 4, 64),         # four levels, odd grid
    ("bf16", 3, 5, 2, 16),        # two levels
    ("f32", 1, 1, 3, 8),          # a single token
    ("bf16", 2, 13, 1, 24),       # one level: nothing pooled, identity map
    ("f16", 1, 27, 3, 4096),      # fp16 operand mode
    ("f16", 4, 27, 3, 4096),      # four crops: 2916 -> 784 -> 196
    ("f16", 2, 7, 4, 64),
])
def test_views_match_oracle(dtype, C, G, K, d):
    rng = np.random.default_rng(100 + C * 7 + G + K)
    v = rng.standard_normal((C * G * G, d)).astype(np.float32)
    if dtype == "bf16":
        v = synth.round_to_bf16(v)
    v = to_mode(v, dtype)[1]
    vd = dev_tensor(v, dtype)
    geom = dv.ViewGeom(C, G, d, K, DTYPE[dtype])
    sizes = dv.davet_view_sizes(geom)
    tdt = torch.float32 if dtype == "f32" else torch.int16
    levels = [torch.full((sizes[l], d), -7, dtype=tdt, device="cuda")
              for l in range(K - 1)]
    offs = [torch.full((sizes[l] + 1,), -1, dtype=torch.int32, device="cuda")
            for l in range(K)]
    mems = [torch.full((C * G * G,), -1, dtype=torch.int32, device="cuda")
            for l in range(K)]
    dv.davet_build_views(geom, vd, levels, offs, mems)
    torch.cuda.synchronize()
    ref_levels, ref_maps = views.build_views(v, C, G, K, dtype)
    for l in range(K):
        assert np.array_equal(offs[l].cpu().numpy(), ref_maps[l][0])
        assert np.array_equal(mems[l].cpu().numpy(), ref_maps[l][1])
    for l in range(K - 1):
        got = levels[l].cpu().numpy()
        if dtype != "f32":
            got = synth.bf16_bits_to_f32(got.view(np.uint16)) \
                if dtype == "bf16" else got.view(np.float16).astype(np.float32)
            assert np.array_equal(got, ref_levels[l])      # bit-exact
        else:
            ref = ref_levels[l]
            rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
            assert rel <= 1e-6
            assert np.array_equal(got, ref)   # same float64 sums, same order


def _unmask_case(rng, n_seqs, L, k):
    vals = np.array([0.1, 0.5, 0.5, 0.9, -np.inf, np.nan, 1.0, 0.25],
                    dtype=np.float32)
    conf = np.where(rng.random((n_seqs, L)) < 0.5,
                    rng.choice(vals, (n_seqs, L)),
                    rng.random((n_seqs, L)).astype(np.float32))
    conf = conf.astype(np.float32)
    masked = (rng.random((n_seqs, L)) < 0.7).astype(np.uint8)
    am = rng.integers(0, 1000, (n_seqs, L)).astype(np.int32)
    ids = np.where(masked == 1, 999, rng.integers(0, 999, (n_seqs, L)))
    return conf, masked, am, ids.astype(np.int32)


@pytest.mark.parametrize("n_seqs,L,k", [(1, 32, 4), (4, 37, 7), (16, 128, 2),
                                        (3, 256, 2), (2, 1024, 9), (5, 1, 3),
                                        (2, 5, 16)])
def test_unmask_matches_oracle(n_seqs, L, k):
    rng = np.random.default_rng(L * 31 + k)
    conf, masked, am, ids = _unmask_case(rng, n_seqs, L, k)
    d_conf = torch.from_numpy(conf).cuda()
    d_am = torch.from_numpy(am).cuda()
    d_ids = torch.from_numpy(ids).cuda()
    d_m = torch.from_numpy(masked).cuda()
    sel = torch.full((n_seqs, k), -5, dtype=torch.int32, device="cuda")
    dv.davet_unmask(n_seqs, L, k, d_conf, d_am, d_ids, d_m, sel)
    torch.cuda.synchronize()
    for s in range(n_seqs):
        ref_sel = decode.select(conf[s], masked[s], k)
        ref_ids, ref_m = decode.commit(ids[s], masked[s], am[s], ref_sel)
        got_sel = sel[s].cpu().numpy()
        live = got_sel[got_sel >= 0]
        assert sorted(live.tolist()) == ref_sel
        assert np.all(got_sel[len(live):] == -1)
        # rank order: confidence descending, position ascending
        keys = [(-decode.rank_key(float(conf[s][i])), int(i)) for i in live]
        assert keys == sorted(keys)
        assert np.array_equal(d_ids[s].cpu().numpy(), ref_ids)
        assert np.array_equal(d_m[s].cpu().numpy(), ref_m)


def test_unmask_reveals_everything_after_enough_steps():
    rng = np.random.default_rng(9)
    L, k = 40, 6
    conf = rng.random((1, L)).astype(np.float32)
    d_conf = torch.from_numpy(conf).cuda()
    d_am = torch.arange(L, dtype=torch.int32, device="cuda").reshape(1, L)
    d_ids = torch.full((1, L), 77, dtype=torch.int32, device="cuda")
    d_m = torch.ones((1, L), dtype=torch.uint8, device="cuda")
    counts = []
    for _ in range(7):
        before = int(d_m.sum())
        dv.davet_unmask(1, L, k, d_conf, d_am, d_ids, d_m)
        counts.append(before - int(d_m.sum()))
    assert counts == [6, 6, 6, 6, 6, 6, 4]
    assert int(d_m.sum()) == 0
    assert np.array_equal(d_ids.cpu().numpy()[0], np.arange(L))


@pytest.mark.parametrize("src,dst", [("bf16", "f16"), ("f32", "f16"),
                                     ("f32", "bf16"), ("f16", "f32")])
def test_convert_matches_numpy(src, dst):
    """davet_convert rounds to nearest even exactly as numpy does, including
    fp16 subnormals, overflow to infinity and tiny bf16 values."""
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(100003) *
         np.exp(rng.uniform(-20, 12, 100003))).astype(np.float32)
    x[:4] = [0.0, -0.0, 70000.0, 2.0 ** -26]
    if src == "bf16":
        x = synth.round_to_bf16(x)
    elif src == "f16":
        x = x.astype(np.float16).astype(np.float32)
    d_src = dev_tensor(x, src)
    tdt = torch.float32 if dst == "f32" else torch.int16
    d_dst = torch.empty(x.size, dtype=tdt, device="cuda")
    dv.davet_convert(d_src, DTYPE[src], d_dst, DTYPE[dst])
    torch.cuda.synchronize()
    got = d_dst.cpu().numpy()
    exp = to_mode(x, dst)[0]
    assert np.array_equal(got.view(np.uint8), exp.view(np.uint8))
