"""Helpers of the GPU parity tests: device upload of the seeded inputs in a
compute mode, the oracle-side values, and the comparison rules.

Compute modes: "f32" (the fp32 configuration), "f16" and "bf16" (16-bit
matrix-core operands).  A bf16 model runs in either 16-bit mode; in "f16"
mode its bf16 weights and encodings are converted to fp16 (round to nearest
even, exact for every value with |x| >= 2^-17).  The oracle is fed either
the very same converted values (``oracle_values="device"``, the default of
the small-shape tests) or the model's own bf16-rounded values
(``oracle_values="model"``: the conversion, and the fp16 rounding of the
pooled views, then sit inside the measured error).

Comparison rules (floating point decides an integer, so the argmax is
compared where it is unique at the tolerance, and checked for validity
elsewhere):
  logits   relative RMS error over the masked rows <= tol (1e-5 for the fp32
           path; 1e-2 for the 16-bit modes, against the oracle fed the same
           16-bit values)
  argmax   equal wherever the oracle's top-two gap exceeds ``gap`` (a few
           times the absolute logit error); elsewhere the GPU's choice must be
           within ``gap`` of the oracle's maximum
  conf     equal to the max softmax probability of the GPU's own stored
           logits to 1e-4, and within exp(2 max|dlogit|) - 1 of the oracle's
"""

import numpy as np
import torch

import paper_2608_01821_amd as dv
import synth
from oracle import decode, model, realizers, views

TOL = {"f32": dict(logits=1e-5, gap=1e-4),
       "bf16": dict(logits=1e-2, gap=None),
       "f16": dict(logits=1e-2, gap=None)}

DTYPE = {"f32": dv.DAVET_F32, "bf16": dv.DAVET_BF16, "f16": dv.DAVET_F16}


def default_mode(cfg):
    return "f32" if cfg.dtype == "f32" else "f16"


def to_mode(arr, mode):
    """(numpy array stored on the device, float32 values the device sees)."""
    a = np.ascontiguousarray(arr, np.float32)
    if mode == "f16":
        h = a.astype(np.float16)
        return h.view(np.int16), h.astype(np.float32)
    if mode == "bf16":
        bits = synth.f32_to_bf16_bits(a)
        return bits.view(np.int16), synth.bf16_bits_to_f32(bits)
    return a, a


def dev_tensor(arr, mode):
    return torch.from_numpy(to_mode(arr, mode)[0]).cuda()


def model_cfg(cfg, mode=None):
    mode = mode or default_mode(cfg)
    return dv.ModelCfg(cfg.n_layers, cfg.d, cfg.n_heads, cfg.head_dim, cfg.ffn,
                       cfg.vocab, cfg.mask_id, cfg.rms_eps, cfg.rope_theta,
                       DTYPE[mode])


def view_geom(cfg, n_crops, mode=None, mixed_stride=0, realizer=0):
    mode = mode or default_mode(cfg)
    return dv.ViewGeom(n_crops, cfg.grid, cfg.d, cfg.K, DTYPE[mode],
                       mixed_stride, realizer)


class Model:
    """Seeded weights on both sides in one compute mode.  ``host`` feeds the
    oracle the values the device holds (oracle_values="device") or the
    model's own values as generated (oracle_values="model": bf16-rounded for
    a bf16 model) -- in memory, or regenerated per layer on demand when
    ``stream_host`` is set (large stacks)."""

    def __init__(self, cfg, mode=None, keep_host=True, stream_host=False,
                 oracle_values="device"):
        assert oracle_values in ("device", "model")
        self.cfg = cfg
        self.mode = mode = mode or default_mode(cfg)
        self.oracle_values = oracle_values

        def host_of(a):
            if oracle_values == "model":
                return np.ascontiguousarray(a, np.float32)
            return to_mode(a, mode)[1]

        def both(a):
            dev, _ = to_mode(a, mode)
            return torch.from_numpy(dev).cuda(), host_of(a)

        self.dev_layers = []
        host_layers = []
        for i in range(cfg.n_layers):
            lw = synth.gen_layer_weights(cfg, i)
            pair = {k: both(v) for k, v in lw.items()}
            del lw
            self.dev_layers.append({k: p[0] for k, p in pair.items()})
            if keep_host and not stream_host:
                host_layers.append({k: p[1] for k, p in pair.items()})
        self.dev_embed, embed = both(synth.gen_embed(cfg))
        self.dev_head, head = both(synth.gen_head(cfg))
        self.weights = dv.Weights(self.dev_embed, self.dev_head,
                                  self.dev_layers)
        self.host = None
        if keep_host:
            if stream_host:
                def layers(i):
                    return {k: host_of(v) for k, v in
                            synth.gen_layer_weights(cfg, i).items()}
            else:
                layers = host_layers
            self.host = dict(embed=embed, head=head, layers=layers)


class Sample:
    """One sample's inputs on both sides and its GPU-built views.  With
    oracle_values="model" the oracle's views are built from the encoding as
    generated (bf16-rounded for a bf16 model) and kept at float32 (the
    float64 window means rounded once to fp32, 2^-24 relative): the
    oracle's inputs are the model's own, and whatever precision the GPU
    stores its views in sits inside the measured error."""

    def __init__(self, cfg, n_crops, visual, prompt, mode=None,
                 mixed_stride=0, realizer=0, oracle_values="device"):
        self.cfg = cfg
        self.mode = mode = mode or default_mode(cfg)
        dev_v, host_v = to_mode(visual, mode)
        ref_dtype = mode
        if oracle_values == "model":
            host_v = np.ascontiguousarray(visual, np.float32)
            ref_dtype = "f32"
        self.visual = host_v
        self.prompt = prompt
        self.n_crops = n_crops
        if realizer:
            self.ref_levels, _ = realizers.build_views(
                host_v, n_crops, cfg.grid, cfg.K, realizer, ref_dtype)
        else:
            self.ref_levels, _ = views.build_views(host_v, n_crops, cfg.grid,
                                                   cfg.K, ref_dtype,
                                                   mixed_stride)
        geom = view_geom(cfg, n_crops, mode, mixed_stride, realizer)
        self.sizes = dv.davet_view_sizes(geom)
        self.dev_v = torch.from_numpy(dev_v).cuda()
        tdt = torch.float32 if mode == "f32" else torch.int16
        self.dev_levels = [torch.empty((self.sizes[l], cfg.d), dtype=tdt,
                                       device="cuda")
                           for l in range(cfg.K - 1)]
        dv.davet_build_views(geom, self.dev_v, self.dev_levels)
        self.dev_levels.append(self.dev_v)
        self.dev_prompt = torch.from_numpy(prompt).cuda()


def workspace(cfg, max_tokens, n_seqs, L, mode=None):
    nbytes = dv.davet_workspace_bytes(model_cfg(cfg, mode), max_tokens,
                                      n_seqs, L)
    return torch.empty(nbytes, dtype=torch.uint8, device="cuda")


def rel_rms(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.sqrt(np.mean((got - ref) ** 2)) /
                 np.sqrt(np.mean(ref ** 2)))


# The head reduces each row's fp32 logits with fp32 exponentials (within 2
# ulp) and fp32 sums in a merge tree over at most ~1000 vocabulary slabs, so
# its confidence lies within 1e-4 relative of the exact value computed from
# the very logits it stored.
HEAD_SELF_RTOL = 1e-4


def check_decode(gpu_am, gpu_conf, ref_logits, ref_am, ref_conf, mask_id,
                 gap, gpu_logits):
    """Argmax / confidence rules above, row by row.

    Two checks on the confidences: (1) against the GPU's own logits
    (`gpu_logits`, the rows the head stored): the argmax is that of the
    stored values exactly (lowest id on ties) and the confidence is their
    max softmax probability to HEAD_SELF_RTOL -- this isolates the head's
    reduction; (2) against the oracle: log conf = max_w l_w - LSE(l) moves by
    at most 2 max_w |dl_w| when the logits move by dl, so the relative error
    per row is bounded by exp(2 max_w |l_gpu - l_ref|) - 1 (plus the
    reduction's own 1e-4)."""
    ref = np.asarray(ref_logits, np.float64).copy()
    ref[:, mask_id] = -np.inf
    top2 = np.sort(ref, axis=1)[:, -2:]
    unique = (top2[:, 1] - top2[:, 0]) > gap
    am = np.asarray(gpu_am)
    assert np.array_equal(am[unique], np.asarray(ref_am)[unique]), \
        "argmax differs where it is unique"
    rows = np.arange(len(am))
    chosen = ref[rows, am]
    assert np.all(chosen >= top2[:, 1] - gap), "argmax not a near-maximum"
    assert np.all(am != mask_id)
    conf = np.asarray(gpu_conf, np.float64)
    # (1) the head's reduction against the logits it stored
    gl = np.asarray(gpu_logits, np.float64).copy()
    gl[:, mask_id] = -np.inf
    self_am = np.argmax(gl, axis=1)              # first index on ties
    assert np.array_equal(am, self_am), "argmax differs from the stored logits'"
    gmax = gl[rows, self_am]
    self_conf = 1.0 / np.exp(gl - gmax[:, None]).sum(axis=1)
    rel_self = np.abs(conf - self_conf) / self_conf
    assert rel_self.max() <= HEAD_SELF_RTOL, ("conf vs own logits", rel_self.max())
    # (2) against the oracle, within the bound the logit error implies
    dl = np.abs(np.asarray(gpu_logits, np.float64) - np.asarray(ref_logits,
                                                                np.float64))
    dl[:, mask_id] = 0.0
    bound = np.expm1(2.0 * dl.max(axis=1)) + 2 * HEAD_SELF_RTOL
    rel = np.abs(conf - ref_conf) / ref_conf
    assert np.all(rel <= bound), ("conf", rel.max(), bound.min())
    return int(unique.sum())


def random_state(rng, L, mask_id, vocab, frac_masked):
    """A partially denoised answer: committed positions hold random ids."""
    masked = (rng.random(L) < frac_masked).astype(np.uint8)
    masked[rng.integers(0, L)] = 1                 # at least one masked
    ids = rng.integers(0, vocab - 1, L).astype(np.int32)
    ids[masked == 1] = mask_id
    return ids, masked


def run_gpu_step(cfg, mdl, samples, levels, ids, masked, want_logits=True):
    n = len(samples)
    L = cfg.resp_len
    mode = mdl.mode
    prompt = torch.cat([s.dev_prompt for s in samples])
    cu = np.concatenate([[0], np.cumsum([len(s.prompt) for s in samples])])
    views_ = [s.dev_levels[lv] for s, lv in zip(samples, levels)]
    nview = [s.sizes[lv] for s, lv in zip(samples, levels)]
    total = sum(nview) + int(cu[-1]) + n * L
    ws = workspace(cfg, total, n, L, mode)
    d_ids = torch.from_numpy(np.ascontiguousarray(ids, np.int32)).cuda()
    d_m = torch.from_numpy(np.ascontiguousarray(masked, np.uint8)).cuda()
    conf = torch.full((n * L,), 123.0, device="cuda")
    am = torch.full((n * L,), -7, dtype=torch.int32, device="cuda")
    logits = torch.full((n * L, cfg.vocab), 55.0, device="cuda") \
        if want_logits else None
    dv.davet_denoise_step(model_cfg(cfg, mode), mdl.weights, views_, nview,
                          prompt, cu, d_ids, d_m, L, conf, am, logits, ws)
    torch.cuda.synchronize()
    return (conf.cpu().numpy().reshape(n, L), am.cpu().numpy().reshape(n, L),
            None if logits is None else
            logits.cpu().numpy().reshape(n, L, cfg.vocab))


def oracle_step(cfg, mdl, sample, level, ids, masked, rows=None):
    pos, lg = model.step_logits(cfg, sample.ref_levels[level], sample.prompt,
                                ids, masked, mdl.host, rows=rows)
    am, cf = decode.argmax_conf(lg, cfg.mask_id)
    return pos, lg, am, cf


def compare(cfg, tol, masked, g_conf, g_am, g_logits, pos, ref_lg, ref_am,
            ref_cf):
    m = masked.astype(bool)
    assert np.all(g_conf[~m] == -np.inf) and np.all(g_am[~m] == -1)
    err = rel_rms(g_logits[pos], ref_lg)
    assert err <= tol["logits"], ("logits rel-RMS", err)
    assert np.all(g_logits[~m] == 55.0)            # only masked rows written
    gap = tol["gap"] or 6.0 * err * float(np.sqrt(np.mean(ref_lg ** 2)))
    check_decode(g_am[pos], g_conf[pos], ref_lg, ref_am, ref_cf, cfg.mask_id,
                 gap, g_logits[pos])
    return err


# The tiled head reduces each row over 256-column vocabulary slabs, the
# row-major head over 128-column ones: the logits are the same bits (same
# products, same K order), the confidence is the same softmax maximum with
# its fp32 sum of exponentials grouped differently.  Along each path of an
# online-softmax reduction tree a level adds at most one rounding of the add
# (2^-24 relative) and one rescale by exp(m_old - m_new) (__expf, within
# 2 ulp: 2^-22); both trees are under 48 levels deep at V <= 2^17 (a lane's
# columns, 5 shuffle levels, 2 wave halves, the slab merge), so the two
# results lie within 2 * 48 * 5 * 2^-24 < 3e-5 of each other.
CONF_REGROUP_RTOL = 3e-5


def assert_conf_regrouped(a, b):
    """Confidences from the two head layouts: -inf (committed rows) at the
    same places, finite values within CONF_REGROUP_RTOL."""
    a = np.asarray(a)
    b = np.asarray(b)
    fa, fb = np.isfinite(a), np.isfinite(b)
    assert np.array_equal(fa, fb)
    assert np.array_equal(a[~fa], b[~fb])
    rel = np.abs(a[fa].astype(np.float64) - b[fb]) / np.abs(b[fb])
    assert rel.size == 0 or rel.max() <= CONF_REGROUP_RTOL, rel.max()
