"""Seeded generators for the synthetic workloads (no method arithmetic here).

Seeds: ``1000 * cid + stream``.  Streams: 0 layer weights (``+16 * layer``,
keyed by tensor), 1 visual encoding (keyed by sample), 2 prompt ids,
3 schedule, 4 batch shapes, 5 token embedding, 6 output head.  Normal draws
are made in independently seeded chunks (numpy SeedSequence spawn keys) so
they can be filled by several threads with the same result.  Weights, embedding and head are N(0, 0.02^2);
visual encodings are N(0, 1); prompt ids are uniform over [0, V-1) so that
the mask id V-1 never appears in a prompt.  The bf16 configurations round
every drawn value to bfloat16 (RNE) before either side sees it.
"""

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .configs import Config

_CHUNK = 1 << 22


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest even (finite inputs)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b >> np.uint32(16)) & np.uint32(1)
    return ((b + np.uint32(0x7FFF) + r) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(f32_to_bf16_bits(x))


def _rng(cfg: Config, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(1000 * cfg.cid + stream))


_POOL = None


def _pool():
    global _POOL
    if _POOL is None:
        n = max(1, min(16, len(os.sched_getaffinity(0))))
        _POOL = ThreadPoolExecutor(n)
    return _POOL


def _normal(seed, key, n, std, dtype, as_bits):
    """n draws of std*N(0,1) in float32; bf16 bits when as_bits, else float32
    (bf16-rounded when dtype == 'bf16').  Chunk c of 2^22 values comes from
    PCG64(SeedSequence(seed, spawn_key=key + (c,))), so the values do not
    depend on how many threads fill them."""
    out = np.empty(n, dtype=np.uint16 if as_bits else np.float32)
    s = np.float32(std)

    def fill(c):
        i = c * _CHUNK
        m = min(_CHUNK, n - i)
        ss = np.random.SeedSequence(seed, spawn_key=tuple(key) + (c,))
        z = np.random.Generator(np.random.PCG64(ss)).standard_normal(
            m, dtype=np.float32)
        if s != 1.0:
            z *= s
        if as_bits:
            out[i:i + m] = f32_to_bf16_bits(z)
        elif dtype == "bf16":
            out[i:i + m] = round_to_bf16(z)
        else:
            out[i:i + m] = z

    list(_pool().map(fill, range((n + _CHUNK - 1) // _CHUNK)))
    return out


def gen_layer_weights(cfg: Config, layer: int, as_bits: bool = False):
    """One layer's matrices, drawn in the order wqkv, wo, wg, wu, wd.

    wqkv [3d, d] (rows: q heads, then k heads, then v heads, head-major),
    wo [d, d], wg [F, d], wu [F, d], wd [d, F]; all row-major, out = x @ W^T.
    Norm gains are 1 and are not drawn.
    """
    seed = 1000 * cfg.cid + 16 * layer
    d, F = cfg.d, cfg.ffn
    shapes = dict(wqkv=(3 * d, d), wo=(d, d), wg=(F, d), wu=(F, d), wd=(d, F))
    out = {}
    for j, (name, shp) in enumerate(shapes.items()):
        out[name] = _normal(seed, (j,), shp[0] * shp[1], cfg.weight_std,
                            cfg.dtype, as_bits and cfg.dtype == "bf16"
                            ).reshape(shp)
    return out


def gen_embed(cfg: Config, as_bits: bool = False) -> np.ndarray:
    """Token embedding E [V, d]."""
    return _normal(1000 * cfg.cid + 5, (), cfg.vocab * cfg.d, cfg.weight_std,
                   cfg.dtype, as_bits and cfg.dtype == "bf16"
                   ).reshape(cfg.vocab, cfg.d)


def gen_head(cfg: Config, as_bits: bool = False) -> np.ndarray:
    """Untied output head W_out [V, d]."""
    return _normal(1000 * cfg.cid + 6, (), cfg.vocab * cfg.d, cfg.weight_std,
                   cfg.dtype, as_bits and cfg.dtype == "bf16"
                   ).reshape(cfg.vocab, cfg.d)


def gen_batch_shapes(cfg: Config):
    """Per-sample (n_crops, prompt_len, category) for a batch.

    Fixed-shape configs give the config's own sizes; the ragged config draws
    crops ~ U{lo..hi}, prompt length ~ U{lo..hi} and a query-operation
    category index in {0..4} per sample from stream 4.
    """
    if cfg.crops_range is None:
        return ([cfg.n_crops] * cfg.n_seqs, [cfg.prompt_len] * cfg.n_seqs,
                [0] * cfg.n_seqs)
    rng = _rng(cfg, 4)
    lo, hi = cfg.crops_range
    crops = rng.integers(lo, hi + 1, size=cfg.n_seqs)
    plo, phi = cfg.prompt_range
    plen = rng.integers(plo, phi + 1, size=cfg.n_seqs)
    cat = rng.integers(0, 5, size=cfg.n_seqs)
    return ([int(c) for c in crops], [int(p) for p in plen],
            [int(c) for c in cat])


def gen_visual(cfg: Config, n_crops_list, as_bits: bool = False):
    """Visual encodings v_s [n_crops_s * G * G, d] ~ N(0,1) from stream 1,
    sample s keyed by its index."""
    out = []
    for i, c in enumerate(n_crops_list):
        n = c * cfg.grid * cfg.grid
        out.append(_normal(1000 * cfg.cid + 1, (i,), n * cfg.d, 1.0,
                           cfg.dtype, as_bits and cfg.dtype == "bf16"
                           ).reshape(n, cfg.d))
    return out


def gen_prompt(cfg: Config, prompt_lens):
    """Prompt ids per sample, uniform over [0, V-1), drawn from stream 2."""
    rng = _rng(cfg, 2)
    return [rng.integers(0, cfg.vocab - 1, size=p).astype(np.int32)
            for p in prompt_lens]


def gen_schedule(cfg: Config):
    """Per-step view level for each sample: [n_seqs, T] int32.

    fixed: the config's own list; iid: uniform over {0..K-1} from stream 3.
    Policy-driven configs return None (the allocation policy decides).
    """
    T = cfg.steps
    if cfg.schedule == "fixed":
        lv = np.asarray(cfg.fixed_levels, dtype=np.int32)
        assert lv.shape == (T,)
        return np.tile(lv, (cfg.n_seqs, 1))
    if cfg.schedule == "iid":
        rng = _rng(cfg, 3)
        return rng.integers(0, cfg.K, size=(cfg.n_seqs, T)).astype(np.int32)
    return None


def gen_sample(cfg: Config, as_bits: bool = False):
    """Everything except the weights, for the whole batch of the config."""
    crops, plens, cats = gen_batch_shapes(cfg)
    return dict(
        n_crops=crops,
        prompt_lens=plens,
        categories=cats,
        visual=gen_visual(cfg, crops, as_bits=as_bits),
        prompts=gen_prompt(cfg, plens),
        schedule=gen_schedule(cfg),
    )
