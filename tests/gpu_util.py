"""Helpers of the GPU parity tests: device upload of the seeded inputs, the
oracle-side weight dicts, and the comparison rules.

Comparison rules (floating point decides an integer, so the argmax is
compared where it is unique at the tolerance, and checked for validity
elsewhere):
  logits   relative RMS error over the masked rows <= tol (1e-5 for the fp32
           path; 1e-2 for bf16, against the oracle fed the same bf16 values)
  argmax   equal wherever the oracle's top-two gap exceeds ``gap`` (a few
           times the absolute logit error); elsewhere the GPU's choice must be
           within ``gap`` of the oracle's maximum
  conf     relative error <= conf_tol
"""

import numpy as np
import torch

import paper_2608_01821_amd as dv
import synth


def dev_tensor(arr, cfg_dtype):
    """float32 numpy array -> device tensor in the model dtype (bf16 bits
    stored as int16; values already bf16-representable)."""
    if cfg_dtype == "bf16":
        bits = synth.f32_to_bf16_bits(np.ascontiguousarray(arr, np.float32))
        return torch.from_numpy(bits.view(np.int16)).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr, np.float32)).cuda()


def model_cfg(cfg):
    return dv.ModelCfg(cfg.n_layers, cfg.d, cfg.n_heads, cfg.head_dim, cfg.ffn,
                       cfg.vocab, cfg.mask_id, cfg.rms_eps, cfg.rope_theta,
                       dv.DAVET_BF16 if cfg.dtype == "bf16" else dv.DAVET_F32)


def view_geom(cfg, n_crops):
    return dv.ViewGeom(n_crops, cfg.grid, cfg.d, cfg.K,
                       dv.DAVET_BF16 if cfg.dtype == "bf16" else dv.DAVET_F32)


class Model:
    """Seeded weights on both sides: ``host`` feeds the oracle (float32
    arrays holding the same values), ``dev`` is the library's struct."""

    def __init__(self, cfg, keep_host=True):
        self.cfg = cfg
        embed = synth.gen_embed(cfg)
        head = synth.gen_head(cfg)
        layers = [synth.gen_layer_weights(cfg, i) for i in range(cfg.n_layers)]
        self.dev_layers = [{k: dev_tensor(v, cfg.dtype) for k, v in lw.items()}
                           for lw in layers]
        self.dev_embed = dev_tensor(embed, cfg.dtype)
        self.dev_head = dev_tensor(head, cfg.dtype)
        self.weights = dv.Weights(self.dev_embed, self.dev_head,
                                  self.dev_layers)
        self.host = dict(embed=embed, head=head, layers=layers) \
            if keep_host else None


def workspace(cfg, max_tokens, n_seqs, L):
    nbytes = dv.davet_workspace_bytes(model_cfg(cfg), max_tokens, n_seqs, L)
    return torch.empty(nbytes, dtype=torch.uint8, device="cuda")


def rel_rms(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.sqrt(np.mean((got - ref) ** 2)) /
                 np.sqrt(np.mean(ref ** 2)))


def check_decode(gpu_am, gpu_conf, ref_logits, ref_am, ref_conf, mask_id,
                 gap, conf_tol):
    """Argmax / confidence rules above, row by row."""
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
    err = np.abs(np.asarray(gpu_conf, np.float64) - ref_conf) / ref_conf
    assert err.max() <= conf_tol, ("conf", err.max())
    return int(unique.sum())


def random_state(rng, L, mask_id, vocab, frac_masked):
    """A partially denoised answer: committed positions hold random ids."""
    masked = (rng.random(L) < frac_masked).astype(np.uint8)
    masked[rng.integers(0, L)] = 1                 # at least one masked
    ids = rng.integers(0, vocab - 1, L).astype(np.int32)
    ids[masked == 1] = mask_id
    return ids, masked
