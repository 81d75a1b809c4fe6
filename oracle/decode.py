"""Deterministic decoding and confidence-ranked commitment (Sec. 3.1, Eq. 2;
Sec. 5.1: commitment by confidence ranking, temperature 0).

Readings: the prediction is the argmax over every token except [MASK]
(ties to the lowest id), and its confidence is the max softmax probability
with [MASK] left out of the normaliser, so a committed position is never
[MASK].  Commitment takes min(k, |M_t|) masked positions with the largest
confidence, ties to the lower position; NaN and -inf confidences rank last.
"""

import math

import numpy as np


def argmax_conf(logits: np.ndarray, mask_id: int):
    """Per row: (argmax over w != mask_id, lowest id on ties;
    conf = 1 / sum_{w != mask} exp(l_w - l_argmax)), float64."""
    lg = np.asarray(logits, dtype=np.float64)
    n, V = lg.shape
    keep = np.ones(V, dtype=bool)
    keep[mask_id] = False
    ids = np.arange(V)[keep]
    sub = lg[:, keep]
    j = np.argmax(sub, axis=1)            # numpy returns the first maximum
    am = ids[j]
    top = sub[np.arange(n), j]
    conf = 1.0 / np.exp(sub - top[:, None]).sum(axis=1)
    return am.astype(np.int32), conf


def rank_key(c: float) -> float:
    """Sort key of a confidence: NaN ranks with -inf, below every number."""
    return -math.inf if math.isnan(c) else c


def select(conf, masked, k: int):
    """Positions committed this step: the min(k, |M_t|) masked positions in
    order of (confidence descending, position ascending)."""
    cand = [i for i in range(len(masked)) if masked[i]]
    cand.sort(key=lambda i: (-rank_key(float(conf[i])), i))
    return sorted(cand[:min(k, len(cand))])


def commit(resp_ids, masked, argmax, selected):
    """Eq. (2): selected positions take their prediction, the other masked
    positions stay [MASK], committed positions never change."""
    ids = np.array(resp_ids, dtype=np.int32, copy=True)
    m = np.array(masked, dtype=np.uint8, copy=True)
    for i in selected:
        ids[i] = argmax[i]
        m[i] = 0
    return ids, m
