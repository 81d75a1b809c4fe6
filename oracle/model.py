"""Bidirectional masked-diffusion denoiser step (Sec. 3.1, Eq. 1).

p_theta(. | y^(t-1), v_t, q) for every answer position, computed by a stack
of pre-norm transformer layers with non-causal attention over the sequence
[view tokens | prompt embeddings | response embeddings].  Masked response
positions are embedded with the [MASK] token (id V-1).

Layer constants (the paper leaves them to the backbone; fixed here): RMSNorm
with gain g and eps 1e-5; rotary embedding with base 10000 and rotate-half
pairing (dim i with dim i + D/2), positions 0..N-1 per sequence; attention
scale 1/sqrt(D); as many key/value heads as query heads; SwiGLU feed-forward
down(silu(gate x) * up x); no biases; untied output head.

Everything is float64; weights arrive as float32 arrays holding bf16 or fp32
values and are widened exactly.
"""

import numpy as np


def rmsnorm(x: np.ndarray, g, eps: float) -> np.ndarray:
    ms = np.mean(x * x, axis=-1, keepdims=True)
    y = x / np.sqrt(ms + eps)
    return y if g is None else y * np.asarray(g, dtype=np.float64)


def rope_angles(n: int, head_dim: int, theta: float) -> np.ndarray:
    half = head_dim // 2
    inv = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / head_dim)
    return np.arange(n, dtype=np.float64)[:, None] * inv[None, :]


def rope(x: np.ndarray, ang: np.ndarray) -> np.ndarray:
    """x [N, H, D]; rotate pairs (i, i + D/2) by angle pos * theta^(-2i/D)."""
    half = x.shape[-1] // 2
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Non-causal softmax attention per head; q, k, v [N, H, D] -> [N, H, D].
    No mask of any kind: every position attends to every position."""
    N, H, D = q.shape
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(D)
    for h in range(H):
        s = (q[:, h, :] @ k[:, h, :].T) * scale
        s = s - s.max(axis=1, keepdims=True)
        e = np.exp(s)
        p = e / e.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, h, :]
    return out


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def _f64(w):
    return np.asarray(w, dtype=np.float64)


def layer_parts(x: np.ndarray, w: dict, n_heads: int, head_dim: int,
                eps: float, ang: np.ndarray):
    """One pre-norm layer: x + O(attn(rope(q), rope(k), v)) then
    x + down(silu(gate a) * up a), with a = RMSNorm of the running x.

    Returns (output, qkv, hdn): the layer output, the projected
    [q | k | v] columns with the rotary embedding applied to q and k, and
    the SwiGLU product fed to the down projection."""
    N, d = x.shape
    a = rmsnorm(x, w.get("attn_norm"), eps)
    qkv = a @ _f64(w["wqkv"]).T
    q = rope(qkv[:, :d].reshape(N, n_heads, head_dim), ang)
    k = rope(qkv[:, d:2 * d].reshape(N, n_heads, head_dim), ang)
    v = qkv[:, 2 * d:].reshape(N, n_heads, head_dim)
    o = attention(q, k, v).reshape(N, d)
    x = x + o @ _f64(w["wo"]).T
    a = rmsnorm(x, w.get("ffn_norm"), eps)
    hdn = silu(a @ _f64(w["wg"]).T) * (a @ _f64(w["wu"]).T)
    qkv_rot = np.concatenate([q.reshape(N, d), k.reshape(N, d),
                              v.reshape(N, d)], axis=1)
    return x + hdn @ _f64(w["wd"]).T, qkv_rot, hdn


def layer(x: np.ndarray, w: dict, n_heads: int, head_dim: int, eps: float,
          ang: np.ndarray) -> np.ndarray:
    """One pre-norm layer (the output of layer_parts)."""
    return layer_parts(x, w, n_heads, head_dim, eps, ang)[0]


def embed_sequence(view, prompt_ids, resp_ids, masked, embed, mask_id):
    """[view rows | E[prompt] | E[response]] with [MASK] at masked positions."""
    resp = np.where(np.asarray(masked, bool), mask_id,
                    np.asarray(resp_ids, np.int64))
    E = np.asarray(embed)
    return np.concatenate([
        _f64(view),
        _f64(E[np.asarray(prompt_ids, np.int64)]),
        _f64(E[resp]),
    ], axis=0)


def forward_hidden(view, prompt_ids, resp_ids, masked, embed, layers,
                   n_layers, n_heads, head_dim, eps, theta, mask_id):
    """Final hidden states of every position, before the final norm.
    ``layers`` is a list of weight dicts or a callable layer -> dict."""
    x = embed_sequence(view, prompt_ids, resp_ids, masked, embed, mask_id)
    ang = rope_angles(x.shape[0], head_dim, theta)
    for li in range(n_layers):
        w = layers(li) if callable(layers) else layers[li]
        x = layer(x, w, n_heads, head_dim, eps, ang)
    return x


def response_logits(hidden, n_resp, masked, head, final_norm, eps,
                    rows=None):
    """Final RMSNorm and logits at the masked response rows (in position
    order), or at the given response positions ``rows``."""
    L = n_resp
    pos = np.nonzero(np.asarray(masked, bool))[0] if rows is None else \
        np.asarray(rows, np.int64)
    h = hidden[hidden.shape[0] - L + pos]
    h = rmsnorm(h, final_norm, eps)
    return pos, h @ _f64(head).T


def step_logits(cfg_like, view, prompt_ids, resp_ids, masked, weights,
                rows=None):
    """Logits of Eq. (1) at masked response positions for one sequence.

    ``cfg_like`` needs n_layers, n_heads, head_dim, rms_eps, rope_theta,
    mask_id.  ``weights`` holds embed, head, optional final_norm, and layers
    (list or callable).  Returns (positions, logits[n, V]) in float64.
    """
    c = cfg_like
    hid = forward_hidden(view, prompt_ids, resp_ids, masked,
                         weights["embed"], weights["layers"], c.n_layers,
                         c.n_heads, c.head_dim, c.rms_eps, c.rope_theta,
                         c.mask_id)
    return response_logits(hid, len(resp_ids), masked, weights["head"],
                           weights.get("final_norm"), c.rms_eps, rows)


def step_flops(n_tokens: int, d: int, ffn: int, n_layers: int,
               n_head_rows: int, vocab: int) -> float:
    """Algorithmic flops of one step: per layer 2N(4d^2 + 3dF) + 4N^2 d
    (full N^2: the attention is non-causal), plus 2 |M_t| d V for the head."""
    per_layer = 2.0 * n_tokens * (4.0 * d * d + 3.0 * d * ffn) \
        + 4.0 * n_tokens * n_tokens * d
    return n_layers * per_layer + 2.0 * n_head_rows * d * vocab
