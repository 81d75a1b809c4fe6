"""Pins of the oracle's denoiser (Sec. 3.1, Eq. 1: bidirectional attention).

Each piece is checked against an independent library routine (torch's
float64 rms_norm, silu and scaled_dot_product_attention; rotary embedding in
its complex-multiplication form), a brute-force loop on tiny inputs, or an
invariant the mathematics fixes (no causal mask, permutation equivariance,
relative-position property of rotary embedding).
"""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import model


def _t(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float64))


def test_rmsnorm_against_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((7, 33))
    g = rng.standard_normal(33)
    y = model.rmsnorm(x, g, 1e-5)
    ref = F.rms_norm(_t(x), (33,), _t(g), eps=1e-5).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-13)
    # unit RMS and scale invariance with eps = 0
    z = model.rmsnorm(x, None, 0.0)
    np.testing.assert_allclose(np.sqrt((z * z).mean(-1)), 1.0, rtol=1e-13)
    np.testing.assert_allclose(model.rmsnorm(3.5 * x, None, 0.0), z,
                               rtol=1e-13)


def test_silu_against_torch_and_values():
    x = np.linspace(-20, 20, 101)
    np.testing.assert_allclose(model.silu(x), F.silu(_t(x)).numpy(),
                               rtol=1e-13, atol=1e-300)
    assert model.silu(np.array([0.0]))[0] == 0.0
    assert model.silu(np.array([1.0]))[0] == pytest.approx(
        1.0 / (1.0 + math.exp(-1.0)), rel=1e-15)


def _rope_complex(x, theta):
    """Rotary embedding as complex multiplication: z_i = x_i + j x_{i+D/2}
    times exp(j * pos * theta^(-2i/D))."""
    N, H, D = x.shape
    half = D // 2
    xt = _t(x)
    z = torch.complex(xt[..., :half], xt[..., half:])
    inv = theta ** (-(2.0 * torch.arange(half, dtype=torch.float64)) / D)
    ang = torch.arange(N, dtype=torch.float64)[:, None] * inv[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)[:, None, :]
    w = z * rot
    return torch.cat([w.real, w.imag], dim=-1).numpy()


def test_rope_complex_form_and_properties():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((20, 3, 16))
    ang = model.rope_angles(20, 16, 10000.0)
    y = model.rope(x, ang)
    np.testing.assert_allclose(y, _rope_complex(x, 10000.0), rtol=1e-12,
                               atol=1e-13)
    # position 0 is the identity; rotation preserves norms
    np.testing.assert_allclose(y[0], x[0], rtol=0, atol=0)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1),
                               np.linalg.norm(x, axis=-1), rtol=1e-13)
    # <rope(q, m), rope(k, n)> depends only on m - n
    q = rng.standard_normal(16)
    k = rng.standard_normal(16)
    Q = model.rope(np.tile(q, (20, 1, 1)), ang)[:, 0]
    Kk = model.rope(np.tile(k, (20, 1, 1)), ang)[:, 0]
    assert Q[5] @ Kk[2] == pytest.approx(Q[13] @ Kk[10], rel=1e-12)
    assert Q[2] @ Kk[5] == pytest.approx(Q[10] @ Kk[13], rel=1e-12)


def _attention_loops(q, k, v):
    N, H, D = q.shape
    out = np.zeros_like(q)
    for h in range(H):
        for i in range(N):
            sc = [sum(q[i, h, e] * k[j, h, e] for e in range(D)) / math.sqrt(D)
                  for j in range(N)]
            m = max(sc)
            ws = [math.exp(s - m) for s in sc]
            z = sum(ws)
            for e in range(D):
                out[i, h, e] = sum(ws[j] * v[j, h, e] for j in range(N)) / z
    return out


def test_attention_brute_force_tiny():
    rng = np.random.default_rng(2)
    q, k, v = (rng.standard_normal((9, 2, 4)) for _ in range(3))
    np.testing.assert_allclose(model.attention(q, k, v),
                               _attention_loops(q, k, v), rtol=1e-12)


def test_attention_against_sdpa_no_mask():
    rng = np.random.default_rng(3)
    q, k, v = (rng.standard_normal((37, 4, 32)) for _ in range(3))
    ref = F.scaled_dot_product_attention(
        _t(q).transpose(0, 1), _t(k).transpose(0, 1), _t(v).transpose(0, 1),
        is_causal=False).transpose(0, 1).numpy()
    np.testing.assert_allclose(model.attention(q, k, v), ref, rtol=1e-11)


def test_attention_is_not_causal():
    rng = np.random.default_rng(4)
    q, k, v = (rng.standard_normal((12, 2, 8)) for _ in range(3))
    base = model.attention(q, k, v)
    k2, v2 = k.copy(), v.copy()
    k2[-1] += 1.0
    v2[-1] += 1.0
    moved = model.attention(q, k2, v2)
    # the first query sees the last key: its output changes
    assert np.abs(moved[0] - base[0]).max() > 1e-3


def test_attention_permutation_equivariant_and_special_cases():
    rng = np.random.default_rng(5)
    q, k, v = (rng.standard_normal((10, 2, 8)) for _ in range(3))
    perm = rng.permutation(10)
    a = model.attention(q, k, v)
    b = model.attention(q[perm], k[perm], v[perm])
    np.testing.assert_allclose(b, a[perm], rtol=1e-12)
    # identical keys: uniform weights, output is the mean of v
    kk = np.repeat(k[:1], 10, axis=0)
    np.testing.assert_allclose(model.attention(q, kk, v),
                               np.broadcast_to(v.mean(0), v.shape),
                               rtol=1e-12)
    # one key: output is that value
    np.testing.assert_allclose(model.attention(q[:1], k[:1], v[:1]), v[:1])


def _torch_layer(x, w, H, D, eps, theta):
    """Same layer from torch float64 library pieces (SDPA, rms_norm, silu)
    with rotary embedding in complex form."""
    N, d = x.shape
    xt = _t(x)
    a = F.rms_norm(xt, (d,), eps=eps)
    qkv = a @ _t(w["wqkv"]).T
    q = _rope_complex(qkv[:, :d].reshape(N, H, D).numpy(), theta)
    k = _rope_complex(qkv[:, d:2 * d].reshape(N, H, D).numpy(), theta)
    v = qkv[:, 2 * d:].reshape(N, H, D)
    o = F.scaled_dot_product_attention(
        _t(q).transpose(0, 1), _t(k).transpose(0, 1), v.transpose(0, 1))
    xt = xt + o.transpose(0, 1).reshape(N, d) @ _t(w["wo"]).T
    a = F.rms_norm(xt, (d,), eps=eps)
    hdn = F.silu(a @ _t(w["wg"]).T) * (a @ _t(w["wu"]).T)
    return (xt + hdn @ _t(w["wd"]).T).numpy()


def test_layer_against_torch_composition():
    rng = np.random.default_rng(6)
    N, d, H, D, Fh = 23, 64, 4, 16, 96
    w = dict(wqkv=rng.standard_normal((3 * d, d)) * 0.1,
             wo=rng.standard_normal((d, d)) * 0.1,
             wg=rng.standard_normal((Fh, d)) * 0.1,
             wu=rng.standard_normal((Fh, d)) * 0.1,
             wd=rng.standard_normal((d, Fh)) * 0.1)
    x = rng.standard_normal((N, d))
    got = model.layer(x, w, H, D, 1e-5, model.rope_angles(N, D, 10000.0))
    np.testing.assert_allclose(got, _torch_layer(x, w, H, D, 1e-5, 1e4),
                               rtol=1e-11, atol=1e-11)


def test_embed_sequence_layout():
    E = np.arange(10 * 3, dtype=np.float32).reshape(10, 3)
    view = -np.ones((2, 3), np.float32)
    x = model.embed_sequence(view, [4, 5], [1, 2, 3], [0, 1, 0], E, 9)
    assert x.shape == (7, 3)
    np.testing.assert_array_equal(x[:2], view)
    np.testing.assert_array_equal(x[2], E[4])
    np.testing.assert_array_equal(x[4], E[1])
    np.testing.assert_array_equal(x[5], E[9])       # masked -> [MASK] row
    np.testing.assert_array_equal(x[6], E[3])


def test_step_flops_closed_form():
    # one 8B-shaped layer at N = 889 with 128 head rows
    f = model.step_flops(889, 4096, 12288, 1, 128, 126464)
    per_layer = 2 * 889 * (4 * 4096 ** 2 + 3 * 4096 * 12288) \
        + 4 * 889 ** 2 * 4096
    assert f == per_layer + 2 * 128 * 4096 * 126464


def _torch_layer_gains(x, w, H, D, eps, theta):
    """_torch_layer with the RMSNorm gains of the layer (attn_norm, ffn_norm)
    passed to torch's rms_norm as its weight."""
    N, d = x.shape
    xt = _t(x)
    a = F.rms_norm(xt, (d,), _t(w["attn_norm"]), eps=eps)
    qkv = a @ _t(w["wqkv"]).T
    q = _rope_complex(qkv[:, :d].reshape(N, H, D).numpy(), theta)
    k = _rope_complex(qkv[:, d:2 * d].reshape(N, H, D).numpy(), theta)
    v = qkv[:, 2 * d:].reshape(N, H, D)
    o = F.scaled_dot_product_attention(
        _t(q).transpose(0, 1), _t(k).transpose(0, 1), v.transpose(0, 1))
    xt = xt + o.transpose(0, 1).reshape(N, d) @ _t(w["wo"]).T
    a = F.rms_norm(xt, (d,), _t(w["ffn_norm"]), eps=eps)
    hdn = F.silu(a @ _t(w["wg"]).T) * (a @ _t(w["wu"]).T)
    return (xt + hdn @ _t(w["wd"]).T).numpy()


def _torch_step(view, prompt, resp, masked, W, H, D, eps, theta, mask_id,
                rows, row_offset=None, final_norm=True):
    """Eq. (1) at the response positions ``rows`` composed from torch float64
    pieces: F.embedding for the prompt and the response (the [MASK] id where
    masked), the layer above per layer, torch's rms_norm with the final gain
    on the hidden states of the response rows, then the head product.
    ``row_offset`` (default: the first response row, N - L) and
    ``final_norm`` exist so that the test can show a misplaced gather or a
    dropped final norm is caught."""
    E = _t(W["embed"])
    tok = torch.where(torch.from_numpy(np.asarray(masked, bool)),
                      torch.tensor(mask_id),
                      torch.from_numpy(np.asarray(resp, np.int64)))
    x = torch.cat([_t(view),
                   F.embedding(torch.from_numpy(np.asarray(prompt, np.int64)),
                               E),
                   F.embedding(tok, E)], dim=0).numpy()
    for w in W["layers"]:
        x = _torch_layer_gains(x, w, H, D, eps, theta)
    n, d = x.shape
    off = n - len(resp) if row_offset is None else row_offset
    h = _t(x)[off + torch.from_numpy(np.asarray(rows, np.int64))]
    if final_norm:
        h = F.rms_norm(h, (d,), _t(W["final_norm"]), eps=eps)
    return (h @ _t(W["head"]).T).numpy()


def _tiny_model(rng, n_layers, d, Fh, V):
    def mat(r, c, s=0.15):
        return rng.standard_normal((r, c)) * s

    layers = [dict(wqkv=mat(3 * d, d), wo=mat(d, d), wg=mat(Fh, d),
                   wu=mat(Fh, d), wd=mat(d, Fh),
                   attn_norm=1.0 + 0.3 * rng.standard_normal(d),
                   ffn_norm=1.0 + 0.3 * rng.standard_normal(d))
              for _ in range(n_layers)]
    return dict(embed=mat(V, d, 1.0), head=mat(V, d, 0.5), layers=layers,
                final_norm=1.0 + 0.3 * rng.standard_normal(d))


class _Cfg:
    n_layers, n_heads, head_dim = 2, 2, 16
    rms_eps, rope_theta, mask_id = 1e-5, 100.0, 40


def test_step_logits_against_torch_composition():
    """The oracle's whole step (sequence layout, rotary positions over the
    full sequence, layer stack, gather of the response rows, final norm,
    head) against an independent composition of torch float64 pieces, on a
    2-layer model with a view, a prompt and a partially committed response;
    once at every masked position, once at an explicit subset of rows that
    includes committed positions."""
    rng = np.random.default_rng(11)
    c = _Cfg()
    d, Fh, V = c.n_heads * c.head_dim, 48, c.mask_id + 1
    W = _tiny_model(rng, c.n_layers, d, Fh, V)
    view = rng.standard_normal((5, d))
    prompt = rng.integers(0, V - 1, 4)
    L = 7
    masked = np.array([1, 0, 1, 1, 0, 0, 1], np.uint8)
    resp = rng.integers(0, V - 1, L)
    resp[masked == 1] = c.mask_id

    pos, got = model.step_logits(c, view, prompt, resp, masked, W)
    np.testing.assert_array_equal(pos, np.nonzero(masked)[0])
    ref = _torch_step(view, prompt, resp, masked, W, c.n_heads, c.head_dim,
                      c.rms_eps, c.rope_theta, c.mask_id, pos)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-11)

    rows = np.array([0, 1, 4, 6])
    pos2, got2 = model.step_logits(c, view, prompt, resp, masked, W,
                                   rows=rows)
    np.testing.assert_array_equal(pos2, rows)
    ref2 = _torch_step(view, prompt, resp, masked, W, c.n_heads, c.head_dim,
                       c.rms_eps, c.rope_theta, c.mask_id, rows)
    np.testing.assert_allclose(got2, ref2, rtol=1e-11, atol=1e-11)

    # the comparison is sharp enough to catch the plausible slips: gathering
    # hidden[pos] instead of hidden[N - L + pos], dropping the final norm,
    # embedding the committed id at a masked position
    bad_off = _torch_step(view, prompt, resp, masked, W, c.n_heads,
                          c.head_dim, c.rms_eps, c.rope_theta, c.mask_id,
                          pos, row_offset=0)
    assert np.abs(bad_off - got).max() > 1e-2
    no_norm = _torch_step(view, prompt, resp, masked, W, c.n_heads,
                          c.head_dim, c.rms_eps, c.rope_theta, c.mask_id,
                          pos, final_norm=False)
    assert np.abs(no_norm - got).max() > 1e-2
    resp_leak = resp.copy()
    resp_leak[0] = 3
    leak = _torch_step(view, prompt, resp_leak, np.zeros(L, np.uint8), W,
                       c.n_heads, c.head_dim, c.rms_eps, c.rope_theta,
                       c.mask_id, pos)
    assert np.abs(leak - got).max() > 1e-2


def test_step_logits_rotary_positions_span_whole_sequence():
    """Rotary positions run 0..N-1 over [view | prompt | response]: moving a
    token from the prompt into the view (same rows, same order) changes
    nothing, while restarting positions at the prompt (a plausible slip)
    changes the logits; checked against the torch composition, whose rotary
    table always has N rows."""
    rng = np.random.default_rng(12)
    c = _Cfg()
    d, Fh, V = c.n_heads * c.head_dim, 48, c.mask_id + 1
    W = _tiny_model(rng, c.n_layers, d, Fh, V)
    prompt = rng.integers(0, V - 1, 3)
    view = rng.standard_normal((4, d))
    L = 5
    masked = np.ones(L, np.uint8)
    resp = np.full(L, c.mask_id)
    _, base = model.step_logits(c, view, prompt, resp, masked, W)
    # the same rows with the first prompt token given as a view row
    view2 = np.concatenate([view, np.asarray(W["embed"])[prompt[:1]]])
    _, moved = model.step_logits(c, view2, prompt[1:], resp, masked, W)
    np.testing.assert_allclose(moved, base, rtol=1e-12, atol=1e-12)
    # positions restarted after the view: compose the two parts by hand
    E = np.asarray(W["embed"])
    x = np.concatenate([view, E[prompt], E[resp]])
    N = x.shape[0]
    ang = model.rope_angles(N, c.head_dim, c.rope_theta)
    ang_restart = np.concatenate([ang[:4], ang[:N - 4]])
    for w in W["layers"]:
        x = model.layer(x, w, c.n_heads, c.head_dim, c.rms_eps, ang_restart)
    h = model.rmsnorm(x[N - L:], W["final_norm"], c.rms_eps)
    wrong = h @ np.asarray(W["head"]).T
    assert np.abs(wrong - base).max() > 1e-2
