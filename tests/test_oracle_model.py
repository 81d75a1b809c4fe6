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
