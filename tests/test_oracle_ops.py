"""Pins of the oracle's sub-operations against library routines, closed forms and invariants."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import dit

rng = np.random.default_rng(1234)


def t64(a):
    return torch.from_numpy(np.asarray(a, np.float64))


def test_layer_norm_matches_torch_and_moments():
    x = rng.standard_normal((7, 96)) * 3 + 1.5
    y = dit.layer_norm(x)
    ref = F.layer_norm(t64(x), (96,), eps=1e-6).numpy()
    np.testing.assert_allclose(y, ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(y.mean(axis=1), 0, atol=1e-12)
    np.testing.assert_allclose(y.var(axis=1), 1, rtol=1e-5)  # eps shifts it by ~1e-7


def test_rms_norm_matches_torch():
    x = rng.standard_normal((5, 64)) * 2
    g = rng.standard_normal(64)
    y = dit.rms_norm(x, g)
    ref = F.rms_norm(t64(x), (64,), weight=t64(g), eps=1e-6).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-13)
    ones = dit.rms_norm(x, np.ones(64))
    np.testing.assert_allclose(np.sqrt((ones ** 2).mean(axis=1)), 1, rtol=1e-6)


def test_gelu_silu_match_torch():
    x = np.linspace(-8, 8, 1001)
    np.testing.assert_allclose(dit.gelu_tanh(x), F.gelu(t64(x), approximate="tanh").numpy(), atol=1e-14)
    np.testing.assert_allclose(dit.silu(x), F.silu(t64(x)).numpy(), atol=1e-14)


def test_linear_matches_torch():
    x = rng.standard_normal((9, 12))
    w = rng.standard_normal((5, 12))
    b = rng.standard_normal(5)
    np.testing.assert_allclose(dit.linear(x, w, b), F.linear(t64(x), t64(w), t64(b)).numpy(), atol=1e-13)


def test_sinusoid_closed_forms():
    s0 = dit.sinusoid(0.0, 256)
    np.testing.assert_array_equal(s0[:128], 1.0)
    np.testing.assert_array_equal(s0[128:], 0.0)
    # frequency 0 is 1 rad per unit time, frequency 64 is 10000^(-1/2) = 0.01
    t = 100.0 * math.pi
    s = dit.sinusoid(t, 256)
    assert s[0] == pytest.approx(math.cos(t), abs=1e-12)
    assert s[128] == pytest.approx(math.sin(t), abs=1e-12)
    assert s[64] == pytest.approx(-1.0, abs=1e-12)      # cos(0.01 * 100 pi) = cos(pi)
    assert s[128 + 64] == pytest.approx(0.0, abs=1e-12)
    # angle addition: [cos, sin](a + b) is the rotation of [cos, sin](a) by b
    a, b = 13.7, 401.25
    sa, sb, sab = dit.sinusoid(a), dit.sinusoid(b), dit.sinusoid(a + b)
    np.testing.assert_allclose(sab[:128], sa[:128] * sb[:128] - sa[128:] * sb[128:], atol=1e-11)
    np.testing.assert_allclose(sab[128:], sa[128:] * sb[:128] + sa[:128] * sb[128:], atol=1e-11)


def _attention_bruteforce(q, k, v):
    Lq, H, dh = q.shape
    out = np.zeros((Lq, H, v.shape[2]))
    for h in range(H):
        for i in range(Lq):
            logits = [sum(q[i, h, c] * k[j, h, c] for c in range(dh)) / math.sqrt(dh) for j in range(k.shape[0])]
            mx = max(logits)
            w = [math.exp(z - mx) for z in logits]
            tot = sum(w)
            for c in range(v.shape[2]):
                out[i, h, c] = sum(w[j] * v[j, h, c] for j in range(k.shape[0])) / tot
    return out


def test_attention_bruteforce_and_torch():
    q = rng.standard_normal((5, 2, 4))
    k = rng.standard_normal((7, 2, 4))
    v = rng.standard_normal((7, 2, 4))
    out = dit.attention(q, k, v)
    np.testing.assert_allclose(out, _attention_bruteforce(q, k, v), atol=1e-13)
    ref = F.scaled_dot_product_attention(t64(q).permute(1, 0, 2), t64(k).permute(1, 0, 2),
                                         t64(v).permute(1, 0, 2)).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(out, ref, atol=1e-13)
    chunked = dit.attention(q, k, v, q_chunk=2)
    np.testing.assert_allclose(chunked, out, rtol=1e-14, atol=1e-15)


def test_attention_invariants():
    q = rng.standard_normal((6, 3, 8))
    k = rng.standard_normal((1, 3, 8))
    v = rng.standard_normal((1, 3, 8))
    np.testing.assert_allclose(dit.attention(q, k, v), np.broadcast_to(v, (6, 3, 8)), atol=1e-15)
    # adding the same vector to every key shifts each row's logits by a constant
    k = rng.standard_normal((9, 3, 8))
    v = rng.standard_normal((9, 3, 8))
    shift = rng.standard_normal((1, 3, 8))
    np.testing.assert_allclose(dit.attention(q, k + shift, v), dit.attention(q, k, v), atol=1e-12)


def test_rope_sections():
    assert dit.rope_sections(128) == (44, 42, 42)
    assert dit.rope_sections(32) == (12, 10, 10)
    assert sum(dit.rope_sections(64)) == 64


def test_rope3d_matches_complex_rotation():
    grid = (3, 4, 5)
    L, H, dh = 60, 2, 32
    x = rng.standard_normal((L, H, dh))
    y = dit.rope3d(x, grid)
    # independent statement: pairs as complex numbers times exp(i * pos * theta^(-2i/n))
    f, h, w = np.meshgrid(np.arange(3), np.arange(4), np.arange(5), indexing="ij")
    pos = [f.ravel(), h.ravel(), w.ravel()]
    z = x[..., 0::2] + 1j * x[..., 1::2]
    phases = []
    for axis, n in enumerate((12, 10, 10)):
        inv = 10000.0 ** (-np.arange(0, n, 2) / n)
        phases.append(np.outer(pos[axis], inv))
    ph = np.concatenate(phases, axis=1)[:, None, :]
    zr = z * np.exp(1j * ph)
    ref = np.empty_like(x)
    ref[..., 0::2] = zr.real
    ref[..., 1::2] = zr.imag
    np.testing.assert_allclose(y, ref, atol=1e-12)


def test_rope3d_invariants():
    grid = (2, 3, 4)
    x = rng.standard_normal((24, 1, 128))
    y = dit.rope3d(x, grid)
    np.testing.assert_allclose(y[0], x[0], atol=0)  # position (0, 0, 0) is the identity
    pair_norm = lambda a: a[..., 0::2] ** 2 + a[..., 1::2] ** 2
    np.testing.assert_allclose(pair_norm(y), pair_norm(x), rtol=1e-12)
    # relative position: <R_p q, R_p' k> depends only on p - p'
    big = (4, 4, 4)
    q = rng.standard_normal((1, 1, 128))
    k = rng.standard_normal((1, 1, 128))
    Q = dit.rope3d(np.broadcast_to(q, (64, 1, 128)).copy(), big)
    K = dit.rope3d(np.broadcast_to(k, (64, 1, 128)).copy(), big)
    idx = lambda f, h, w: (f * 4 + h) * 4 + w
    d1 = Q[idx(2, 1, 3)] @ K[idx(1, 0, 1)].T
    d2 = Q[idx(3, 3, 2)] @ K[idx(2, 2, 0)].T
    np.testing.assert_allclose(d1, d2, rtol=1e-10)


def test_patchify_roundtrip_and_conv3d():
    C, Fr, H, W = 3, 4, 6, 8
    patch = (1, 2, 2)
    x = rng.standard_normal((C, Fr, H, W))
    u = dit.patchify(x, patch)
    assert u.shape == (4 * 3 * 4, 12)
    np.testing.assert_array_equal(dit.unpatchify(u, C, Fr, H, W, patch), x)
    # a linear map of patch vectors is the stride = kernel conv3d
    d = 5
    wconv = rng.standard_normal((d, C, *patch))
    b = rng.standard_normal(d)
    ref = F.conv3d(t64(x)[None], t64(wconv), t64(b), stride=patch)[0]       # [d, F', H', W']
    ref = ref.reshape(d, -1).T.numpy()
    np.testing.assert_allclose(dit.linear(u, wconv.reshape(d, -1), b), ref, atol=1e-12)


def test_patchify_temporal_patch_roundtrip():
    x = rng.standard_normal((2, 4, 4, 6))
    for patch in [(2, 2, 2), (1, 1, 1), (2, 1, 3)]:
        u = dit.patchify(x, patch)
        np.testing.assert_array_equal(dit.unpatchify(u, 2, 4, 4, 6, patch), x)
        wconv = rng.standard_normal((3, 2, *patch))
        ref = F.conv3d(t64(x)[None], t64(wconv), stride=patch)[0].reshape(3, -1).T.numpy()
        np.testing.assert_allclose(u @ wconv.reshape(3, -1).T, ref, atol=1e-12)
