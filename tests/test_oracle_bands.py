"""Pins of the oracle's band decomposition (oracle/bands.py): an explicit DFT
with exact rational band tests on tiny latents, Parseval, pure tones whose
energy must land in one known band, and consistency with Eq. 4."""
import cmath
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import bands, sampler

rng = np.random.default_rng(31)


def _nu(k, n):
    a = k if k <= n // 2 else n - k
    return Fraction(2 * a, n)


def _band(nu_sq):
    # nu^2 < 1/9 low, < 4/9 mid, else high (exact rationals)
    return 0 if nu_sq < Fraction(1, 9) else (1 if nu_sq < Fraction(4, 9) else 2)


def test_explicit_dft_with_rational_band_tests():
    C, F, H, W = 2, 5, 4, 6
    d = rng.standard_normal((C, F, H, W))
    sp = [0.0, 0.0, 0.0]
    tp = [0.0, 0.0, 0.0]
    for c in range(C):
        for f in range(F):
            for kh in range(H):
                for kw in range(W):
                    z = sum(d[c, f, h, w] * cmath.exp(-2j * math.pi * (kh * h / H + kw * w / W))
                            for h in range(H) for w in range(W)) / math.sqrt(H * W)
                    sp[_band(_nu(kh, H) ** 2 + _nu(kw, W) ** 2)] += abs(z) ** 2
        for h in range(H):
            for w in range(W):
                for kf in range(F):
                    z = sum(d[c, f, h, w] * cmath.exp(-2j * math.pi * kf * f / F) for f in range(F)) / math.sqrt(F)
                    tp[_band(_nu(kf, F) ** 2)] += abs(z) ** 2
    s, t = bands.band_energies(d)
    np.testing.assert_allclose(s, sp, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(t, tp, rtol=1e-12, atol=1e-12)


def test_band_maps_match_rational_definition():
    for H, W in [(60, 104), (7, 9), (1, 1), (2, 3), (90, 160)]:
        sb = bands.spatial_bands(H, W)
        for kh in range(H):
            for kw in range(W):
                assert sb[kh, kw] == _band(_nu(kh, H) ** 2 + _nu(kw, W) ** 2)
    for n in [1, 2, 3, 4, 6, 21, 31, 100]:
        assert list(bands.axis_bands(n)) == [_band(_nu(k, n) ** 2) for k in range(n)]


def test_parseval_both_decompositions():
    d = rng.standard_normal((3, 7, 10, 12))
    s, t = bands.band_energies(d)
    tot = float(np.sum(d * d))
    assert s.sum() == pytest.approx(tot, rel=1e-12)
    assert t.sum() == pytest.approx(tot, rel=1e-12)


@pytest.mark.parametrize("a,b", [(0, 0), (1, 2), (5, 9), (10, 17), (20, 30), (29, 51), (30, 52)])
def test_spatial_tone_lands_in_its_band(a, b):
    C, F, H, W = 2, 3, 60, 104
    h = np.arange(H)[:, None]
    w = np.arange(W)[None, :]
    tone = np.cos(2 * np.pi * (a * h / H + b * w / W))
    d = np.broadcast_to(tone, (C, F, H, W))
    s, t = bands.band_energies(d)
    band = _band(_nu(a, H) ** 2 + _nu(b, W) ** 2)
    nyq = (a in (0, H // 2)) and (b in (0, W // 2))  # a real tone at DC / Nyquist has full energy
    expect = C * F * H * W * (1.0 if nyq else 0.5)
    assert s[band] == pytest.approx(expect, rel=1e-10)
    assert s.sum() == pytest.approx(expect, rel=1e-10)
    # constant over frames: all temporal energy at frequency 0 (low band)
    assert t[0] == pytest.approx(expect, rel=1e-10) and t[1] == pytest.approx(0, abs=1e-8) and t[2] == pytest.approx(0, abs=1e-8)


@pytest.mark.parametrize("m", [0, 1, 3, 4, 7, 10])
def test_temporal_tone_lands_in_its_band(m):
    C, F, H, W = 2, 21, 6, 8
    f = np.arange(F)[None, :, None, None]
    d = np.broadcast_to(np.sin(2 * np.pi * m * f / F + 0.3), (C, F, H, W))
    s, t = bands.band_energies(d)
    band = _band(_nu(m, F) ** 2)
    tot = float(np.sum(d * d))
    assert t[band] == pytest.approx(tot, rel=1e-10)
    # constant over space: all spatial energy at (0, 0)
    assert s[0] == pytest.approx(tot, rel=1e-10)


def test_band_scores_square_sum_to_r_and_zero_prediction():
    pL = rng.standard_normal((4, 5, 6, 8))
    pS = pL + 0.1 * rng.standard_normal(pL.shape)
    rb = bands.band_disagreement(pS, pL, 1e-8)
    r = sampler.relative_disagreement(pS, pL, 1e-8)
    assert float(np.sum(rb[:3] ** 2)) == pytest.approx(r * r, rel=1e-12)
    assert float(np.sum(rb[3:] ** 2)) == pytest.approx(r * r, rel=1e-12)
    # p_L = 0: the denominator becomes eps
    z = np.zeros_like(pL)
    rb0 = bands.band_disagreement(pS, z, 1e-8)
    assert float(np.sqrt(np.sum(rb0[:3] ** 2))) == pytest.approx(float(np.linalg.norm(pS)) / 1e-8, rel=1e-12)


def test_calibrate_bands_closed_form():
    # L: p = x, S: p = x + c0 with c0 a pure temporal tone of frequency index 4
    # of 12 frames (nu = 2/3: high band) that is constant in space.  On the
    # all-large path every step's difference is c0, so the temporal high band
    # carries all of r and the spatial low band (frequency (0, 0)) does too.
    from paper_2609_30096_amd import synth
    scfg = synth.SamplerConfig(steps=5, shift=2.0, guidance=1.0, use_cfg=False)
    F = 12
    c0 = np.broadcast_to(np.cos(2 * np.pi * 4 * np.arange(F) / F)[None, :, None, None], (2, F, 4, 4)).copy()
    den = lambda params, cfg, x, t, c: x + (c0 if params == "S" else 0.0)
    xs = [rng.standard_normal(c0.shape) for _ in range(2)]
    r, q, rb, qb = bands.calibrate_bands(("L", None), ("S", None), xs, [None] * 2, None, scfg, den)
    r2, q2 = sampler.calibrate(("L", None), ("S", None), xs, [None] * 2, None, scfg, den)
    np.testing.assert_array_equal(r, r2)
    np.testing.assert_array_equal(q, q2)
    np.testing.assert_allclose(rb[..., 0], r, rtol=1e-12)  # spatial low
    np.testing.assert_allclose(rb[..., 5], r, rtol=1e-12)  # temporal high
    np.testing.assert_allclose(rb[..., [1, 2, 3, 4]], 0, atol=1e-12 * float(r.max()))
    np.testing.assert_allclose(qb, rb.mean(axis=0), rtol=1e-15)
