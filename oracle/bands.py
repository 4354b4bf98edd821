"""Oracle for the frequency-band decomposition of the calibration disagreement;
float64, numpy.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper passage followed: Sec. "Frequency Analysis" (and its appendix figures)
decomposes the disagreement between the two models' guided predictions over
spatial and latent-temporal frequency bands (low, mid, high) with an
orthonormal Fourier transform.

Readings where the paper is silent:
  * the decomposed quantity is d = p_S - p_L of Eq. 4 on the C x F x H x W
    latent (guided predictions, as in Eq. 4);
  * spatial: a 2D orthonormal DFT over (H, W) of every (c, f) slice;
    temporal: a 1D orthonormal DFT over F of every (c, h, w) series;
  * the normalised frequency of index k on an axis of length n is
    nu = 2 |k'| / n with k' = k for k <= n / 2 and k - n above (so nu = 1 is
    the Nyquist frequency); the spatial nu is the radius
    sqrt(nu_h^2 + nu_w^2), the temporal nu is nu_f;
  * bands are equal thirds of the Nyquist range: low nu < 1/3,
    mid 1/3 <= nu < 2/3, high nu >= 2/3 (spatial radii above 1, the corners of
    the spectrum, are high);
  * a band's score is ||P_b d||_2 / max(||p_L||_2, eps), P_b the orthogonal
    projection onto the band, so the squares of the three spatial (or the
    three temporal) scores add up to r^2 of Eq. 4; per step the scores are
    averaged over the calibration samples like Eq. 5.
"""
from __future__ import annotations

import numpy as np

from . import dit, sampler


def folded(n):
    """|k'| for k = 0..n-1: the distance of each DFT index from frequency 0."""
    k = np.arange(n)
    return np.where(k <= n // 2, k, n - k)


def axis_bands(n):
    """Band (0 low, 1 mid, 2 high) of each frequency index of an axis of length n.

    nu = 2a/n < 1/3  <=>  6a < n;   nu < 2/3  <=>  3a < n   (integer tests).
    """
    a = folded(n)
    return np.where(6 * a < n, 0, np.where(3 * a < n, 1, 2))


def spatial_bands(H, W):
    """Band of each (k_h, k_w): nu^2 = 4 (a_h^2 / H^2 + a_w^2 / W^2), compared in integers."""
    ah = folded(H).astype(np.int64)[:, None]
    aw = folded(W).astype(np.int64)[None, :]
    s = ah * ah * W * W + aw * aw * H * H  # (nu / 2)^2 H^2 W^2
    hw2 = H * H * W * W
    # nu < 1/3 <=> 36 s < H^2 W^2;  nu < 2/3 <=> 9 s < H^2 W^2
    return np.where(36 * s < hw2, 0, np.where(9 * s < hw2, 1, 2))


def band_energies(d):
    """Energies ||P_b d||^2 of a latent d [C, F, H, W]: (spatial [3], temporal [3])."""
    d = np.asarray(d, np.float64)
    _, F, H, W = d.shape
    Xs = np.fft.fft2(d, axes=(2, 3), norm="ortho")
    Ps = (Xs.real ** 2 + Xs.imag ** 2).sum(axis=(0, 1))  # [H, W]
    sb = spatial_bands(H, W)
    Xt = np.fft.fft(d, axis=1, norm="ortho")
    Pt = (Xt.real ** 2 + Xt.imag ** 2).sum(axis=(0, 2, 3))  # [F]
    tb = axis_bands(F)
    spatial = np.array([Ps[sb == b].sum() for b in range(3)])
    temporal = np.array([Pt[tb == b].sum() for b in range(3)])
    return spatial, temporal


def band_disagreement(p_small, p_large, eps):
    """Six band scores of d = p_S - p_L: spatial low, mid, high, temporal low, mid, high."""
    p_small = np.asarray(p_small, np.float64)
    p_large = np.asarray(p_large, np.float64)
    sp, tp = band_energies(p_small - p_large)
    den = max(float(np.sqrt(np.sum(p_large * p_large))), eps)
    return np.sqrt(np.concatenate([sp, tp])) / den


def calibrate_bands(large, small, x_T, conds, uncond, scfg, denoise=dit.dit_forward):
    """Reference-trajectory calibration with the band decomposition.

    Returns r [M, N], q [N] (as sampler.calibrate), the band scores
    rb [M, N, 6] and their per-step means qb [N, 6].
    """
    sig = sampler.sigmas(scfg.steps, scfg.shift)
    M, N = len(x_T), scfg.steps
    r = np.zeros((M, N), dtype=np.float64)
    rb = np.zeros((M, N, 6), dtype=np.float64)
    for j in range(M):
        sched = sampler.scheduler(scfg, sig)
        x = np.asarray(x_T[j], np.float64)
        for k in range(N):
            t = 1000.0 * sig[k]
            p_L = sampler.guided_prediction(large, x, t, conds[j], uncond, scfg, denoise)
            p_S = sampler.guided_prediction(small, x, t, conds[j], uncond, scfg, denoise)
            r[j, k] = sampler.relative_disagreement(p_S, p_L, scfg.eps)
            rb[j, k] = band_disagreement(p_S, p_L, scfg.eps)
            x = sched(k, x, p_L)
    qb = np.zeros((N, 6), dtype=np.float64)
    for j in range(M):
        qb += rb[j]
    return r, sampler.mean_score(r), rb, qb / M
