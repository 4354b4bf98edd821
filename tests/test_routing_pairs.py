"""The structured pairs used for routing parity have score maps that can tell
a right routing from a wrong one: pinned on the oracle, host only."""
import dataclasses

import numpy as np

from oracle import sampler
from paper_2609_30096_amd import synth
from structured_pairs import TIMESTEP_SHIFT_BF16, TIMESTEP_SHIFT_F32, boundary_gaps, score_tolerance, timestep_pair

BF_PAIR = synth.DiTConfig(blocks=2, dim=256, heads=2, head_dim=128, ffn_dim=512, text_dim=256)
BF_LATENT = synth.LatentShape(16, 3, 10, 14, 7)
SAMPLER8 = synth.SamplerConfig(steps=8, shift=3.0, guidance=5.0)


def _q(cfg, shape, alpha, M=4):
    pL = synth.gen_params(cfg, synth.SEED_LARGE)
    pS = timestep_pair(cfg, pL, alpha)
    xs = [synth.gen_latent(shape, j) for j in range(M)]
    cs = [synth.gen_text(shape, cfg.text_dim, j, cfg.dtype) for j in range(M)]
    u = synth.gen_null_text(shape, cfg.text_dim, cfg.dtype)
    return sampler.calibrate((pL, cfg), (pS, cfg), xs, cs, u, SAMPLER8)


def test_score_tolerance_bound_holds_for_planted_errors():
    # velocities with planted relative errors of size delta stay within the stated score bound
    rng = np.random.default_rng(5)
    for delta in (1e-4, 2e-2):
        for _ in range(200):
            pL = rng.standard_normal(64)
            pS = pL + rng.uniform(0, 3) * rng.standard_normal(64)
            eL = rng.standard_normal(64)
            eS = rng.standard_normal(64)
            eL *= delta * np.linalg.norm(pL) / np.linalg.norm(eL)
            eS *= delta * np.linalg.norm(pS) / np.linalg.norm(eS)
            r = sampler.relative_disagreement(pS, pL, 1e-8)
            r2 = sampler.relative_disagreement(pS + eS, pL + eL, 1e-8)
            assert abs(r2 - r) <= score_tolerance(r, delta)


def test_timestep_pair_float32_scores_resolve_every_boundary():
    r, q = _q(synth.TINY_LARGE, synth.TINY_LATENT, TIMESTEP_SHIFT_F32)
    gaps = boundary_gaps(q, 1e-4)
    assert all(g > 10 * tol for _, g, tol in gaps), gaps
    # non-monotone in the step index: the K lowest are neither the first K nor the last K
    top = set(sampler.route_topk(q, 4).tolist())
    assert top not in ({0, 1, 2, 3}, {4, 5, 6, 7})


def test_timestep_pair_bf16_scores_resolve_the_routed_boundaries():
    cfg = BF_PAIR
    r, q = _q(cfg, BF_LATENT, TIMESTEP_SHIFT_BF16)
    gaps = dict((K, (g, tol)) for K, g, tol in boundary_gaps(q, 2e-2))
    for K in (2, 4):
        g, tol = gaps[K]
        assert g > 2 * tol, (K, g, tol)
