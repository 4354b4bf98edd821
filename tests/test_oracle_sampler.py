"""Pins of the oracle's scheduler, guidance, scores, routing and sampling.

Closed forms, invariants, brute force and hand-written fixtures (tests/golden)
tie oracle/sampler.py to the paper's equations rather than to itself.
"""
import dataclasses
import itertools
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import dit, sampler
from paper_2609_30096_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
rng = np.random.default_rng(99)


# ------------------------------------------------------------------ sigma table
def test_sigmas_golden_fractions():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "sigmas_n8_shift3.txt")) if l.strip() and l[0] != "#"]
    sig = sampler.sigmas(8, 3.0)
    assert len(sig) == len(rows) == 9
    for i, num, den in rows:
        assert sig[int(i)] == pytest.approx(float(Fraction(int(num), int(den))), abs=1e-15)


def test_sigmas_shift1_is_linear_and_monotone():
    np.testing.assert_allclose(sampler.sigmas(50, 1.0), 1 - np.arange(51) / 50, atol=1e-15)
    for N, s in [(4, 5.0), (50, 5.0), (8, 3.0)]:
        sig = sampler.sigmas(N, s)
        assert sig[0] == 1.0 and sig[-1] == 0.0
        assert np.all(np.diff(sig) < 0)
        assert np.sum(np.diff(sig)) == pytest.approx(-1.0, abs=1e-14)
    t = sampler.timesteps(8, 3.0)
    assert len(t) == 8 and t[0] == 1000.0 and np.all(np.diff(t) < 0)


# ------------------------------------------------------------------ Euler
def _field(fn):
    """A closed-form 'denoiser' f(params, cfg, x, t, c) = fn(x, t, c)."""
    return lambda params, cfg, x, t, c: fn(x, t, c)


def test_euler_exact_on_constant_velocity():
    scfg = synth.SamplerConfig(steps=8, shift=3.0, guidance=1.0, use_cfg=False)
    v = rng.standard_normal((2, 3, 4, 4))
    x_T = rng.standard_normal((2, 3, 4, 4))
    den = _field(lambda x, t, c: v)
    x0 = sampler.sample(np.zeros(8, bool), (None, None), (None, None), x_T, None, None, scfg, den)
    # sum of the steps telescopes to sigma_N - sigma_0 = -1
    np.testing.assert_allclose(x0, x_T - v, atol=8 * np.finfo(np.float64).eps * 4)


def test_euler_point_mass_lands_on_target():
    # v(x, sigma) = (x - mu)/sigma is the exact flow of a point mass at mu; every
    # Euler step stays on the straight path, so x_N = mu after any N.
    scfg = synth.SamplerConfig(steps=7, shift=2.5, guidance=1.0, use_cfg=False)
    mu = rng.standard_normal((3, 2, 2, 2))
    x_T = rng.standard_normal((3, 2, 2, 2))
    den = _field(lambda x, t, c: (x - mu) / (t / 1000.0))
    x0 = sampler.sample(np.zeros(7, bool), (None, None), (None, None), x_T, None, None, scfg, den)
    np.testing.assert_allclose(x0, mu, atol=1e-12)


# ------------------------------------------------------------------ CFG (Eq. 1)
def test_guidance_special_cases():
    c = rng.standard_normal(1000)
    u = rng.standard_normal(1000)
    np.testing.assert_array_equal(sampler.guided(c, u, 0.0), u)
    err = np.abs(sampler.guided(c, u, 1.0) - c)
    assert np.all(err <= np.spacing(np.maximum(np.abs(c), np.abs(u))) * 2)
    # affine in w
    g = [sampler.guided(c, u, w) for w in (0.0, 2.0, 5.0)]
    np.testing.assert_allclose(g[2], g[0] + 2.5 * (g[1] - g[0]), atol=1e-12)
    # w scales the conditional direction
    np.testing.assert_allclose(sampler.guided(c, u, 5.0) - u, 5.0 * (c - u), atol=1e-12)


def test_guided_prediction_uses_both_branches():
    scfg = synth.SamplerConfig(steps=4, shift=1.0, guidance=3.0)
    den = _field(lambda x, t, c: x * c)
    x = rng.standard_normal(10)
    p = sampler.guided_prediction((None, None), x, 0.0, 2.0, 0.5, scfg, den)
    np.testing.assert_allclose(p, 0.5 * x + 3.0 * (2.0 * x - 0.5 * x))
    p1 = sampler.guided_prediction((None, None), x, 0.0, 2.0, 0.5, dataclasses.replace(scfg, use_cfg=False), den)
    np.testing.assert_allclose(p1, 2.0 * x)


# ------------------------------------------------------------------ r (Eq. 4), q (Eq. 5)
def test_relative_disagreement_pins():
    pL = rng.standard_normal((4, 5, 6))
    assert sampler.relative_disagreement(pL, pL, 1e-8) == 0.0
    assert sampler.relative_disagreement(np.zeros_like(pL), pL, 1e-8) == pytest.approx(1.0, abs=1e-15)
    for a in (0.3, -0.7, 2.0):
        assert sampler.relative_disagreement((1 + a) * pL, pL, 1e-8) == pytest.approx(abs(a), rel=1e-13)
    pS = rng.standard_normal(pL.shape)
    r = sampler.relative_disagreement(pS, pL, 1e-8)
    assert sampler.relative_disagreement(7.5 * pS, 7.5 * pL, 1e-8) == pytest.approx(r, rel=1e-13)
    # the norm is over the whole latent: a 2-element example by hand
    assert sampler.relative_disagreement(np.array([[3.0], [4.0]]), np.array([[0.0], [1.0]]), 1e-8) == \
        pytest.approx(math.sqrt(9 + 9) / 1.0, rel=1e-15)
    # eps binds only when ||p_L|| < eps
    assert sampler.relative_disagreement(pS, np.zeros_like(pS), 1e-8) == \
        pytest.approx(np.linalg.norm(pS) / 1e-8, rel=1e-13)


def test_mean_score_pins():
    r = rng.random((5, 9))
    np.testing.assert_array_equal(sampler.mean_score(r[:1]), r[0])
    np.testing.assert_allclose(sampler.mean_score(r[::-1]), sampler.mean_score(r), rtol=1e-15)
    np.testing.assert_allclose(sampler.mean_score(r), r.mean(axis=0), rtol=1e-15)


# ------------------------------------------------------------------ routing (Eqs. 6-7, top-K)
def test_topk_golden():
    for line in open(os.path.join(GOLDEN, "topk_cases.txt")):
        if not line.strip() or line[0] == "#":
            continue
        k, q, exp = [p.split() for p in line.split("|")]
        got = sampler.route_topk([float(v) for v in q], int(k[0]))
        assert list(got) == [int(v) for v in exp], line


def test_topk_equals_bruteforce_and_threshold():
    for trial in range(20):
        N = 8
        q = rng.random(N)
        W = q ** 2
        for K in range(N + 1):
            sel = sampler.route_topk(q, K)
            best, args = sampler.route_bruteforce(q, K)
            assert tuple(sel) in args
            assert sum(W[sel]) == pytest.approx(best, abs=1e-15)
            # Eq. 7 with C_0 between the K-th and (K+1)-th smallest W selects the same set
            Ws = np.sort(W)
            lo = Ws[K - 1] if K > 0 else -1.0
            hi = Ws[K] if K < N else Ws[-1] + 1.0
            C0 = 0.5 * (lo + hi)
            beta = sampler.threshold_solution(W, C0)
            assert list(np.nonzero(beta)[0]) == list(sel)
            # and that beta minimises the LP objective over every vertex of the box
            obj = sampler.lp_objective(W, C0, beta)
            for bits in itertools.product([0, 1], repeat=N):
                assert obj <= sampler.lp_objective(W, C0, np.array(bits)) + 1e-15


def test_topk_bounds():
    q = rng.random(6)
    assert len(sampler.route_topk(q, 0)) == 0
    assert list(sampler.route_topk(q, 6)) == list(range(6))
    with pytest.raises(ValueError):
        sampler.route_topk(q, 7)
    with pytest.raises(ValueError):
        sampler.route_topk(q, -1)


# ------------------------------------------------------------------ calibration and routed sampling
def _linear_models(a_L, a_S):
    """Models whose prediction is a_m * x (independent of t and conditioning)."""
    den = lambda params, cfg, x, t, c: params * x
    return (a_L, None), (a_S, None), den


def test_calibrate_closed_form_scaled_pair():
    scfg = synth.SamplerConfig(steps=6, shift=3.0, guidance=5.0)
    L, S, den = _linear_models(1.0, 1.4)
    xs = [rng.standard_normal((2, 2, 4, 4)) for _ in range(3)]
    r, q = sampler.calibrate(L, S, xs, [None] * 3, None, scfg, den)
    np.testing.assert_allclose(r, 0.4, rtol=1e-13)
    np.testing.assert_allclose(q, 0.4, rtol=1e-13)


def test_calibrate_advances_with_large_model():
    # L: p = x, S: p = x + c0.  On the all-large path x_k = x_T prod_{i<k}(1 + dsigma_i),
    # so r_{j,k} = ||c0|| / ||x_k||; advancing with S would give another path.
    scfg = synth.SamplerConfig(steps=5, shift=2.0, guidance=1.0, use_cfg=False)
    c0 = rng.standard_normal((2, 3, 4, 4))
    den = lambda params, cfg, x, t, c: x + (c0 if params == "S" else 0.0)
    xs = [rng.standard_normal(c0.shape) for _ in range(2)]
    r, q = sampler.calibrate(("L", None), ("S", None), xs, [None] * 2, None, scfg, den)
    sig = sampler.sigmas(5, 2.0)
    for j in range(2):
        fac = 1.0
        for k in range(5):
            assert r[j, k] == pytest.approx(np.linalg.norm(c0) / (abs(fac) * np.linalg.norm(xs[j])), rel=1e-12)
            fac *= 1 + (sig[k + 1] - sig[k])
    np.testing.assert_allclose(q, r.mean(axis=0), rtol=1e-15)


def test_routed_sample_closed_form():
    # Eq. 3 with p_m = a_m x: x_N = x_T prod_i (1 + dsigma_i a_{pi(i)})
    scfg = synth.SamplerConfig(steps=8, shift=3.0, guidance=5.0)
    L, S, den = _linear_models(-0.9, -1.3)
    x_T = rng.standard_normal((2, 2, 2, 2))
    sig = sampler.sigmas(8, 3.0)
    for use_small in [np.zeros(8, bool), np.ones(8, bool), sampler.policy_from_indices(8, [1, 2, 5, 6])]:
        x0 = sampler.sample(use_small, L, S, x_T, None, None, scfg, den)
        fac = np.prod([1 + (sig[i + 1] - sig[i]) * (-1.3 if use_small[i] else -0.9) for i in range(8)])
        np.testing.assert_allclose(x0, fac * x_T, rtol=1e-13)


def _tiny_pair():
    L = synth.TINY_LARGE
    S = synth.TINY_SMALL
    return (synth.gen_params(L, synth.SEED_LARGE), L), (synth.gen_params(S, synth.SEED_SMALL), S)


def test_dit_pair_k0_matches_all_large_path_and_self_disagreement_is_zero():
    shape = synth.TINY_LATENT
    scfg = dataclasses.replace(synth.TINY_SAMPLER, steps=3)
    large, small = _tiny_pair()
    x_T = synth.gen_latent(shape, 0)
    cond = synth.gen_text(shape, 128, 0)
    unc = synth.gen_null_text(shape, 128)
    r_self, _ = sampler.calibrate(large, large, [x_T], [cond], unc, scfg)
    assert np.all(r_self == 0.0)
    # K = 0 (all-large) equals the path the calibration advanced along
    x_all_L, path = sampler.sample(np.zeros(3, bool), large, small, x_T, cond, unc, scfg, return_path=True)
    sig = sampler.sigmas(3, scfg.shift)
    x = np.asarray(x_T, np.float64)
    for k in range(3):
        p = sampler.guided_prediction(large, x, 1000 * sig[k], cond, unc, scfg)
        x = sampler.euler_step(x, p, sig[k], sig[k + 1])
        np.testing.assert_array_equal(x, path[k + 1])
    # the prefix before the first small step is the all-large prefix
    _, path2 = sampler.sample(np.array([False, True, False]), large, small, x_T, cond, unc, scfg, return_path=True)
    np.testing.assert_array_equal(path2[1], path[1])
    assert not np.array_equal(path2[2], path[2])


def test_dit_scaled_head_pair_gives_constant_r():
    cfg = synth.TINY_LARGE
    params = synth.gen_params(cfg, synth.SEED_LARGE)
    scaled = dict(params)
    scaled["head.w"] = params["head.w"].astype(np.float64) * 1.3
    scaled["head.b"] = params["head.b"].astype(np.float64) * 1.3
    shape = synth.TINY_LATENT
    scfg = dataclasses.replace(synth.TINY_SAMPLER, steps=3)
    r, q = sampler.calibrate((params, cfg), (scaled, cfg), [synth.gen_latent(shape, 0)],
                             [synth.gen_text(shape, 128, 0)], synth.gen_null_text(shape, 128), scfg)
    np.testing.assert_allclose(r, 0.3, rtol=1e-10)


# ------------------------------------------------------------------ C_0 threshold form and baseline policies
def test_route_threshold_selects_topk_between_order_statistics():
    # the paper's equivalence: a C_0 strictly between the K-th and (K+1)-th
    # smallest W_k selects exactly the top-K steps
    for N in (1, 5, 50):
        q = rng.uniform(0.05, 2.0, N)
        W = np.sort(q ** 2)
        for K in range(N + 1):
            lo = W[K - 1] if K > 0 else 0.0
            hi = W[K] if K < N else W[-1] * 2 + 1
            C0 = 0.5 * (lo + hi)
            np.testing.assert_array_equal(sampler.route_threshold(q, C0), sampler.route_topk(q, K))


def test_route_threshold_minimises_the_box_lp_over_all_vertices():
    N = 8
    q = rng.uniform(0.1, 1.5, N)
    W = q ** 2
    for C0 in (0.0, float(np.median(W)), float(W.max()) + 1.0, float(W[3])):
        beta = np.zeros(N)
        beta[sampler.route_threshold(q, C0)] = 1.0
        best = min(sampler.lp_objective(W, C0, np.array(v, float)) for v in itertools.product((0, 1), repeat=N))
        assert sampler.lp_objective(W, C0, beta) == pytest.approx(best, abs=1e-12)
    # at W_k = C_0 the step stays on the large model (either choice is optimal)
    assert 3 not in sampler.route_threshold(q, float(W[3]))


def test_first_and_last_k():
    for N, K in [(1, 0), (1, 1), (50, 25), (4, 2), (7, 7)]:
        f, l = sampler.first_k(N, K), sampler.last_k(N, K)
        assert list(f) == list(range(K)) and list(l) == list(range(N - K, N))
        assert sorted(set(sampler.first_k(N, K)) | set(sampler.last_k(N, N - K))) == list(range(N))
        assert not set(sampler.first_k(N, K)) & set(sampler.last_k(N, N - K))
    with pytest.raises(ValueError):
        sampler.first_k(3, 4)
    with pytest.raises(ValueError):
        sampler.last_k(3, -1)


def test_splitmix64_reference_outputs():
    # the generator's published output sequence for seed 0
    expect = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F, 0xF88BB8A8724C81EC, 0x1B39896A51A8749B]
    state = 0
    for e in expect:
        state, z = sampler.splitmix64(state)
        assert z == e


def test_random_k_is_a_uniform_k_subset():
    for N, K in [(1, 1), (50, 25), (4, 0), (4, 4), (9, 3)]:
        idx = sampler.random_k(N, K, 12345)
        assert len(idx) == K and len(set(idx)) == K and list(idx) == sorted(idx)
        assert all(0 <= i < N for i in idx)
        np.testing.assert_array_equal(idx, sampler.random_k(N, K, 12345))
    # all 6 subsets of 2 out of 4 steps are about equally likely (6000 seeds:
    # each count ~ Binomial(6000, 1/6), sd ~ 29)
    counts = {}
    for seed in range(6000):
        key = tuple(sampler.random_k(4, 2, seed))
        counts[key] = counts.get(key, 0) + 1
    assert len(counts) == 6
    assert all(abs(c - 1000) < 150 for c in counts.values()), counts
