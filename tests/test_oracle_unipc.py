"""Pins of the oracle's UniPC scheduler (oracle/unipc.py): its first-order
case is the Euler step, it is exact on a point mass, its weights reduce to
the Adams-Bashforth / Adams-Moulton coefficients for small uniform steps,
and its one-step errors on a Gaussian-data flow (whose ODE solution is known
in closed form) shrink at the rates of the stated orders."""
import math

import numpy as np
import pytest

from oracle import sampler, unipc
from paper_2609_30096_amd import synth

rng = np.random.default_rng(17)

MU, S2 = 0.7, 0.3 ** 2


def gauss_velocity(x, sig):
    """Flow-matching velocity for data N(MU, S2): p = (x - E[x_0 | x]) / sigma."""
    k = (1 - sig) * S2 / ((1 - sig) ** 2 * S2 + sig ** 2)
    m = MU + k * (x - (1 - sig) * MU)
    return (x - m) / sig


def gauss_path(sig, z):
    """The probability-flow ODE solution through x(1) = z."""
    return (1 - sig) * MU + math.sqrt((1 - sig) ** 2 * S2 + sig ** 2) * z


def test_first_order_without_corrector_is_euler():
    for N, shift in [(8, 3.0), (50, 5.0), (1, 1.0)]:
        sig = sampler.sigmas(N, shift)
        S = unipc.UniPC(sig, order=1, corrector=False)
        x = rng.standard_normal(5)
        for i in range(N):
            p = rng.standard_normal(5)
            got = S.step(i, x, p)
            ref = sampler.euler_step(x, p, sig[i], sig[i + 1])
            np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
            x = ref


@pytest.mark.parametrize("order", [1, 2, 3])
@pytest.mark.parametrize("N,shift", [(1, 1.0), (2, 3.0), (5, 3.0), (50, 5.0)])
def test_point_mass_lands_exactly(order, N, shift):
    # data = a point mass mu: the data prediction is mu everywhere, every
    # history difference vanishes and each update stays on the straight path
    mu = rng.standard_normal(4)
    sig = sampler.sigmas(N, shift)
    S = unipc.UniPC(sig, order=order)
    x = rng.standard_normal(4)
    for i in range(N):
        x = S.step(i, x, (x - mu) / sig[i])
        assert np.all(np.isfinite(x))
    np.testing.assert_allclose(x, mu, rtol=0, atol=1e-12)


def test_small_step_weights_are_adams_coefficients():
    # h = 1e-3: the deviation from the limit is O(h), and the series recursion
    # for b loses digits to cancellation as h -> 0 (about eps / h^2 at order 3)
    h = 1e-3
    # predictor, order 3, history at r = -1, -2: Adams-Bashforth 3 (23, -16, 5) / 12
    rho = unipc.rho_weights([-1.0, -2.0], h, predictor=True)
    np.testing.assert_allclose([1 + rho[0] + rho[1] / 2, -rho[0], -rho[1] / 2], [23 / 12, -16 / 12, 5 / 12], atol=2e-3)
    # predictor, order 2 (rho = 1/2): Adams-Bashforth 2 (3, -1) / 2
    rho = unipc.rho_weights([-1.0], h, predictor=True)
    np.testing.assert_allclose([1 + rho[0], -rho[0]], [1.5, -0.5], atol=1e-12)
    # corrector, order 1 (rho = 1/2): trapezoid
    np.testing.assert_allclose(unipc.rho_weights([1.0], h, predictor=False), [0.5])
    # corrector, order 2: Adams-Moulton 3 (5, 8, -1) / 12 on (new, base, previous)
    rho = unipc.rho_weights([-1.0, 1.0], h, predictor=False)
    np.testing.assert_allclose([rho[1], 1 - rho[1] + rho[0], -rho[0]], [5 / 12, 8 / 12, -1 / 12], atol=2e-3)
    # corrector, order 3: Adams-Moulton 4 (9, 19, -5, 1) / 24
    rho = unipc.rho_weights([-1.0, -2.0, 1.0], h, predictor=False)
    np.testing.assert_allclose([rho[2], 1 - rho[2] + rho[0] + rho[1] / 2, -rho[0], -rho[1] / 2],
                               [9 / 24, 19 / 24, -5 / 24, 1 / 24], atol=2e-3)


@pytest.mark.parametrize("order,corrector,min_ratio", [
    (2, False, 100),   # UniP-2, local error O(h^3): 64 expected over two halvings
    (3, False, 200),   # UniP-3, O(h^4): 256
    (1, True, 100),    # UniC-1 (order 2)
    (2, True, 200),    # UniC-2 (order 3)
    (3, True, 120),    # UniC-3 behind lower-order warm-up correctors
])
def test_one_step_error_rates_on_gaussian_flow(order, corrector, min_ratio):
    # teacher-forced: the exact solution is fed in at lambda-uniform points;
    # a wrong weight, sign or series term drops these ratios to about 16-70
    z = np.array([1.3, -0.4, 0.05])
    errs = []
    for h in (0.2, 0.05):
        lam = -1.0 + h * np.arange(8)
        sig = list(1 / (1 + np.exp(lam)))
        S = unipc.UniPC(sig, order=order, corrector=corrector)
        for i in range(5):
            xe = gauss_path(sig[i], z)
            xn = S.step(i, xe, gauss_velocity(xe, sig[i]))
        e = xn - gauss_path(sig[5], z) if not corrector else S.x_last - gauss_path(sig[4], z)
        errs.append(float(np.abs(e).max()))
    assert errs[0] / errs[1] > min_ratio, errs


def test_last_step_returns_the_data_prediction_and_first_step_is_euler():
    N = 6
    sig = sampler.sigmas(N, 3.0)
    S = unipc.UniPC(sig, order=2)
    x = rng.standard_normal(3)
    x0 = x.copy()
    for i in range(N):
        p = gauss_velocity(x, sig[i])
        xn = S.step(i, x, p)
        if i == 0:
            np.testing.assert_allclose(xn, sampler.euler_step(x0, p, sig[0], sig[1]), rtol=1e-14, atol=1e-14)
        if i == N - 1:
            np.testing.assert_array_equal(xn, x - sig[i] * p)  # sigma_N = 0: x_N = m_{N-1}
        x = xn


def test_unipc_beats_euler_on_gaussian_flow():
    z = np.array([1.3, -0.4, 0.05])
    exact = MU + math.sqrt(S2) * z
    # the uncorrected last step into sigma = 0 dominates at large shift
    for shift, factor in ((1.0, 8.0), (5.0, 2.0)):
        sig = sampler.sigmas(40, shift)
        err = {}
        for name, order in [("euler", 1), ("unipc", 2)]:
            scfg = synth.SamplerConfig(steps=40, shift=shift, guidance=1.0, use_cfg=False, solver=name, order=order)
            step = sampler.scheduler(scfg, sig)
            x = z.copy()
            for i in range(40):
                x = step(i, x, gauss_velocity(x, sig[i]))
            err[name] = float(np.abs(x - exact).max())
        assert err["unipc"] < err["euler"] / factor, err


def test_history_is_kept_across_model_switches():
    # with S and L the same function every policy must reproduce the all-large
    # path bit for bit; a history reset at a switch would change the result
    scfg = synth.SamplerConfig(steps=9, shift=3.0, guidance=1.0, use_cfg=False, solver="unipc", order=3)
    den = lambda params, cfg, x, t, c: gauss_velocity(x, t / 1000.0)
    x_T = rng.standard_normal((2, 3, 4, 4))
    ref = sampler.sample(np.zeros(9, bool), ("L", None), ("S", None), x_T, None, None, scfg, den)
    for pol in [np.arange(9) % 2 == 0, np.arange(9) >= 5, np.ones(9, bool)]:
        got = sampler.sample(pol, ("L", None), ("S", None), x_T, None, None, scfg, den)
        np.testing.assert_array_equal(got, ref)
