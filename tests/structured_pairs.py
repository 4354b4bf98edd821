"""Model pairs with a known structure, built from the seeded recipe, and the
score tolerance that routing parity is judged by.

``timestep_pair``: the small model is the large model with one column of
its timestep MLP's first layer moved, the column that reads cos(omega_j t)
of the sinusoidal features.  The two models then differ by a first-layer
offset proportional to cos(omega_j t), so their disagreement (Eq. 4) rises
and falls with the step's timestep instead of being nearly the same at
every step, as it is for two unrelated random models.  Frequency 72 of 128
(omega = 10^(-4 * 72 / 128)) puts the |cos| of the eight timesteps of the
8-step, shift-3 table at well separated, non-monotone values, so the top-K
sets are neither first-K nor last-K and every boundary between consecutive
scores is wide.
"""
import numpy as np

from paper_2609_30096_amd import synth

TIMESTEP_FREQ = 72
TIMESTEP_SHIFT_F32 = 50.0     # offset scale for the float32 pair: q in [0.003, 0.13]
TIMESTEP_SHIFT_BF16 = 1000.0  # for the bfloat16 pair: q in [0.12, 4.7]


def timestep_pair(cfg, params, alpha, j=TIMESTEP_FREQ):
    """Parameters of the small model: ``params`` with time.w1[:, j] += alpha * v, v ~ N(0, 0.02^2) seeded."""
    small = dict(params)
    w1 = np.array(params["time.w1"], dtype=np.float32, copy=True)
    v = synth.gen_normal((9200,), (cfg.dim,), 0.02)
    w1[:, j] += np.float32(alpha) * v
    small["time.w1"] = synth.bf16_round(w1) if cfg.dtype == synth.BF16 else w1
    return small


def score_tolerance(q, delta):
    """Largest |q_device - q_oracle| that per-step velocity errors of relative L2 size delta allow.

    With p_L' = p_L + e_L, p_S' = p_S + e_S, ||e_L|| <= delta ||p_L|| and
    ||e_S|| <= delta ||p_S|| <= delta (1 + r) ||p_L||, the score
    r' = ||p_S' - p_L'|| / ||p_L'|| differs from r by at most
    (||e_S|| + ||e_L|| + r ||e_L||) / ||p_L'|| <= 2 delta (1 + r) / (1 - delta),
    and the mean over samples (Eq. 5) keeps the bound.
    """
    q = np.asarray(q, np.float64)
    return 2.0 * delta * (1.0 + q) / (1.0 - delta)


def boundary_gaps(q, delta):
    """For K = 1 .. N-1: (K, gap between the K-th and (K+1)-th smallest score, their summed tolerance)."""
    q = np.asarray(q, np.float64)
    tau = score_tolerance(q, delta)
    order = np.argsort(q, kind="stable")
    return [(K, float(q[order[K]] - q[order[K - 1]]), float(tau[order[K]] + tau[order[K - 1]]))
            for K in range(1, len(q))]
