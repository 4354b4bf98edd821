"""Oracle for TRACK's sampling, calibration and routing; float64, numpy.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper passages followed, in the paper's notation:
  Eq. 1  guided prediction  p_m = f_m(x, t, null) + w (f_m(x, t, tau) - f_m(x, t, null))
  Eq. 2  scheduler update   x_{t_{i+1}} = S(x_{t_i}, p, t_i, h_i); here S is the
         flow-matching Euler step on a shifted sigma table, with empty history
  Eq. 3  routed sampling    x_{t_{i+1}} = S(x_{t_i}, p_{pi(i)}(x_{t_i}, t_i), t_i, h_i)
  Sec. "Reference-Trajectory Calibration": roll out the all-large trajectory;
         before each update evaluate both models on the same latent, timestep,
         conditioning and guidance; advance with the large model's prediction
  Eq. 4  r_{j,k} = ||p_S - p_L||_2 / max(||p_L||_2, eps)
  Eq. 5  q_k = (1/M) sum_j r_{j,k}
  Eq. 6  min over beta in [0,1]^N of sum_k (W_k - C_0) beta_k, W_k = q_k^2
  Eq. 7  beta_k = 1 if W_k < C_0, 0 if W_k > C_0
  Sec. "Constrained Trajectory Divergence Minimization using Top-K Switching":
         route the K steps with the lowest q_k to the small model.

Readings where the paper is silent: the sigma table is the shifted linear
flow-matching table sigma_i = s u / (1 + (s - 1) u), u = 1 - i/N, with model
timestep t_i = 1000 sigma_i; the prediction is a velocity and the Euler step
is x + (sigma_{i+1} - sigma_i) p; the norm of Eq. 4 is the Frobenius norm of
the whole latent of one sample; equal scores are ranked by lower step index.

A model is passed as a (params, cfg) pair; ``denoise`` is the function that
evaluates f_m (oracle.dit.dit_forward unless a test substitutes a closed-form
velocity field).
"""
from __future__ import annotations

import itertools

import numpy as np

from . import dit, unipc


# ---------------------------------------------------------------- scheduler
def sigmas(steps, shift):
    """Shifted flow-matching noise levels sigma_0 = 1 > ... > sigma_N = 0 (N + 1 values)."""
    u = 1.0 - np.arange(steps + 1, dtype=np.float64) / steps
    return shift * u / (1.0 + (shift - 1.0) * u)


def timesteps(steps, shift):
    """Model timesteps t_i = 1000 sigma_i for i = 0..N-1 (decreasing)."""
    return 1000.0 * sigmas(steps, shift)[:-1]


def euler_step(x, p, sigma_i, sigma_next):
    """Eq. 2 with the Euler scheduler: x_{t_{i+1}} = x_{t_i} + (sigma_{i+1} - sigma_i) p."""
    return x + (sigma_next - sigma_i) * p


# ---------------------------------------------------------------- guidance
def scheduler(scfg, sig):
    """The update S of Eq. 2 for one trajectory, as a function (i, x_i, p_i) -> x_{i+1}."""
    solver = getattr(scfg, "solver", "euler")
    if solver == "euler":
        return lambda i, x, p: euler_step(x, p, sig[i], sig[i + 1])
    if solver == "unipc":
        return unipc.UniPC(sig, order=scfg.order).step
    raise ValueError(f"unknown solver {solver!r}")


def guided(f_cond, f_uncond, w):
    """Eq. 1: f(null) + w (f(tau) - f(null))."""
    return f_uncond + w * (f_cond - f_uncond)


def guided_prediction(model, x, t, cond, uncond, scfg, denoise=dit.dit_forward):
    """p_m(x, t): Eq. 1 when guidance is on, else the conditional prediction."""
    params, cfg = model
    f_c = denoise(params, cfg, x, t, cond)
    if not scfg.use_cfg:
        return f_c
    f_u = denoise(params, cfg, x, t, uncond)
    return guided(f_c, f_u, scfg.guidance)


# ---------------------------------------------------------------- scores
def relative_disagreement(p_small, p_large, eps):
    """Eq. 4: ||p_S - p_L||_2 / max(||p_L||_2, eps) over the whole latent."""
    diff = np.asarray(p_small, np.float64) - np.asarray(p_large, np.float64)
    num = np.sqrt(np.sum(diff * diff))
    den = np.sqrt(np.sum(np.asarray(p_large, np.float64) ** 2))
    return num / max(den, eps)


def mean_score(r):
    """Eq. 5: q_k = (1/M) sum_j r_{j,k}; r is [M, N], summed in sample order."""
    r = np.asarray(r, np.float64)
    q = np.zeros(r.shape[1], dtype=np.float64)
    for j in range(r.shape[0]):
        q = q + r[j]
    return q / r.shape[0]


def calibrate(large, small, x_T, conds, uncond, scfg, denoise=dit.dit_forward):
    """Reference-trajectory calibration; returns r [M, N] and q [N].

    For each calibration sample j: start at x_T[j]; at every step k evaluate
    p_L and p_S on the same x, t_k, conditioning and guidance; record r_{j,k};
    then advance the latent with p_L, so every probe stays on the all-large
    reference trajectory.
    """
    sig = sigmas(scfg.steps, scfg.shift)
    M, N = len(x_T), scfg.steps
    r = np.zeros((M, N), dtype=np.float64)
    for j in range(M):
        sched = scheduler(scfg, sig)
        x = np.asarray(x_T[j], np.float64)
        for k in range(N):
            t = 1000.0 * sig[k]
            p_L = guided_prediction(large, x, t, conds[j], uncond, scfg, denoise)
            p_S = guided_prediction(small, x, t, conds[j], uncond, scfg, denoise)
            r[j, k] = relative_disagreement(p_S, p_L, scfg.eps)
            x = sched(k, x, p_L)
    return r, mean_score(r)


# ---------------------------------------------------------------- policy
def lp_objective(W, C0, beta):
    """Eq. 6 objective sum_k (W_k - C_0) beta_k."""
    return float(np.sum((np.asarray(W, np.float64) - C0) * np.asarray(beta, np.float64)))


def threshold_solution(W, C0):
    """Eq. 7: beta_k = 1 where W_k < C_0, 0 where W_k > C_0 (0 is chosen at equality)."""
    return (np.asarray(W, np.float64) < C0).astype(np.float64)


def route_topk(q, K):
    """Indices of the K lowest scores, ascending; equal scores go to the lower step index."""
    q = np.asarray(q, np.float64)
    N = q.shape[0]
    if not 0 <= K <= N:
        raise ValueError("K must satisfy 0 <= K <= N")
    order = sorted(range(N), key=lambda k: (q[k], k))
    return np.array(sorted(order[:K]), dtype=np.int32)


def route_bruteforce(q, K):
    """All K-subsets minimising sum_k W_k over the subset (Eq. 6 at a fixed budget)."""
    W = np.asarray(q, np.float64) ** 2
    best, arg = None, []
    for sub in itertools.combinations(range(len(W)), K):
        v = float(sum(W[list(sub)])) if sub else 0.0
        if best is None or v < best - 1e-300:
            best, arg = v, [sub]
        elif v == best:
            arg.append(sub)
    return best, arg


def route_threshold(q, C0):
    """Eqs. 6-7 in the C_0 form: the steps with W_k = q_k^2 < C_0 go to the small model.

    At W_k = C_0 every beta in [0, 1] is optimal; this reading keeps the large
    model there (beta = 0).  Returns the selected indices, ascending.
    """
    W = np.asarray(q, np.float64) ** 2
    beta = threshold_solution(W, C0)
    return np.flatnonzero(beta > 0.5).astype(np.int32)


# ---------------------------------------------------------------- equal-budget baseline policies
def first_k(N, K):
    """First-K: the initial K steps run the small model (Sec. "Equal-Budget Policy Ablations")."""
    if not 0 <= K <= N:
        raise ValueError("K must satisfy 0 <= K <= N")
    return np.arange(K, dtype=np.int32)


def last_k(N, K):
    """Last-K: the final K steps run the small model."""
    if not 0 <= K <= N:
        raise ValueError("K must satisfy 0 <= K <= N")
    return np.arange(N - K, N, dtype=np.int32)


_MASK64 = (1 << 64) - 1


def splitmix64(state):
    """One SplitMix64 step (Steele, Lea and Flood, 2014): returns (new_state, output)."""
    state = (state + 0x9E3779B97F4A7C15) & _MASK64
    z = state
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
    return state, z ^ (z >> 31)


def random_k(N, K, seed):
    """Random-K: K distinct steps chosen at random, ascending.

    Step k draws the k-th SplitMix64 output of a generator started at `seed`
    (a uniform 64-bit key per step); the K steps with the smallest keys are
    taken, equal keys going to the lower index, which makes every K-subset
    equally likely up to the generator's quality.
    """
    if not 0 <= K <= N:
        raise ValueError("K must satisfy 0 <= K <= N")
    state, keys = seed & _MASK64, []
    for _ in range(N):
        state, z = splitmix64(state)
        keys.append(z)
    order = sorted(range(N), key=lambda k: (keys[k], k))
    return np.array(sorted(order[:K]), dtype=np.int32)


def policy_from_indices(N, small_idx):
    """pi as a bool array: True where the step runs the small model."""
    use_small = np.zeros(N, dtype=bool)
    use_small[np.asarray(small_idx, dtype=np.int64)] = True
    return use_small


# ---------------------------------------------------------------- routed sampling
def sample(use_small, large, small, x_T, cond, uncond, scfg, denoise=dit.dit_forward, return_path=False):
    """Eq. 3: one model per step, chosen by the policy; returns x after N steps.

    The scheduler state (UniPC's history) evolves the same way whichever
    model supplied each prediction.
    """
    sig = sigmas(scfg.steps, scfg.shift)
    sched = scheduler(scfg, sig)
    x = np.asarray(x_T, np.float64)
    path = [x]
    for i in range(scfg.steps):
        model = small if use_small[i] else large
        p = guided_prediction(model, x, 1000.0 * sig[i], cond, uncond, scfg, denoise)
        x = sched(i, x, p)
        path.append(x)
    return (x, path) if return_path else x
