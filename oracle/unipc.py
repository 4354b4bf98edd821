"""Oracle for the UniPC multistep scheduler S(x, p, t_i, h_i) of Eq. 2; float64, numpy.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper leaves the scheduler to the pipeline: Eq. 2 allows a history h_i,
the routing must keep the scheduler-state evolution unchanged whichever model
supplies p (Sec. "Preliminaries", "Inference"), and Wan 2.1 samples with
UniPC.  This module restates UniPC (Zhao et al., "UniPC: A Unified
Predictor-Corrector Framework for Fast Sampling of Diffusion Models", 2023) in
its data-prediction form with B(h) = e^h - 1, for the flow-matching path
x_sigma = (1 - sigma) x_0 + sigma eps:

  alpha = 1 - sigma,  lambda = log(alpha / sigma),  data prediction m = x - sigma p.

Step i (sigma_i -> sigma_{i+1}) receives the sample x_i at which the model was
evaluated and the guided velocity p_i there:
  1. m_i = x_i - sigma_i p_i joins the history (whichever model produced p_i);
  2. corrector UniC (i >= 1): x_i is replaced by
        x_i^c = (sigma_i / sigma_{i-1}) x_{i-1}^c - alpha_i phi_1 m_{i-1}
                - alpha_i B (sum_k rho_k D_k + rho_q (m_i - m_{i-1})),
     with h = lambda_i - lambda_{i-1}, phi_1 = e^{-h} - 1 = B,
     D_k = (m_{i-1-k} - m_{i-1}) / r_k, r_k = (lambda_{i-1-k} - lambda_{i-1}) / h
     (k = 1 .. q-1, q the order of step i-1's predictor); the model is not
     evaluated again at x_i^c;
  3. predictor UniP of order q:
        x_{i+1} = (sigma_{i+1} / sigma_i) x_i^c - alpha_{i+1} phi_1 m_i
                  - alpha_{i+1} B sum_{k=1}^{q-1} rho_k D_k,
     D_k = (m_{i-k} - m_i) / r_k, r_k = (lambda_{i-k} - lambda_i) / h, h = lambda_{i+1} - lambda_i.
The weights rho solve R rho = b with R[a][k] = r_k^a and
b[a] = g_{a+1} (a+1)! / B, g_1 = phi_1 / (-h) - 1, g_{a+1} = g_a / (-h) - 1 / (a+1)!
(predictor: the history columns only; corrector: the history columns and r = 1
for m_i), except that the order-2 predictor and the order-1 corrector use
rho = 1/2.  The predictor order is q = min(order, i + 1, N - i): one more than
the history available (warm-up) and first order on the last step.

Readings where the method meets this sampler's sigma table: sigma_0 = 1 gives
lambda_0 = -inf and sigma_N = 0 gives lambda_N = +inf.  A base point or a
target at an infinite lambda only makes e^{-h} - 1 = -1, which is finite; a
*history* entry at lambda = -inf would make r infinite, so such entries are
left out and the order drops accordingly (for the predictor this is the
r -> -inf limit, D -> 0).  The last step is first order, as stated above.
With order 1 and no corrector the update is exactly the Euler step.
"""
from __future__ import annotations

import math

import numpy as np


def _lam(s):
    if s >= 1.0:
        return -math.inf
    if s <= 0.0:
        return math.inf
    return math.log((1.0 - s) / s)


def rho_weights(rks, h, predictor):
    """Weights rho for the r list rks (history r_k, plus 1.0 last for the corrector)."""
    q = len(rks)
    if q == 0:
        return np.zeros(0)
    if predictor and q == 1:
        return np.array([0.5])  # order-2 predictor
    if not predictor and q == 1:
        return np.array([0.5])  # order-1 corrector
    hh = -h
    phi1 = math.expm1(hh)
    B = phi1
    g = phi1 / hh - 1.0
    fact = 1.0
    R = np.zeros((q, q))
    b = np.zeros(q)
    for a in range(q):
        R[a] = np.asarray(rks, np.float64) ** a
        b[a] = g * fact / B
        fact *= a + 2
        g = g / hh - 1.0 / fact
    return np.linalg.solve(R, b)


class UniPC:
    """Scheduler state for one trajectory: call step(i, x_i, p_i) for i = 0 .. N-1."""

    def __init__(self, sig, order=2, corrector=True):
        self.sig = [float(s) for s in sig]
        self.N = len(self.sig) - 1
        self.order = int(order)
        self.corrector = corrector
        self.lam = [_lam(s) for s in self.sig]
        self.m = []          # data predictions m_0 .. m_i
        self.x_last = None   # corrected sample at the previous step's sigma
        self.q_last = None   # order of the previous step's predictor

    def _history(self, base, q):
        """Usable history for an update whose base point is step `base`: at most q-1 entries."""
        ks = []
        for k in range(1, q):
            j = base - k
            if j < 0 or math.isinf(self.lam[j]):
                break
            ks.append(j)
        return ks

    def step(self, i, x, p):
        sig, lam = self.sig, self.lam
        x = np.asarray(x, np.float64)
        m_i = x - sig[i] * np.asarray(p, np.float64)
        if self.corrector and i >= 1:
            s, t = sig[i - 1], sig[i]
            h = lam[i] - lam[i - 1]
            m0 = self.m[i - 1]
            hist = self._history(i - 1, self.q_last)
            rks = [(lam[j] - lam[i - 1]) / h for j in hist] + [1.0]
            rho = rho_weights(rks, h, predictor=False)
            phi1 = math.expm1(-h)
            B = phi1
            res = sum(rho[n] * (self.m[j] - m0) / rks[n] for n, j in enumerate(hist))
            res = res + rho[-1] * (m_i - m0)
            x = (t / s) * self.x_last - (1.0 - t) * phi1 * m0 - (1.0 - t) * B * res
        self.m.append(m_i)
        q = min(self.order, i + 1, self.N - i)
        hist = self._history(i, q)
        q = len(hist) + 1
        s, t = sig[i], sig[i + 1]
        h = lam[i + 1] - lam[i]
        phi1 = math.expm1(-h)
        B = phi1
        x_next = (t / s) * x - (1.0 - t) * phi1 * m_i
        if hist:
            rks = [(lam[j] - lam[i]) / h for j in hist]
            rho = rho_weights(rks, h, predictor=True)
            res = sum(rho[n] * (self.m[j] - m_i) / rks[n] for n, j in enumerate(hist))
            x_next = x_next - (1.0 - t) * B * res
        self.x_last = x
        self.q_last = q
        return x_next
