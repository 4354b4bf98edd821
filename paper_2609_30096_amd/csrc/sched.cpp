// Host-side plan of the UniPC scheduler (the multistep update S of Eq. 2 with
// history h_i): per step, the weights of the fused corrector + predictor
// update that the unipc kernel applies element-wise.
//
// UniPC (Zhao et al., 2023), data-prediction form, B(h) = e^h - 1, on the
// flow-matching path alpha = 1 - sigma, lambda = log(alpha / sigma), with the
// data prediction m = x - sigma p.  For an update from base point b to
// target t with h = lambda_t - lambda_b and history points j (r_j =
// (lambda_j - lambda_b) / h):
//   x_t = (sigma_t / sigma_b) x_b - alpha_t (e^{-h} - 1) m_b
//         - alpha_t B(-h) sum_j rho_j (m_j - m_b) / r_j   [+ rho_new (m_t - m_b), corrector]
// Expanding the differences gives one weight per stored array, which is what
// the plan holds.  The weights rho solve R rho = b, R[a][k] = r_k^a,
// b[a] = g_{a+1} (a+1)! / B with g_1 = (e^{-h} - 1) / (-h) - 1 and
// g_{a+1} = g_a / (-h) - 1 / (a+1)!; the order-2 predictor and the order-1
// corrector take rho = 1/2.  Predictor order min(order, i + 1, N - i);
// history points at sigma = 1 (lambda = -inf) are left out.
#include <math.h>

#include <vector>

#include "kernels.h"

namespace track {

namespace {

double lambda_of(double s) {
  if (s >= 1.0) return -INFINITY;
  if (s <= 0.0) return INFINITY;
  return log((1.0 - s) / s);
}

// Solves the q x q system (q <= 3) by Gaussian elimination with partial pivoting.
void solve_small(int q, double R[3][3], double* b, double* x) {
  double A[3][4];
  for (int i = 0; i < q; ++i) {
    for (int j = 0; j < q; ++j) A[i][j] = R[i][j];
    A[i][q] = b[i];
  }
  for (int c = 0; c < q; ++c) {
    int p = c;
    for (int i = c + 1; i < q; ++i)
      if (fabs(A[i][c]) > fabs(A[p][c])) p = i;
    if (p != c)
      for (int j = 0; j <= q; ++j) {
        const double t = A[c][j];
        A[c][j] = A[p][j];
        A[p][j] = t;
      }
    for (int i = c + 1; i < q; ++i) {
      const double f = A[i][c] / A[c][c];
      for (int j = c; j <= q; ++j) A[i][j] -= f * A[c][j];
    }
  }
  for (int i = q - 1; i >= 0; --i) {
    double acc = A[i][q];
    for (int j = i + 1; j < q; ++j) acc -= A[i][j] * x[j];
    x[i] = acc / A[i][i];
  }
}

// rho for the ratio list r[0..q-1] (corrector: the last entry is the new
// point, r = 1).  A single weight is 1/2 for both the order-2 predictor and
// the order-1 corrector.
void rho_weights(int q, const double* r, double h, double* rho) {
  if (q == 1) {
    rho[0] = 0.5;
    return;
  }
  const double hh = -h;
  const double B = expm1(hh);
  double g = B / hh - 1.0;
  double fact = 1.0;
  double R[3][3], b[3];
  for (int a = 0; a < q; ++a) {
    for (int k = 0; k < q; ++k) R[a][k] = pow(r[k], a);
    b[a] = g * fact / B;
    fact *= a + 2;
    g = g / hh - 1.0 / fact;
  }
  solve_small(q, R, b, rho);
}

// Indices of the usable history points before `base` (at most q - 1 of them).
int history(const std::vector<double>& lam, int base, int q, int* js) {
  int n = 0;
  for (int k = 1; k < q; ++k) {
    const int j = base - k;
    if (j < 0 || isinf(lam[j])) break;
    js[n++] = j;
  }
  return n;
}

}  // namespace

std::vector<UniPCStep> unipc_plan(const std::vector<double>& sig, int order) {
  const int N = (int)sig.size() - 1;
  std::vector<double> lam(sig.size());
  for (size_t j = 0; j < sig.size(); ++j) lam[j] = lambda_of(sig[j]);
  std::vector<UniPCStep> plan(N);
  int q_last = 1;
  for (int i = 0; i < N; ++i) {
    UniPCStep& c = plan[i];
    c = UniPCStep{};
    if (i >= 1) {  // corrector: base i-1, target i, the new point m_i at r = 1
      const int base = i - 1;
      int js[2];
      const int nh = history(lam, base, q_last, js);
      const double s = sig[base], t = sig[i], at = 1.0 - t;
      const double h = lam[i] - lam[base];
      const double B = expm1(-h);  // also e^{-h} - 1
      double r[3], rho[3];
      for (int k = 0; k < nh; ++k) r[k] = (lam[js[k]] - lam[base]) / h;
      r[nh] = 1.0;
      rho_weights(nh + 1, r, h, rho);
      double sum = rho[nh];
      for (int k = 0; k < nh; ++k) sum += rho[k] / r[k];
      c.corr = 1;
      c.nh_c = nh;
      c.cx = t / s;
      c.c_m0 = -at * B + at * B * sum;
      c.c_h[0] = nh > 0 ? -at * B * rho[0] / r[0] : 0.0;  // m_{i-2}
      c.c_h[1] = nh > 1 ? -at * B * rho[1] / r[1] : 0.0;  // m_{i-3}
      c.c_new = -at * B * rho[nh];
    }
    int q = order;
    if (q > i + 1) q = i + 1;
    if (q > N - i) q = N - i;
    int js[2];
    const int nh = history(lam, i, q, js);
    q = nh + 1;
    const double s = sig[i], t = sig[i + 1], at = 1.0 - t;
    const double h = lam[i + 1] - lam[i];
    const double B = expm1(-h);
    double r[2] = {0.0, 0.0}, rho[2] = {0.0, 0.0};
    for (int k = 0; k < nh; ++k) r[k] = (lam[js[k]] - lam[i]) / h;
    if (nh > 0) rho_weights(nh, r, h, rho);
    double sum = 0.0;
    for (int k = 0; k < nh; ++k) sum += rho[k] / r[k];
    c.nh_p = nh;
    c.px = t / s;
    c.p_m = -at * B + at * B * sum;
    c.p_h[0] = nh > 0 ? -at * B * rho[0] / r[0] : 0.0;  // m_{i-1}
    c.p_h[1] = nh > 1 ? -at * B * rho[1] / r[1] : 0.0;  // m_{i-2}
    q_last = q;
  }
  return plan;
}

}  // namespace track
