// Host side: convex non-decreasing least-squares regression of a verification-
// cost profile (Sec. 4.6, eq. convex-reg) and the cost table built from it.
//
// On a strictly increasing grid x_0 < .. < x_{N-1} the convex non-decreasing
// functions are c + b_0 (x - x_0) + sum_{k=1}^{N-2} b_k max(0, x - x_k) with
// b >= 0 and c free, so the program is non-negative least squares in b.  It
// is solved exactly by the Lawson-Hanson active-set method, with every
// product by the hinge matrix done in O(N):
//   * A b is a running sum of slopes along the grid;
//   * A^T r is a suffix recurrence, w_{k-1} = w_k + (x_k - x_{k-1}) sum_{j>=k} r_j;
//   * the least-squares fit on a passive set (free intercept, first slope if
//     b_0 is passive, slope changes at the passive knots) is the best
//     continuous piecewise-linear function on those knots; in the hat basis on
//     the knots its normal equations are tridiagonal and positive definite
//     (every hat is 1 at its own grid point, where the others vanish), solved
//     by elimination, and its hinge coefficients are the slope changes.

#include <algorithm>
#include <cmath>
#include <vector>

#include "internal.h"

namespace caddtree {
namespace {

struct Fitter {
  const double* x;
  const double* y;
  int N;
  std::vector<double> f;      // fitted values of the last least-squares solve

  // least squares on the passive set: z (hinge coefficients, zero off the set) and f
  void solve(const std::vector<char>& passive, std::vector<double>& z) {
    std::vector<int> node;    // grid indices of the hat nodes
    const bool free_slope = passive[0] != 0;
    if (free_slope) node.push_back(0);
    for (int k = 1; k <= N - 2; ++k)
      if (passive[k]) node.push_back(k);
    if (node.empty() || node.back() != N - 1) node.push_back(N - 1);
    const int m = (int)node.size();
    std::vector<double> D(m, 0.0), E(m, 0.0), R(m, 0.0);   // diagonal, super-diagonal, right side
    for (int j = 0; j < N; ++j) {
      // segment i: node[i] <= j < node[i + 1]; points left of node[0] (no free first slope) load hat 0 alone
      if (j < node[0]) {
        D[0] += 1.0;
        R[0] += y[j];
        continue;
      }
      const int i = (int)(std::upper_bound(node.begin(), node.end(), j) - node.begin()) - 1;
      if (i == m - 1) {
        D[i] += 1.0;
        R[i] += y[j];
        continue;
      }
      const double t = (x[j] - x[node[i]]) / (x[node[i + 1]] - x[node[i]]);
      const double a = 1.0 - t;
      D[i] += a * a;
      D[i + 1] += t * t;
      E[i] += a * t;
      R[i] += a * y[j];
      R[i + 1] += t * y[j];
    }
    // tridiagonal elimination (symmetric positive definite: no pivoting needed)
    std::vector<double> v(m);
    for (int i = 1; i < m; ++i) {
      const double w = E[i - 1] / D[i - 1];
      D[i] -= w * E[i - 1];
      R[i] -= w * R[i - 1];
    }
    v[m - 1] = R[m - 1] / D[m - 1];
    for (int i = m - 2; i >= 0; --i) v[i] = (R[i] - E[i] * v[i + 1]) / D[i];
    // fitted values
    f.assign(N, 0.0);
    for (int j = 0; j < N; ++j) {
      if (j <= node[0]) { f[j] = v[0]; continue; }
      const int i = (int)(std::upper_bound(node.begin(), node.end(), j) - node.begin()) - 1;
      if (i == m - 1) { f[j] = v[m - 1]; continue; }
      const double t = (x[j] - x[node[i]]) / (x[node[i + 1]] - x[node[i]]);
      f[j] = (1.0 - t) * v[i] + t * v[i + 1];
    }
    // hinge coefficients: the slope of each segment, and its change at each knot
    z.assign(N - 1, 0.0);
    double prev = 0.0;   // slope left of the first node (zero unless b_0 is free, then node[0] = 0)
    for (int i = 0; i + 1 < m; ++i) {
      const double s = (v[i + 1] - v[i]) / (x[node[i + 1]] - x[node[i]]);
      if (i == 0 && free_slope) z[0] = s;
      else z[node[i]] = s - prev;
      prev = s;
    }
  }
};

// f = c + A b with c = mean(y - A b)
void evaluate(const double* x, const double* y, int N, const std::vector<double>& b, std::vector<double>& f) {
  f.assign(N, 0.0);
  double slope = b[0], g = 0.0, mean = 0.0;
  for (int j = 1; j < N; ++j) {
    g += slope * (x[j] - x[j - 1]);
    f[j] = g;
    if (j <= N - 2) slope += b[j];
  }
  for (int j = 0; j < N; ++j) mean += y[j] - f[j];
  mean /= N;
  for (int j = 0; j < N; ++j) f[j] += mean;
}

// w = A^T r, r = y - f
void gradient(const double* x, const double* y, int N, const std::vector<double>& f, std::vector<double>& w) {
  w.assign(N - 1, 0.0);
  double tail = 0.0, acc = 0.0;   // tail = sum_{j>k} r_j, acc = sum_{j>k} (x_j - x_k) r_j
  for (int k = N - 1; k >= 1; --k) {
    tail += y[k] - f[k];
    acc += (x[k] - x[k - 1]) * tail;
    w[k - 1] = acc;              // w[k - 1] = sum_{j > k - 1} (x_j - x_{k-1}) r_j
  }
}

}  // namespace

// Inputs are validated by the caller (finite, x strictly increasing, N >= 1).
bool fit_convex_cost(const double* x_host, const double* y_host, int n, double* fit_host, int32_t cap,
                     double* table_host) {
  std::vector<double> f(n, y_host[0]);
  if (n >= 2) {
    Fitter F{x_host, y_host, n, {}};
    std::vector<char> passive(n - 1, 0), banned(n - 1, 0);
    std::vector<double> b(n - 1, 0.0), z, w;
    evaluate(x_host, y_host, n, b, f);
    double ysc = 0.0, ymean = 0.0;
    for (int j = 0; j < n; ++j) ymean += y_host[j];
    ymean /= n;
    for (int j = 0; j < n; ++j) ysc += std::fabs(y_host[j] - ymean);
    const double tol = 1e-12 * (x_host[n - 1] - x_host[0]) * ysc + 1e-300;
    const int max_outer = 4 * n + 10;
    for (int outer = 0;; ++outer) {
      if (outer > max_outer) return false;
      gradient(x_host, y_host, n, f, w);
      int t = -1;
      double best = tol;
      for (int k = 0; k < n - 1; ++k)
        if (!passive[k] && !banned[k] && w[k] > best) { best = w[k]; t = k; }
      if (t < 0) break;
      passive[t] = 1;
      F.solve(passive, z);
      if (!(z[t] > 0.0)) {
        // rounding: the entering variable's least-squares value is not positive, so it
        // cannot improve the fit; leave b unchanged and try the next candidate
        passive[t] = 0;
        banned[t] = 1;
        continue;
      }
      for (int inner = 0;; ++inner) {
        if (inner > n + 5) return false;
        double alpha = 2.0;
        int arg = -1;
        for (int k = 0; k < n - 1; ++k)
          if (passive[k] && !(z[k] > 0.0)) {
            const double den = b[k] - z[k];
            const double a = den > 0.0 ? b[k] / den : 0.0;
            if (a < alpha) { alpha = a; arg = k; }
          }
        if (arg < 0) {
          b = z;
          break;
        }
        // step towards z until the first passive coefficient reaches zero, and drop it
        for (int k = 0; k < n - 1; ++k) b[k] += alpha * (z[k] - b[k]);
        b[arg] = 0.0;
        for (int k = 0; k < n - 1; ++k)
          if (passive[k] && !(b[k] > 0.0)) { passive[k] = 0; b[k] = 0.0; }
        F.solve(passive, z);
      }
      std::fill(banned.begin(), banned.end(), 0);
      evaluate(x_host, y_host, n, b, f);
    }
    // the final fitted values come from the last least-squares solve on the passive set
    F.solve(passive, z);
    f = F.f;
  }
  if (fit_host)
    for (int j = 0; j < n; ++j) fit_host[j] = f[j];
  if (table_host) {
    for (int m = 0; m <= cap; ++m) {
      const double q = (double)m;
      double v;
      if (n == 1) {
        v = f[0];
      } else if (q <= x_host[0]) {
        v = f[0] + (q - x_host[0]) * ((f[1] - f[0]) / (x_host[1] - x_host[0]));
      } else if (q >= x_host[n - 1]) {
        v = f[n - 1] + (q - x_host[n - 1]) * ((f[n - 1] - f[n - 2]) / (x_host[n - 1] - x_host[n - 2]));
      } else {
        const int i = (int)(std::upper_bound(x_host, x_host + n, q) - x_host) - 1;
        const double t = (q - x_host[i]) / (x_host[i + 1] - x_host[i]);
        v = (1.0 - t) * f[i] + t * f[i + 1];
      }
      table_host[m] = v;
    }
  }
  return true;
}

}  // namespace caddtree
