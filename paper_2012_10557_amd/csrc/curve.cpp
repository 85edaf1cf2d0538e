// Accuracy-curve extrapolation of the micro-profiler (section 4.3): per-epoch
// held-out accuracies of a short run on a small subset are fitted to the
// training-progress curve of Optimus (Peng et al., EuroSys 2018) by
// non-negative least squares and evaluated at a full retraining.
//
// Model: held-out error e = 1 - accuracy after x passes over the whole
// window's data (E epochs on a fraction f: x = E f) is
// e(x) = 1 / (b0 x + b1) + b2, b0, b1, b2 >= 0.  For a fixed b2 below every
// measured error, 1 / (e - b2) = b0 x + b1 is linear in (b0, b1) >= 0 and
// is solved by NNLS; b2 is chosen on a grid over [0, min e) and refined by
// golden-section search to minimise the squared error in accuracy.
//
// Host code only (no GPU work).
#include "curve.hpp"

#include <algorithm>
#include <cmath>
#include <limits>
#include <vector>

namespace ekya {

namespace {

// min || A[:, cols] z - b || by Householder QR of the selected columns
// (A row-major m x n).  Returns false if a diagonal of R vanishes.
bool lstsq_cols(const double* A, int m, int n, const std::vector<int>& cols, const double* b,
                std::vector<double>& z) {
  const int p = (int)cols.size();
  std::vector<double> Q((size_t)m * p), r(b, b + m);
  for (int i = 0; i < m; ++i)
    for (int j = 0; j < p; ++j) Q[(size_t)i * p + j] = A[(size_t)i * n + cols[j]];
  std::vector<double> diag(p);
  for (int j = 0; j < p; ++j) {
    double nrm = 0.0;
    for (int i = j; i < m; ++i) nrm += Q[(size_t)i * p + j] * Q[(size_t)i * p + j];
    nrm = std::sqrt(nrm);
    if (nrm == 0.0 || j >= m) return false;
    const double alpha = Q[(size_t)j * p + j] > 0 ? -nrm : nrm;
    // v = x - alpha e1, stored in column j from row j
    Q[(size_t)j * p + j] -= alpha;
    double vnorm2 = 0.0;
    for (int i = j; i < m; ++i) vnorm2 += Q[(size_t)i * p + j] * Q[(size_t)i * p + j];
    if (vnorm2 > 0.0) {
      for (int k = j + 1; k < p; ++k) {
        double s = 0.0;
        for (int i = j; i < m; ++i) s += Q[(size_t)i * p + j] * Q[(size_t)i * p + k];
        s = 2.0 * s / vnorm2;
        for (int i = j; i < m; ++i) Q[(size_t)i * p + k] -= s * Q[(size_t)i * p + j];
      }
      double s = 0.0;
      for (int i = j; i < m; ++i) s += Q[(size_t)i * p + j] * r[i];
      s = 2.0 * s / vnorm2;
      for (int i = j; i < m; ++i) r[i] -= s * Q[(size_t)i * p + j];
    }
    diag[j] = alpha;
  }
  z.assign(p, 0.0);
  for (int j = p - 1; j >= 0; --j) {
    double s = r[j];
    for (int k = j + 1; k < p; ++k) s -= Q[(size_t)j * p + k] * z[k];
    if (diag[j] == 0.0) return false;
    z[j] = s / diag[j];
  }
  return true;
}

}  // namespace

// Lawson and Hanson's active-set NNLS ("Solving Least Squares Problems",
// 1974, chapter 23).
bool nnls(const double* A, int m, int n, const double* b, double* x, double* rnorm) {
  std::vector<char> free_(n, 0);
  std::fill(x, x + n, 0.0);
  double norm1 = 0.0;  // max column sum, as numpy's 1-norm
  for (int j = 0; j < n; ++j) {
    double s = 0.0;
    for (int i = 0; i < m; ++i) s += std::fabs(A[(size_t)i * n + j]);
    norm1 = std::max(norm1, s);
  }
  const double tol = 10.0 * std::numeric_limits<double>::epsilon() * norm1 * std::max(m, n);
  std::vector<double> res(m), w(n), z;
  auto residual = [&]() {
    for (int i = 0; i < m; ++i) {
      double s = b[i];
      for (int j = 0; j < n; ++j) s -= A[(size_t)i * n + j] * x[j];
      res[i] = s;
    }
  };
  for (int it = 0; it < 3 * n; ++it) {
    residual();
    for (int j = 0; j < n; ++j) {
      double s = 0.0;
      for (int i = 0; i < m; ++i) s += A[(size_t)i * n + j] * res[i];
      w[j] = s;
    }
    int best = -1;
    for (int j = 0; j < n; ++j)
      if (!free_[j] && w[j] > tol && (best < 0 || w[j] > w[best])) best = j;
    if (best < 0) break;
    free_[best] = 1;
    for (;;) {
      std::vector<int> cols;
      for (int j = 0; j < n; ++j)
        if (free_[j]) cols.push_back(j);
      std::vector<double> zf(n, 0.0);
      if (!cols.empty()) {
        if (!lstsq_cols(A, m, n, cols, b, z)) return false;
        for (size_t q = 0; q < cols.size(); ++q) zf[cols[q]] = z[q];
      }
      bool all_pos = true;
      for (int j : cols)
        if (zf[j] <= tol) all_pos = false;
      if (all_pos) {
        std::copy(zf.begin(), zf.end(), x);
        break;
      }
      double alpha = std::numeric_limits<double>::infinity();
      for (int j : cols)
        if (zf[j] <= tol) alpha = std::min(alpha, x[j] / (x[j] - zf[j]));
      for (int j = 0; j < n; ++j) x[j] += alpha * (zf[j] - x[j]);
      for (int j = 0; j < n; ++j)
        if (free_[j] && x[j] <= tol) free_[j] = 0;
      for (int j = 0; j < n; ++j)
        if (!free_[j]) x[j] = 0.0;
    }
  }
  residual();
  double s = 0.0;
  for (int i = 0; i < m; ++i) s += res[i] * res[i];
  if (rnorm) *rnorm = std::sqrt(s);
  return true;
}

double curve_error(const Curve& c, double x) {
  const double d = c.b0 * x + c.b1;
  return d > 0 ? 1.0 / d + c.b2 : std::numeric_limits<double>::infinity();
}

double curve_accuracy(const Curve& c, double x) {
  return std::min(1.0, std::max(0.0, 1.0 - curve_error(c, x)));
}

static Curve fit_given_b2(const std::vector<double>& x, const std::vector<double>& e, double b2) {
  const int m = (int)x.size();
  std::vector<double> A((size_t)m * 2), t(m);
  for (int i = 0; i < m; ++i) {
    A[2 * i] = x[i];
    A[2 * i + 1] = 1.0;
    t[i] = 1.0 / (e[i] - b2);
  }
  double beta[2] = {0.0, 0.0};
  Curve c;
  if (!nnls(A.data(), m, 2, t.data(), beta, nullptr)) beta[0] = beta[1] = 0.0;
  c.b0 = beta[0];
  c.b1 = beta[1];
  c.b2 = b2;
  double rss = 0.0;
  for (int i = 0; i < m; ++i) {
    const double d = curve_error(c, x[i]) - e[i];
    rss += d * d;
  }
  c.rss = rss;
  return c;
}

// A candidate replaces the best fit only if its squared error is smaller by
// more than a relative 1e-9 and an absolute 1e-20 (among the exact fits of
// too few points, which differ only by rounding, the smallest b2 tried is
// kept).
static bool better(const Curve& a, const Curve& b) {
  return a.rss < b.rss * (1.0 - 1e-9) - 1e-20;
}

bool fit_accuracy_curve(const double* xs, const double* acc, int n, Curve* out) {
  if (n < 1) return false;
  std::vector<double> x(xs, xs + n), e(n);
  double emin = std::numeric_limits<double>::infinity();
  for (int i = 0; i < n; ++i) {
    e[i] = 1.0 - acc[i];
    emin = std::min(emin, e[i]);
  }
  if (emin <= 0.0) {  // a perfect point: the curve must reach error 0
    for (double& v : e) v = std::max(v, 1e-12);
    *out = fit_given_b2(x, e, 0.0);
    return true;
  }
  const int grid = 64, refine = 60;
  const double hi = emin * (1.0 - 1e-9);
  Curve best;
  int bi = 0;
  for (int i = 0; i < grid; ++i) {
    Curve c = fit_given_b2(x, e, hi * i / grid);
    if (i == 0 || better(c, best)) {
      best = c;
      bi = i;
    }
  }
  const double g = (std::sqrt(5.0) - 1.0) / 2.0;
  double a = hi * std::max(bi - 1, 0) / grid, d = hi * std::min(bi + 1, grid) / grid;
  double c1 = d - g * (d - a), c2 = a + g * (d - a);
  Curve f1 = fit_given_b2(x, e, c1), f2 = fit_given_b2(x, e, std::min(c2, hi));
  for (int it = 0; it < refine; ++it) {
    if (f1.rss <= f2.rss) {
      d = c2;
      c2 = c1;
      f2 = f1;
      c1 = d - g * (d - a);
      f1 = fit_given_b2(x, e, c1);
    } else {
      a = c1;
      c1 = c2;
      f1 = f2;
      c2 = a + g * (d - a);
      f2 = fit_given_b2(x, e, std::min(c2, hi));
    }
  }
  if (better(f1, best)) best = f1;
  if (better(f2, best)) best = f2;
  *out = best;
  return true;
}

}  // namespace ekya
