// Greedy Polar Express schedule (library side, host code, double precision).
//
// Sec. 3 ("Computing the polar factor") and App. E.1 fix the method: Polar
// Express with lower bound l = 1e-3, odd polynomials of degree d = 5, T steps,
// applied after normalising by ||W||_F + eps. The schedule is defined by
// greedy minimax: p_t minimises max_{x in [l_t, u_t]} |1 - p_t(x)| over odd
// polynomials of degree d, [l_1, u_1] = [l, 1], and the next interval is the
// image [1 - E_t, 1 + E_t] of the current one (E_t = optimal error).
//
// Solved by Remez exchange: d = 5 -> alternation at l_t, two interior extrema
// of the error, u_t (signs +, -, +, -); d = 3 -> l_t, one interior extremum,
// u_t. Unknowns are written in the odd basis x, x(x^2-1), x(x^2-1)^2, which
// stays well conditioned while the interval contracts around 1; the
// interior extrema are the roots in z = x^2 - 1 of p'(x) = 0, taken with the
// cancellation-free quadratic formula. Once E_t < 1e-4 the next minimax
// problem is below double-precision resolution (its error would be ~E_t^3);
// every later step then uses the limit of the greedy polynomial as the
// interval shrinks to {1}: p(1) = 1 with the most vanishing derivatives at 1,
// i.e. the Newton-Schulz polynomial (15x - 10x^3 + 3x^5)/8 (degree 5) or
// (3x - x^3)/2 (degree 3).
#include <cmath>
#include <stdexcept>
#include <vector>

namespace slorr {

namespace {

constexpr double kStop = 1e-4;

// Gaussian elimination with partial pivoting, n <= 4.
void solve(int n, double a[4][5]) {
  for (int c = 0; c < n; ++c) {
    int piv = c;
    for (int r = c + 1; r < n; ++r)
      if (std::fabs(a[r][c]) > std::fabs(a[piv][c])) piv = r;
    if (a[piv][c] == 0.0) throw std::runtime_error("singular Remez system");
    if (piv != c)
      for (int k = 0; k <= n; ++k) std::swap(a[c][k], a[piv][k]);
    for (int r = c + 1; r < n; ++r) {
      double f = a[r][c] / a[c][c];
      for (int k = c; k <= n; ++k) a[r][k] -= f * a[c][k];
    }
  }
  for (int c = n - 1; c >= 0; --c) {
    double s = a[c][n];
    for (int k = c + 1; k < n; ++k) s -= a[c][k] * a[k][n];
    a[c][n] = s / a[c][c];
  }
}

struct Step {
  double coeff[3];  // monomial a, b, c
  double err;
};

Step minimax_step(double lo, double hi, int degree) {
  const int nin = (degree - 1) / 2;        // interior alternation points
  const int npts = nin + 2;
  const double pi = 3.14159265358979323846;
  double inner[2];
  const double mid = 0.5 * (lo + hi), rad = 0.5 * (hi - lo);
  for (int k = 0; k < nin; ++k) inner[k] = mid - rad * std::cos(pi * (k + 1) / (nin + 1));
  double w[3] = {0, 0, 0}, err = 0;
  for (int it = 0; it < 200; ++it) {
    double pts[4];
    pts[0] = lo;
    for (int k = 0; k < nin; ++k) pts[1 + k] = inner[k];
    pts[npts - 1] = hi;
    double m[4][5];
    for (int i = 0; i < npts; ++i) {
      const double x = pts[i], z = (x - 1.0) * (x + 1.0);
      m[i][0] = x;
      m[i][1] = x * z;
      if (degree == 5) m[i][2] = x * z * z;
      m[i][nin + 1] = (i & 1) ? -1.0 : 1.0;   // error sign +, -, +, -
      m[i][npts] = 1.0;
    }
    solve(npts, m);
    for (int k = 0; k <= nin; ++k) w[k] = m[k][npts];
    err = m[nin + 1][npts];
    double z[2];
    if (degree == 3) {
      // p' = (alpha + 2 beta) + 3 beta z
      z[0] = -(w[0] + 2.0 * w[1]) / (3.0 * w[1]);
    } else {
      // p' = alpha + beta (3z + 2) + gamma (5 z^2 + 4 z)
      const double qa = 5.0 * w[2], qb = 3.0 * w[1] + 4.0 * w[2], qc = w[0] + 2.0 * w[1];
      const double disc = qb * qb - 4.0 * qa * qc;
      if (disc < 0.0 || qa == 0.0) throw std::runtime_error("no interior extrema");
      const double s = std::sqrt(disc);
      const double q = -0.5 * (qb + (qb >= 0.0 ? s : -s));
      z[0] = q / qa;
      z[1] = qc / q;
      if (z[0] > z[1]) std::swap(z[0], z[1]);
    }
    const double zlo = (lo - 1.0) * (lo + 1.0), zhi = (hi - 1.0) * (hi + 1.0);
    double change = 0.0;
    for (int k = 0; k < nin; ++k) {
      if (!(z[k] > zlo && z[k] < zhi)) throw std::runtime_error("extrema left the interval");
      const double x = std::sqrt(1.0 + z[k]);
      change = std::fmax(change, std::fabs(x - inner[k]));
      inner[k] = x;
    }
    if (change <= 4e-16 * hi) break;
  }
  Step s;
  if (degree == 3) {
    s.coeff[0] = w[0] - w[1];
    s.coeff[1] = w[1];
    s.coeff[2] = 0.0;
  } else {
    s.coeff[0] = w[0] - w[1] + w[2];
    s.coeff[1] = w[1] - 2.0 * w[2];
    s.coeff[2] = w[2];
  }
  s.err = std::fabs(err);
  return s;
}

}  // namespace

// Writes iters rows (a, b, c). Throws std::runtime_error on failure.
void greedy_schedule(double ell, int degree, int iters, double *out) {
  double lo = ell, hi = 1.0;
  bool limit = false;
  for (int t = 0; t < iters; ++t) {
    double *row = out + 3 * t;
    if (limit) {
      row[0] = degree == 5 ? 1.875 : 1.5;
      row[1] = degree == 5 ? -1.25 : -0.5;
      row[2] = degree == 5 ? 0.375 : 0.0;
      continue;
    }
    const Step s = minimax_step(lo, hi, degree);
    for (int k = 0; k < 3; ++k) row[k] = s.coeff[k];
    lo = 1.0 - s.err;
    hi = 1.0 + s.err;
    limit = s.err < kStop;
  }
}

}  // namespace slorr
