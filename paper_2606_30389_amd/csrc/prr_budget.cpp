// Critical-path-aware speculation budget (Section 4.4): from a table of selection and
// speculation latencies profiled offline per context length and budget ratio delta, the
// largest delta whose speculation fits in the selection window at the current context.
// Latencies at a context that was not profiled are estimated by polynomial regression
// (appendix "Profiling Overheads"), here least squares in log2(context).  Host code.
#include <math.h>

#include <algorithm>
#include <vector>

#include "prr_launch.h"

namespace {

// Least-squares polynomial of degree `deg` through (x[i], y[i]), evaluated at x0; solved by
// Gaussian elimination with partial pivoting on the normal equations of the centred and
// scaled abscissae (at most 4 unknowns).
double poly_fit_eval(const std::vector<double>& x, const std::vector<double>& y, int deg, double x0) {
  const int n = (int)x.size(), m = deg + 1;
  double mean = 0.0, span = 0.0;
  for (double v : x) mean += v;
  mean /= n;
  for (double v : x) span = std::max(span, fabs(v - mean));
  if (span == 0.0) span = 1.0;
  double A[4][5] = {};
  for (int i = 0; i < n; ++i) {
    const double u = (x[i] - mean) / span;
    double pw[8];
    pw[0] = 1.0;
    for (int k = 1; k < 2 * m; ++k) pw[k] = pw[k - 1] * u;
    for (int r = 0; r < m; ++r) {
      for (int c = 0; c < m; ++c) A[r][c] += pw[r + c];
      A[r][m] += pw[r] * y[i];
    }
  }
  for (int c = 0; c < m; ++c) {
    int piv = c;
    for (int r = c + 1; r < m; ++r)
      if (fabs(A[r][c]) > fabs(A[piv][c])) piv = r;
    for (int k = 0; k <= m; ++k) std::swap(A[c][k], A[piv][k]);
    const double d = A[c][c];
    if (d == 0.0) continue;
    for (int r = 0; r < m; ++r) {
      if (r == c) continue;
      const double f = A[r][c] / d;
      for (int k = c; k <= m; ++k) A[r][k] -= f * A[c][k];
    }
  }
  const double u0 = (x0 - mean) / span;
  double v = 0.0, pw = 1.0;
  for (int c = 0; c < m; ++c) {
    if (A[c][c] != 0.0) v += (A[c][m] / A[c][c]) * pw;
    pw *= u0;
  }
  return v;
}

}  // namespace

namespace prr {

// Arguments were validated by the C ABI (prr_pick_delta).
float pick_delta(const int32_t* context, const float* delta, const float* select_us, const float* spec_us, int n_rows,
                 int32_t query_context, int degree, float* select_est, float* spec_est) {
  std::vector<float> deltas(delta, delta + n_rows);
  std::sort(deltas.begin(), deltas.end());
  deltas.erase(std::unique(deltas.begin(), deltas.end()), deltas.end());
  float best = 1.0f;
  const double x0 = log2((double)query_context);
  for (float d : deltas) {
    std::vector<double> x, ys, yp;
    bool exact = false;
    double es = 0.0, ep = 0.0;
    for (int i = 0; i < n_rows; ++i) {
      if (delta[i] != d) continue;
      if (context[i] == query_context) {  // a profiled context: the measurement itself
        exact = true;
        es = select_us[i];
        ep = spec_us[i];
      }
      x.push_back(log2((double)context[i]));
      ys.push_back(select_us[i]);
      yp.push_back(spec_us[i]);
    }
    if (!exact) {
      std::vector<double> ux(x);
      std::sort(ux.begin(), ux.end());
      const int distinct = (int)(std::unique(ux.begin(), ux.end()) - ux.begin());
      const int deg = std::max(0, std::min(degree, distinct - 1));
      es = poly_fit_eval(x, ys, deg, x0);
      ep = poly_fit_eval(x, yp, deg, x0);
    }
    // deltas ascend: the estimates reported are those of the smallest delta until a
    // delta fits, then of the largest one that fits
    if (d == deltas.front() || ep <= es) {
      if (select_est) *select_est = (float)es;
      if (spec_est) *spec_est = (float)ep;
    }
    if (ep <= es) best = std::max(best, d);
  }
  return best;
}

}  // namespace prr
