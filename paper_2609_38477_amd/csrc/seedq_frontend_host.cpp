// Host parts of the importance front end: Gauss-Hermite nodes and weights, the
// channel sort before blocking, and the ranking of outlier-column candidates
// (appendix on outlier columns).
#include <algorithm>
#include <cmath>
#include <cstring>
#include <tuple>
#include <vector>

#include "seedq_internal.h"

namespace seedq {
namespace {

// Orthonormal Hermite polynomials for the weight e^{-x^2}:
// q_0 = pi^{-1/4}, q_j = x sqrt(2/j) q_{j-1} - sqrt((j-1)/j) q_{j-2}.
// Returns q_n(x) and, in *sumsq, sum_{j<n} q_j(x)^2.
double hermite_q(int n, double x, double* sumsq) {
  double qm = 0.0, q = std::pow(M_PI, -0.25), s = 0.0;
  for (int j = 1; j <= n; ++j) {
    s += q * q;
    const double qn = x * std::sqrt(2.0 / j) * q - std::sqrt(double(j - 1) / j) * qm;
    qm = q;
    q = qn;
  }
  if (sumsq) *sumsq = s;
  return q;
}

}  // namespace

// Gauss-Hermite rule for the weight e^{-x^2}: the nodes are the zeros of q_n,
// bracketed by sign changes on a grid finer than their smallest spacing and
// refined by bisection to the last bit; the weights come from the
// Christoffel-Darboux identity w_i = 1 / sum_{j<n} q_j(x_i)^2. Nodes ascending.
int gauss_hermite(int n, double* x, double* w) {
  if (n < 1 || n > 256 || !x || !w) return SEEDQ_EINVAL;
  std::vector<double> pos;  // non-negative roots, ascending
  const double top = std::sqrt(2.0 * n + 1.0) + 1.0;
  const double step = 0.25 / std::sqrt(2.0 * n + 1.0);  // well below the root spacing
  double a = 0.0, fa = hermite_q(n, a, nullptr);
  if (n % 2 == 1) pos.push_back(0.0);  // odd n: 0 is a root
  if (n % 2 == 1) {
    a = step;
    fa = hermite_q(n, a, nullptr);
  }
  for (double b = a + step; a < top; b += step) {
    const double fb = hermite_q(n, b, nullptr);
    if ((fa < 0) != (fb < 0)) {
      double lo = a, hi = b, flo = fa;
      for (int it = 0; it < 200 && std::nextafter(lo, hi) < hi; ++it) {
        const double mid = 0.5 * (lo + hi);
        const double fm = hermite_q(n, mid, nullptr);
        if ((fm < 0) == (flo < 0)) {
          lo = mid;
          flo = fm;
        } else {
          hi = mid;
        }
      }
      pos.push_back(0.5 * (lo + hi));
    }
    a = b;
    fa = fb;
  }
  if (int(pos.size()) != (n + 1) / 2) return SEEDQ_EINVAL;
  for (int i = 0; i < int(pos.size()); ++i) {
    double s;
    hermite_q(n, pos[i], &s);
    const double wi = 1.0 / s;
    x[n / 2 + i] = pos[i];
    w[n / 2 + i] = wi;
    x[(n - 1) / 2 - i] = -pos[i];
    w[(n - 1) / 2 - i] = wi;
  }
  return SEEDQ_OK;
}

void channel_order(const float* a, int64_t n, int32_t* perm) {
  for (int64_t i = 0; i < n; ++i) perm[i] = int32_t(i);
  std::stable_sort(perm, perm + n, [&](int32_t i, int32_t j) { return a[i] < a[j]; });
}

int select_outliers(int32_t ntensors, const int64_t* ncols, const double* const* maxabs,
                    const double* const* median, const double* const* a, int32_t keep,
                    int32_t* out_tensor, int32_t* out_col, int32_t* out_count) {
  if (ntensors < 0 || keep < 0 || !out_count || (ntensors > 0 && (!ncols || !maxabs || !median || !a)))
    return SEEDQ_EINVAL;
  if (keep > 0 && (!out_tensor || !out_col)) return SEEDQ_EINVAL;
  const double kDR = 1.0e3, kAct = 1.0e2, kEps = std::ldexp(1.0, -24);
  const size_t kPerRule = 32;
  // (-statistic, tensor, column): ascending order = largest statistic first,
  // ties by tensor then column
  std::vector<std::tuple<double, int32_t, int32_t>> dr, act;
  for (int32_t t = 0; t < ntensors; ++t) {
    if (ncols[t] <= 0 || !maxabs[t] || !median[t] || !a[t]) return SEEDQ_EINVAL;
    double s = 0.0;
    for (int64_t j = 0; j < ncols[t]; ++j) s += a[t][j];
    const double mean = s / double(ncols[t]);
    for (int64_t j = 0; j < ncols[t]; ++j) {
      const double mx = maxabs[t][j];
      const double r = mx > 0.0 ? mx / (median[t][j] + kEps * mx) : 0.0;
      if (r >= kDR) dr.emplace_back(-r, t, int32_t(j));
      if (a[t][j] >= kAct * mean) act.emplace_back(-a[t][j], t, int32_t(j));
    }
  }
  std::sort(dr.begin(), dr.end());
  std::sort(act.begin(), act.end());
  if (dr.size() > kPerRule) dr.resize(kPerRule);
  if (act.size() > kPerRule) act.resize(kPerRule);
  // better position of every candidate in the two lists
  std::vector<std::tuple<size_t, int32_t, int32_t>> ranked;
  auto add = [&](const std::vector<std::tuple<double, int32_t, int32_t>>& lst) {
    for (size_t i = 0; i < lst.size(); ++i) {
      const int32_t t = std::get<1>(lst[i]), j = std::get<2>(lst[i]);
      bool found = false;
      for (auto& e : ranked)
        if (std::get<1>(e) == t && std::get<2>(e) == j) {
          std::get<0>(e) = std::min(std::get<0>(e), i);
          found = true;
        }
      if (!found) ranked.emplace_back(i, t, j);
    }
  };
  add(dr);
  add(act);
  std::sort(ranked.begin(), ranked.end());
  const int32_t n = int32_t(std::min(ranked.size(), size_t(keep)));
  for (int32_t i = 0; i < n; ++i) {
    out_tensor[i] = std::get<1>(ranked[i]);
    out_col[i] = std::get<2>(ranked[i]);
  }
  *out_count = n;
  return SEEDQ_OK;
}

}  // namespace seedq
