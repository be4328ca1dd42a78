// Host driver for the importance front end's host code (Gauss-Hermite rule,
// channel sort, outlier selection), built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_schedule_sanitized.py. Valid and
// invalid arguments, ties, zeros, infinities and NaN statistics go through
// every function; results are checked for their invariants. Any memory or
// undefined-behaviour error aborts.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <vector>

#include "seedq.h"

namespace seedq {
int gauss_hermite(int n, double* x, double* w);
void channel_order(const float* a, int64_t n, int32_t* perm);
int select_outliers(int32_t ntensors, const int64_t* ncols, const double* const* maxabs,
                    const double* const* median, const double* const* a, int32_t keep,
                    int32_t* out_tensor, int32_t* out_col, int32_t* out_count);
}  // namespace seedq

namespace {

uint64_t state = 0x2545F4914F6CDD1Dull;
uint64_t next() {  // splitmix64
  uint64_t z = (state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
double unit() { return double(next() >> 11) * 0x1p-53; }
int below(int n) { return int(next() % uint64_t(n)); }

int failures = 0;
void check(bool ok, const char* what, int c) {
  if (!ok) {
    std::printf("case %d: %s\n", c, what);
    ++failures;
  }
}

}  // namespace

int main() {
  // Gauss-Hermite: every n the library accepts, and the ones it rejects
  for (int n = -2; n <= 260; ++n) {
    std::vector<double> x(n > 0 ? n : 1), w(n > 0 ? n : 1);
    const int rc = seedq::gauss_hermite(n, x.data(), w.data());
    if (n < 1 || n > 256) {
      check(rc != SEEDQ_OK, "bad node count accepted", n);
      continue;
    }
    check(rc == SEEDQ_OK, "valid node count rejected", n);
    double s = 0.0;
    for (int i = 0; i < n; ++i) s += w[i];
    check(std::fabs(s - std::sqrt(M_PI)) <= 1e-10, "weights do not sum to sqrt(pi)", n);
    for (int i = 1; i < n; ++i) check(x[i] > x[i - 1], "nodes not ascending", n);
  }
  check(seedq::gauss_hermite(8, nullptr, nullptr) != SEEDQ_OK, "null outputs accepted", 0);
  // channel sort: ties, zeros and wide ranges
  for (int c = 0; c < 300; ++c) {
    const int64_t n = below(300);
    std::vector<float> a(static_cast<size_t>(n));
    for (auto& v : a) v = below(3) == 0 ? float(below(4)) : float(std::ldexp(unit(), below(60) - 30));
    std::vector<int32_t> perm(size_t(n), -1);
    seedq::channel_order(a.data(), n, perm.data());
    std::vector<int32_t> seen(size_t(n), 0);
    for (int64_t k = 0; k < n; ++k) {
      check(perm[k] >= 0 && perm[k] < n, "index out of range", c);
      if (perm[k] >= 0 && perm[k] < n) seen[perm[k]]++;
      if (k > 0 && perm[k] >= 0 && perm[k - 1] >= 0)
        check(a[perm[k - 1]] < a[perm[k]] || (a[perm[k - 1]] == a[perm[k]] && perm[k - 1] < perm[k]),
              "not ordered by (a, index)", c);
    }
    for (int32_t v : seen) check(v == 1, "not a permutation", c);
  }
  // outlier selection over random tensors with extreme statistics
  for (int c = 0; c < 400; ++c) {
    const int nt = below(9);
    std::vector<int64_t> ncols(nt);
    std::vector<std::vector<double>> mx(nt), md(nt), aa(nt);
    std::vector<const double*> pmx(nt), pmd(nt), pa(nt);
    for (int t = 0; t < nt; ++t) {
      ncols[t] = 1 + below(200);
      for (int64_t j = 0; j < ncols[t]; ++j) {
        double m = std::ldexp(unit(), below(40) - 20), med = m * unit();
        const int kind = below(40);
        if (kind == 0) med = 0.0;                 // one weight in the column
        if (kind == 1) m = med = 0.0;             // an all-zero column
        if (kind == 2) m = INFINITY;
        if (kind == 3) med = std::nan("");
        mx[t].push_back(m);
        md[t].push_back(med);
        aa[t].push_back(below(30) == 0 ? 1e4 * unit() : unit());
      }
      pmx[t] = mx[t].data();
      pmd[t] = md[t].data();
      pa[t] = aa[t].data();
    }
    const int keep = below(8);
    std::vector<int32_t> ot(size_t(keep) + 1, -7), oc(size_t(keep) + 1, -7);
    int32_t cnt = -1;
    const int rc = seedq::select_outliers(nt, ncols.data(), pmx.data(), pmd.data(), pa.data(), keep,
                                          ot.data(), oc.data(), &cnt);
    check(rc == SEEDQ_OK, "valid selection rejected", c);
    if (rc != SEEDQ_OK) continue;
    check(cnt >= 0 && cnt <= keep, "count out of range", c);
    for (int i = 0; i < cnt; ++i) {
      check(ot[i] >= 0 && ot[i] < nt, "tensor index out of range", c);
      if (ot[i] >= 0 && ot[i] < nt) check(oc[i] >= 0 && oc[i] < ncols[ot[i]], "column out of range", c);
      for (int k = 0; k < i; ++k) check(ot[k] != ot[i] || oc[k] != oc[i], "duplicate column", c);
    }
    check(ot[keep] == -7 && oc[keep] == -7, "wrote past keep entries", c);
  }
  int32_t cnt = 0;
  check(seedq::select_outliers(-1, nullptr, nullptr, nullptr, nullptr, 4, nullptr, nullptr, &cnt) != SEEDQ_OK,
        "negative tensor count accepted", 0);
  check(seedq::select_outliers(0, nullptr, nullptr, nullptr, nullptr, 4, nullptr, nullptr, &cnt) != SEEDQ_OK,
        "null outputs accepted", 0);
  std::printf("failures %d\n", failures);
  return failures == 0 ? 0 : 1;
}
