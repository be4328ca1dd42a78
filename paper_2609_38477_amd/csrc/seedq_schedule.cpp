// Host planner for the rung schedule (sections 3.2-3.4, Algorithms 1-2).
//
// Importance (eq. (imp)): imp_b = abar_g * rho_r, abar_g the mean of the fp32
// column importances a_j over the block's 8 columns, both factors normalised to
// unit mean; every sum runs in index order in fp64 (appendix "Agreement").
// Floor (section 3.3): q = sorted(imp)[ceil(f * nblocks) - 1], imp <- max(imp, q).
// Hull (section 3.4): the lower convex hull of the rungs' (rate, damage) points, slopes
// s_j = (e_j - e_{j+1}) / (r_{j+1} - r_j) in bits per weight.
// Ladder (eq. (ladder)): a block of importance v sits at hull position
// |{j : fl(lambda / s_j) <= v}|.
//
// Instead of bisecting on lambda, the planner sweeps the exact breakpoints of
// that ladder: for every distinct importance v and hull step j, the largest
// double lambda with fl(lambda / s_j) <= v. Walking the breakpoints from the
// largest down promotes whole groups of equally important blocks; the first
// group that does not fit is the tied group of the tie pass: its blocks are
// lowered one rung, earliest first in row-major order, until the total fits
// the budget (Algorithm 2 lowers T_t of them). The result equals bisection plus the tie
// pass (Everett's theorem), without floating-point search.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <thread>
#include <vector>

#include "seedq_internal.h"

namespace seedq {
namespace {

struct Breakpoint {
  double lam;
  int cls;   // importance class
  int step;  // hull step j (promotion from position j to j + 1)
};

// The sweep's order: larger lambda first, then the lower class, then the
// lower step.
bool before(const Breakpoint& a, const Breakpoint& b) {
  if (a.lam != b.lam) return a.lam > b.lam;
  if (a.cls != b.cls) return a.cls < b.cls;
  return a.step < b.step;
}

// Runs f(t, begin, end) on nt threads over [0, n) in contiguous chunks (the
// planner's large-input loops; every chunk's work is independent, so the
// result does not depend on the thread count).
template <typename F>
void parallel_chunks(int64_t n, int nt, F&& f) {
  if (nt <= 1 || n < 2 * nt) {
    f(0, int64_t(0), n);
    return;
  }
  std::vector<std::thread> th;
  th.reserve(size_t(nt - 1));
  for (int t = 1; t < nt; ++t)
    th.emplace_back([&, t] { f(t, n * t / nt, n * (t + 1) / nt); });
  f(0, int64_t(0), n / nt);
  for (auto& x : th) x.join();
}

int planner_threads(int64_t n) {
  if (n < (int64_t(1) << 18)) return 1;
  const unsigned hc = std::thread::hardware_concurrency();
  return int(std::max(1u, std::min(hc, 16u)));
}

// Indices 0..n-1 ordered by v ascending, equal values by index (and the values
// in that order, in sorted_v). Large inputs take a stable LSD radix sort on the
// bit patterns of v (the values are positive and finite, so their bits order
// like them), 11 bits per pass (a bucket table that stays in cache), passes
// whose digit every key shares skipped, each pass split over threads (per-thread
// counts, offsets in thread order, so the scatter stays stable); small inputs
// std::sort.
std::vector<int64_t> order_by_value(const std::vector<double>& v, std::vector<double>& sorted_v) {
  const int64_t n = int64_t(v.size());
  std::vector<int64_t> idx(n);
  sorted_v.resize(size_t(n));
  if (n < (int64_t(1) << 16)) {
    for (int64_t i = 0; i < n; ++i) idx[i] = i;
    std::sort(idx.begin(), idx.end(), [&](int64_t a, int64_t b) {
      return v[a] < v[b] || (v[a] == v[b] && a < b);
    });
    for (int64_t k = 0; k < n; ++k) sorted_v[k] = v[idx[k]];
    return idx;
  }
  const int nt = planner_threads(n);
  std::vector<uint64_t> key(n), key2(n);
  std::vector<int64_t> idx2(n);
  parallel_chunks(n, nt, [&](int, int64_t b, int64_t e) {
    for (int64_t i = b; i < e; ++i) {
      std::memcpy(&key[i], &v[i], sizeof(double));
      idx[i] = i;
    }
  });
  constexpr int kBits = 11, kBuckets = 1 << kBits;
  constexpr uint64_t kMask = kBuckets - 1;
  std::vector<int64_t> cnt(size_t(nt) * kBuckets);
  for (int shift = 0; shift < 64; shift += kBits) {
    std::fill(cnt.begin(), cnt.end(), 0);
    parallel_chunks(n, nt, [&](int t, int64_t b, int64_t e) {
      int64_t* c = cnt.data() + size_t(t) * kBuckets;
      for (int64_t i = b; i < e; ++i) ++c[(key[i] >> shift) & kMask];
    });
    const uint64_t d0 = (key[0] >> shift) & kMask;
    int64_t same = 0;
    for (int t = 0; t < nt; ++t) same += cnt[size_t(t) * kBuckets + d0];
    if (same == n) continue;   // one digit for all
    int64_t run = 0;
    for (int d = 0; d < kBuckets; ++d)
      for (int t = 0; t < nt; ++t) {
        int64_t& c = cnt[size_t(t) * kBuckets + d];
        const int64_t x = c;
        c = run;
        run += x;
      }
    parallel_chunks(n, nt, [&](int t, int64_t b, int64_t e) {
      int64_t* c = cnt.data() + size_t(t) * kBuckets;
      for (int64_t i = b; i < e; ++i) {
        const int64_t pos = c[(key[i] >> shift) & kMask]++;
        key2[pos] = key[i];
        idx2[pos] = idx[i];
      }
    });
    key.swap(key2);
    idx.swap(idx2);
  }
  std::memcpy(sorted_v.data(), key.data(), sizeof(double) * size_t(n));
  return idx;
}

// The neighbouring doubles of a non-negative finite x: for these the bit
// pattern counts the representable values (std::nextafter's result, without
// the library call).
double next_up(double x) {
  uint64_t b;
  std::memcpy(&b, &x, sizeof b);
  ++b;
  std::memcpy(&x, &b, sizeof b);
  return x;
}
double next_down(double x) {   // x > 0
  uint64_t b;
  std::memcpy(&b, &x, sizeof b);
  --b;
  std::memcpy(&x, &b, sizeof b);
  return x;
}

// Largest lambda >= 0 with fl(lambda / s) <= v (v > 0, s > 0).
double breakpoint(double v, double s) {
  double lam = v * s;
  if (!std::isfinite(lam)) lam = std::nextafter(INFINITY, 0.0);
  while (lam > 0.0 && lam / s > v) lam = next_down(lam);
  for (;;) {
    const double up = next_up(lam);
    if (std::isfinite(up) && up / s <= v) lam = up;
    else break;
  }
  return lam;
}

// What the encoder and the decoder both derive from the descriptor: block
// importance factors (unit mean, fixed evaluation order), the hull and its
// slopes. Returns SEEDQ_OK or the error code of the first problem found.
struct Prepared {
  int64_t nrows = 0, G = 0, nb = 0;
  std::vector<double> bits;   // K + 4P + 4 per rung
  std::vector<double> abar;   // per column group, unit mean
  std::vector<double> rho;    // per row, unit mean; empty for rho = 1
  std::vector<int> H;         // hull vertices (rung indices), increasing rate
  std::vector<double> slope;  // s_j, bits per weight
  double imp(int64_t b) const { return rho.empty() ? 1.0 * abar[b % G] : rho[b / G] * abar[b % G]; }
};

int prepare(const seedq_schedule_desc* d, Prepared& p) {
  if (!d || !d->rungs || !d->col_importance) return SEEDQ_EINVAL;
  if (d->C != kC) return SEEDQ_EUNSUPPORTED;
  if (d->nrows <= 0 || d->ncols <= 0 || d->ncols % kC != 0) return SEEDQ_EINVAL;
  if (d->nrungs < 1 || d->nrungs > SEEDQ_MAX_RUNGS) return SEEDQ_EINVAL;
  const int R = d->nrungs;
  for (int r = 0; r < R; ++r)
    if (!rung_supported(d->rungs[r].K, d->rungs[r].P)) return SEEDQ_EUNSUPPORTED;
  if (R > 1) {
    if (!d->damage) return SEEDQ_EHULL;
    for (int r = 0; r < R; ++r)
      if (!std::isfinite(d->damage[r])) return SEEDQ_EHULL;
  }
  p.nrows = d->nrows;
  p.G = d->ncols / kC;
  if (p.nrows > (int64_t(1) << 40) / p.G) return SEEDQ_EINVAL;
  p.nb = p.nrows * p.G;
  p.bits.resize(R);
  for (int r = 0; r < R; ++r) p.bits[r] = double(d->rungs[r].K + 4 * d->rungs[r].P + 4);

  // ---- importance (eq. (imp)), fixed evaluation order
  const int64_t G = p.G, nrows = p.nrows;
  p.abar.assign(G, 0.0);
  for (int64_t g = 0; g < G; ++g) {
    double s = 0.0;
    for (int j = 0; j < kC; ++j) {
      const double a = double(d->col_importance[g * kC + j]);
      if (!(a > 0.0) || !std::isfinite(a)) return SEEDQ_EINVAL;
      s = s + a;
    }
    p.abar[g] = s / 8.0;
  }
  double tot = 0.0;
  for (int64_t g = 0; g < G; ++g) tot = tot + p.abar[g];
  const double amean = tot / double(G);
  for (int64_t g = 0; g < G; ++g) p.abar[g] = p.abar[g] / amean;
  p.rho.clear();
  if (d->row_importance) {
    p.rho.resize(nrows);
    double tr = 0.0;
    for (int64_t r = 0; r < nrows; ++r) {
      const double v = double(d->row_importance[r]);
      if (!(v > 0.0) || !std::isfinite(v)) return SEEDQ_EINVAL;
      tr = tr + v;
    }
    const double rmean = tr / double(nrows);
    for (int64_t r = 0; r < nrows; ++r) p.rho[r] = double(d->row_importance[r]) / rmean;
  }

  // ---- hull (section 3.4)
  const std::vector<double>& bits = p.bits;
  std::vector<int>& H = p.H;
  H.clear();
  if (R == 1) {
    H.push_back(0);
  } else {
    std::vector<int> order(R);
    for (int r = 0; r < R; ++r) order[r] = r;
    std::sort(order.begin(), order.end(), [&](int a, int b) {
      if (bits[a] != bits[b]) return bits[a] < bits[b];
      if (d->damage[a] != d->damage[b]) return d->damage[a] < d->damage[b];
      return a < b;
    });
    for (int i : order) {
      if (!H.empty() && bits[H.back()] == bits[i]) continue;
      while (H.size() >= 2) {
        const int a = H[H.size() - 2], b = H.back();
        const double cross = (bits[b] - bits[a]) * (d->damage[i] - d->damage[a]) -
                             (d->damage[b] - d->damage[a]) * (bits[i] - bits[a]);
        if (cross <= 0.0) H.pop_back();
        else break;
      }
      H.push_back(i);
    }
    while (H.size() >= 2 && d->damage[H.back()] >= d->damage[H[H.size() - 2]]) H.pop_back();
  }
  const int J = int(H.size());
  if (J < 1) return SEEDQ_EHULL;
  p.slope.assign(J > 1 ? J - 1 : 0, 0.0);
  for (int j = 0; j + 1 < J; ++j)
    p.slope[j] = (d->damage[H[j]] - d->damage[H[j + 1]]) / ((bits[H[j + 1]] - bits[H[j]]) / 8.0);
  return SEEDQ_OK;
}

}  // namespace

int plan_schedule(const seedq_schedule_desc* d, uint8_t* rob, seedq_schedule_report* rep) {
  if (!rob) return SEEDQ_EINVAL;
  Prepared pr;
  const int rc = prepare(d, pr);
  if (rc != SEEDQ_OK) return rc;
  if (!(d->floor_fraction >= 0.0 && d->floor_fraction < 1.0)) return SEEDQ_EINVAL;
  const int R = d->nrungs;
  const int64_t nrows = pr.nrows, G = pr.G, nb = pr.nb;
  const double budget_f = 8.0 * d->target_bpw * double(nb);
  if (!std::isfinite(budget_f) || budget_f < 0.0 || budget_f >= 9.0e18 ||
      budget_f != std::floor(budget_f))
    return SEEDQ_ERATE;
  const int64_t budget = int64_t(budget_f);
  const std::vector<double>& bits = pr.bits;
  const std::vector<double>& abar = pr.abar;
  const std::vector<double>& rho = pr.rho;
  auto imp_of = [&](int64_t b) -> double { return pr.imp(b); };

  // ---- floor (section 3.3)
  int64_t kq = int64_t(std::ceil(double(nb) * d->floor_fraction)) - 1;
  if (kq < 0) kq = 0;
  if (kq > nb - 1) kq = nb - 1;
  double qf;
  if (rho.empty()) {
    std::vector<double> sg(abar);
    std::sort(sg.begin(), sg.end());
    qf = 1.0 * sg[kq / nrows];
  } else {
    std::vector<double> all(nb);
    parallel_chunks(nrows, planner_threads(nb), [&](int, int64_t r0, int64_t r1) {
      for (int64_t r = r0; r < r1; ++r)
        for (int64_t g = 0; g < G; ++g) all[r * G + g] = rho[r] * abar[g];   // = imp_of(r G + g)
    });
    std::nth_element(all.begin(), all.begin() + kq, all.end());
    qf = all[kq];
  }

  // ---- importance classes: equal floored importance
  // cls_of_group (rho == 1) or cls_of_block (general); members listed in block order
  std::vector<double> cls_val;
  std::vector<int64_t> cls_count;
  std::vector<int32_t> cls_of;  // per group (rho == 1) or per block
  {
    const int64_t n = rho.empty() ? G : nb;
    auto val = [&](int64_t i) { return std::max(rho.empty() ? 1.0 * abar[i] : imp_of(i), qf); };
    std::vector<double> v(n);
    if (rho.empty()) {
      for (int64_t i = 0; i < n; ++i) v[i] = val(i);
    } else {
      parallel_chunks(nrows, planner_threads(n), [&](int, int64_t r0, int64_t r1) {
        for (int64_t r = r0; r < r1; ++r)
          for (int64_t g = 0; g < G; ++g) v[r * G + g] = std::max(rho[r] * abar[g], qf);   // = val(r G + g)
      });
    }
    std::vector<double> sv;
    const std::vector<int64_t> idx = order_by_value(v, sv);
    // class of every rank (a new class where the value changes), then the
    // scatter to block order
    std::vector<int32_t> cls_at(static_cast<size_t>(n));
    for (int64_t k = 0; k < n; ++k) {
      if (cls_val.empty() || sv[k] != cls_val.back()) {
        cls_val.push_back(sv[k]);
        cls_count.push_back(0);
      }
      cls_at[k] = int32_t(cls_val.size() - 1);
      cls_count.back() += rho.empty() ? nrows : 1;
    }
    cls_of.assign(n, -1);
    parallel_chunks(n, planner_threads(n), [&](int, int64_t k0, int64_t k1) {
      for (int64_t k = k0; k < k1; ++k) cls_of[idx[k]] = cls_at[k];
    });
  }
  const int ncls = int(cls_val.size());

  const std::vector<int>& H = pr.H;
  const int J = int(H.size());
  const std::vector<double>& slope = pr.slope;

  if (double(nb) * bits[H[0]] > double(budget)) return SEEDQ_ERATE;

  // ---- breakpoint sweep
  // For one step the breakpoint grows with the class value, and the classes
  // are numbered by increasing value: each step's list comes out in sweep
  // order by walking the classes downwards (equal breakpoints of neighbouring
  // classes put back in class order), and the lists are merged.
  std::vector<int> level(ncls, 0);
  std::vector<Breakpoint> ev;
  ev.reserve(size_t(ncls) * (J > 1 ? J - 1 : 0));
  {
    std::vector<std::vector<Breakpoint>> lists(J > 1 ? J - 1 : 0);
    for (int j = 0; j + 1 < J; ++j) {
      std::vector<Breakpoint>& L = lists[j];
      L.resize(size_t(ncls));
      parallel_chunks(ncls, planner_threads(ncls), [&](int, int64_t b, int64_t e) {
        for (int64_t i = b; i < e; ++i) {
          const int c = ncls - 1 - int(i);
          L[size_t(i)] = {breakpoint(cls_val[c], slope[j]), c, j};
        }
      });
      for (size_t a = 0; a < L.size();) {
        size_t b = a + 1;
        while (b < L.size() && L[b].lam == L[a].lam) ++b;
        std::reverse(L.begin() + long(a), L.begin() + long(b));
        a = b;
      }
    }
    std::vector<size_t> at(lists.size(), 0);
    for (;;) {
      int best = -1;
      for (int j = 0; j < int(lists.size()); ++j)
        if (at[j] < lists[j].size() && (best < 0 || before(lists[j][at[j]], lists[best][at[best]])))
          best = j;
      if (best < 0) break;
      ev.push_back(lists[best][at[best]++]);
    }
  }

  int64_t total = nb * int64_t(bits[H[0]]);
  double lam = 0.0;
  int64_t T = 0;
  // tied group (if any): classes promoted at the final threshold, and how many
  // of their blocks (in block order) keep the lower position
  std::vector<int> tied_cls;
  std::vector<int> tied_from;  // position before the threshold, per tied class
  size_t k = 0;
  bool done = false;
  while (k < ev.size() && !done) {
    size_t k1 = k;
    while (k1 < ev.size() && ev[k1].lam == ev[k].lam) ++k1;
    const double lk = ev[k].lam;
    if (total == budget) {
      lam = std::nextafter(lk, INFINITY);
      done = true;
      break;
    }
    int64_t delta = 0;
    for (size_t t = k; t < k1; ++t) {
      const int c = ev[t].cls, j = ev[t].step;
      delta += cls_count[c] * int64_t(bits[H[j + 1]] - bits[H[j]]);
    }
    if (total + delta <= budget) {
      for (size_t t = k; t < k1; ++t) level[ev[t].cls] = ev[t].step + 1;
      total += delta;
      k = k1;
      continue;
    }
    // tie pass over the classes promoted at lk
    std::vector<int> from_of(ncls, -1);
    for (size_t t = k; t < k1; ++t) {
      const int c = ev[t].cls;
      if (from_of[c] < 0) {
        from_of[c] = level[c];
        tied_cls.push_back(c);
      }
    }
    std::sort(tied_cls.begin(), tied_cls.end());
    std::vector<int> to_of(ncls, -1);
    for (size_t t = k; t < k1; ++t) to_of[ev[t].cls] = std::max(to_of[ev[t].cls], ev[t].step + 1);
    int64_t cur = total + delta;
    int64_t members = 0;
    for (int c : tied_cls) members += cls_count[c];
    // lower members, earliest block first, until the total fits the budget
    auto gain = [&](int c) {
      return int64_t(bits[H[to_of[c]]] - bits[H[from_of[c]]]);
    };
    T = 0;
    if (rho.empty()) {
      // block order over the tied groups: rows outer, groups inner
      std::vector<int64_t> groups;
      for (int64_t g = 0; g < G; ++g)
        if (from_of[cls_of[g]] >= 0) groups.push_back(g);
      for (int64_t r = 0; r < nrows && cur > budget; ++r)
        for (size_t gi = 0; gi < groups.size() && cur > budget; ++gi) {
          cur -= gain(cls_of[groups[gi]]);
          ++T;
        }
    } else {
      for (int64_t b = 0; b < nb && cur > budget; ++b) {
        const int c = cls_of[b];
        if (from_of[c] >= 0) {
          cur -= gain(c);
          ++T;
        }
      }
    }
    if (T == members) {
      lam = std::nextafter(lk, INFINITY);
      T = 0;
      tied_cls.clear();
    } else {
      lam = lk;
      for (int c : tied_cls) {
        tied_from.push_back(from_of[c]);
        level[c] = to_of[c];
      }
      total = cur;
    }
    done = true;
  }
  if (!done) lam = 0.0;

  // ---- write the allocation
  int64_t count[SEEDQ_MAX_RUNGS] = {0};
  std::vector<int> cls_tied_from(ncls, -1);
  for (size_t t = 0; t < tied_cls.size(); ++t) cls_tied_from[tied_cls[t]] = tied_from[t];
  int64_t demote_left = T;
  if (rho.empty()) {
    // every row has the same rungs; the first T tied blocks in block order
    // (row-major) take the lower rung
    std::vector<uint8_t> row(G);
    for (int64_t g = 0; g < G; ++g) row[g] = uint8_t(H[level[cls_of[g]]]);
    for (int64_t r = 0; r < nrows; ++r) std::memcpy(rob + r * G, row.data(), size_t(G));
    for (int64_t g = 0; g < G; ++g) count[row[g]] += nrows;
    for (int64_t r = 0; r < nrows && demote_left > 0; ++r)
      for (int64_t g = 0; g < G && demote_left > 0; ++g) {
        const int c = cls_of[g];
        if (cls_tied_from[c] < 0) continue;
        const int rr = H[cls_tied_from[c]];
        count[rob[r * G + g]] -= 1;
        rob[r * G + g] = uint8_t(rr);
        count[rr] += 1;
        --demote_left;
      }
  } else {
    for (int64_t b = 0; b < nb; ++b) {
      const int c = cls_of[b];
      int pos = level[c];
      if (cls_tied_from[c] >= 0 && demote_left > 0) {
        pos = cls_tied_from[c];
        --demote_left;
      }
      const int rr = H[pos];
      rob[b] = uint8_t(rr);
      count[rr] += 1;
    }
  }
  int64_t check_total = 0;
  for (int r = 0; r < R; ++r) check_total += count[r] * int64_t(bits[r]);
  if (rep) {
    std::memset(rep, 0, sizeof(*rep));
    rep->lambda = lam;
    rep->floor_q = qf;
    rep->tie_count = T;
    rep->total_bits = check_total;
    rep->budget_bits = budget;
    for (int r = 0; r < R; ++r) rep->count[r] = count[r];
    for (int j = 0; j < J; ++j) rep->on_hull[H[j]] = 1;
    rep->nhull = J;
  }
  return SEEDQ_OK;
}

// Decoder side of Algorithm 2: the same importance, floor value and hull as the
// encoder, the ladder at the stored lambda, and the first T blocks (row-major)
// that sit exactly at a threshold -- promoted at lambda but not at the next
// larger double -- taking the lower rung. With the lambda, floor value and tie
// count that plan_schedule reports, this reproduces its allocation exactly.
int derive_schedule(const seedq_schedule_desc* d, double lam, double qf, int64_t T, uint8_t* rob) {
  if (!rob) return SEEDQ_EINVAL;
  if (!(lam >= 0.0) || !std::isfinite(lam) || !std::isfinite(qf) || T < 0) return SEEDQ_EINVAL;
  Prepared pr;
  const int rc = prepare(d, pr);
  if (rc != SEEDQ_OK) return rc;
  const int64_t nrows = pr.nrows, G = pr.G, nb = pr.nb;
  const std::vector<int>& H = pr.H;
  const int J = int(H.size());
  const std::vector<double>& slope = pr.slope;

  const double lam_up = std::nextafter(lam, INFINITY);
  auto position = [&](double l, double v) {
    int pos = 0;
    for (int j = 0; j + 1 < J; ++j) pos += (l / slope[j] <= v) ? 1 : 0;
    return pos;
  };
  if (pr.rho.empty()) {
    std::vector<uint8_t> row(G), lower(G);
    std::vector<char> tied(G);
    int64_t ntied = 0;
    for (int64_t g = 0; g < G; ++g) {
      const double v = std::max(1.0 * pr.abar[g], qf);
      const int p = position(lam, v), pu = position(lam_up, v);
      row[g] = uint8_t(H[p]);
      lower[g] = uint8_t(H[pu]);
      tied[g] = p != pu;
      ntied += tied[g] ? nrows : 0;
    }
    if (T > ntied) return SEEDQ_EINVAL;
    for (int64_t r = 0; r < nrows; ++r) std::memcpy(rob + r * G, row.data(), size_t(G));
    int64_t left = T;
    for (int64_t r = 0; r < nrows && left > 0; ++r)
      for (int64_t g = 0; g < G && left > 0; ++g)
        if (tied[g]) {
          rob[r * G + g] = lower[g];
          --left;
        }
  } else {
    std::vector<uint8_t> pos(nb), pos_up(nb);
    int64_t ntied = 0;
    for (int64_t b = 0; b < nb; ++b) {
      const double v = std::max(pr.imp(b), qf);
      pos[b] = uint8_t(position(lam, v));
      pos_up[b] = uint8_t(position(lam_up, v));
      ntied += pos[b] != pos_up[b] ? 1 : 0;
    }
    if (T > ntied) return SEEDQ_EINVAL;
    int64_t left = T;
    for (int64_t b = 0; b < nb; ++b) {
      int p = pos[b];
      if (left > 0 && pos_up[b] != p) {
        p = pos_up[b];
        --left;
      }
      rob[b] = uint8_t(H[p]);
    }
  }
  return SEEDQ_OK;
}

}  // namespace seedq
