// Host driver for the rung planner and its decoder-side re-derivation, built
// with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_schedule_sanitized.py: random descriptors (valid ones, and ones
// each argument check must reject) go through seedq_plan_schedule and
// seedq_derive_schedule; every valid plan must be re-derived bit for bit and
// meet its budget exactly. Any memory or undefined-behaviour error aborts.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "seedq.h"

namespace seedq {
int plan_schedule(const seedq_schedule_desc* d, uint8_t* rob, seedq_schedule_report* rep);
int derive_schedule(const seedq_schedule_desc* d, double lam, double qf, int64_t T, uint8_t* rob);
}  // namespace seedq

namespace {

uint64_t state = 0x9E3779B97F4A7C15ull;
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

int main(int argc, char** argv) {
  const int cases = argc > 1 ? std::atoi(argv[1]) : 2000;
  int planned = 0, rejected = 0;
  for (int c = 0; c < cases; ++c) {
    const int64_t nrows = 1 + below(40), ncols = 8 * (1 + below(50));
    const int64_t nb = nrows * (ncols / 8);
    const int nr = 1 + below(5);
    std::vector<seedq_rung> rungs;
    int K = 8 + below(4), P = 1 + below(2);
    for (int r = 0; r < nr; ++r) {  // ascending rate K + 4P + 4
      rungs.push_back({K, P});
      K += 1 + below(3);
      P = P + below(2) > 6 ? 6 : P + below(2);
      if (K > 24) K = 24;
    }
    std::vector<double> damage(nr);
    double d = 1.0 + 4.0 * unit(), slope = 0.5 + unit();
    for (int r = 0; r < nr; ++r) {
      damage[r] = d;
      d = std::fmax(0.0, d - slope * (rungs[r + 1 < nr ? r + 1 : r].K + 4 * rungs[r + 1 < nr ? r + 1 : r].P - rungs[r].K - 4 * rungs[r].P + 1));
      slope *= 0.3 + 0.8 * unit();   // sometimes not convex: the hull drops rungs
    }
    std::vector<float> col(ncols), row(nrows);
    for (auto& v : col) v = float(0.01 + 10.0 * unit() * unit());
    for (auto& v : row) v = float(0.1 + unit());
    const int64_t lo = int64_t(rungs[0].K + 4 * rungs[0].P + 4) * nb;
    const int64_t hi = int64_t(rungs[nr - 1].K + 4 * rungs[nr - 1].P + 4) * nb;
    int64_t bits = lo + int64_t(unit() * double(hi - lo + 1));
    if (bits > hi) bits = hi;
    seedq_schedule_desc desc;
    std::memset(&desc, 0, sizeof(desc));
    desc.nrows = nrows;
    desc.ncols = ncols;
    desc.C = 8;
    desc.nrungs = nr;
    desc.rungs = rungs.data();
    desc.damage = damage.data();
    desc.target_bpw = double(bits) / double(8 * nb);
    desc.col_importance = col.data();
    desc.row_importance = below(2) == 0 ? nullptr : row.data();
    desc.floor_fraction = below(3) == 0 ? 0.0 : 0.3 * unit();
    // one argument in four is broken in a way the checks must catch
    const int fault = below(4) == 0 ? 1 + below(9) : 0;
    switch (fault) {
      case 1: desc.ncols = ncols + 3; break;
      case 2: desc.nrungs = 0; break;
      case 3: desc.nrungs = SEEDQ_MAX_RUNGS + 1; break;
      case 4: desc.target_bpw = std::nan(""); break;
      case 5: desc.target_bpw = double(lo - 8) / double(8 * nb); break;
      case 6: if (below(2)) col[below(int(ncols))] = -1.0f; else desc.col_importance = nullptr; break;
      case 7: if (desc.row_importance) row[below(int(nrows))] = std::nanf(""); else desc.rungs = nullptr; break;
      case 8: desc.floor_fraction = -0.5; break;
      case 9: rungs[0].K = 30; break;
      default: break;
    }
    std::vector<uint8_t> rob(size_t(nb), 0xEE), rob2(size_t(nb), 0xDD);
    seedq_schedule_report rep;
    const int rc = seedq::plan_schedule(&desc, rob.data(), &rep);
    if (fault) {
      check(rc != SEEDQ_OK, "a broken argument was accepted", c);
      for (uint8_t v : rob) check(v == 0xEE, "output written on error", c);
      ++rejected;
      continue;
    }
    if (rc != SEEDQ_OK) {
      // a valid descriptor may still be infeasible once the hull drops rungs
      check(rc == SEEDQ_ERATE || rc == SEEDQ_EHULL, "unexpected error code", c);
      ++rejected;
      continue;
    }
    ++planned;
    int64_t total = 0;
    for (int64_t b = 0; b < nb; ++b) {
      check(rob[b] < nr, "rung index out of range", c);
      if (rob[b] < nr) total += rungs[rob[b]].K + 4 * rungs[rob[b]].P + 4;
    }
    // the tie pass meets the budget from below, within one block's rate step,
    // unless the budget is above what the top rung of the hull gives every block
    int top = -1;
    for (int r = 0; r < nr; ++r)
      if (rep.on_hull[r]) top = r;
    bool all_top = top >= 0;
    for (int64_t b = 0; b < nb; ++b) all_top = all_top && rob[b] == top;
    const int64_t step = hi / nb - lo / nb;
    check(total == rep.total_bits && total <= rep.budget_bits, "total above the budget", c);
    check(rep.budget_bits - total < (step > 0 ? step : 1) || all_top, "budget missed by more than a step", c);
    const int rc2 = seedq::derive_schedule(&desc, rep.lambda, rep.floor_q, rep.tie_count, rob2.data());
    check(rc2 == SEEDQ_OK && rob2 == rob, "re-derivation differs", c);
  }
  std::printf("cases %d planned %d rejected %d failures %d\n", cases, planned, rejected, failures);
  return failures == 0 ? 0 : 1;
}
