"""Oracle for the rung schedule (test infrastructure only).

Follows the paper's allocation in its own order (Algorithm 1, first five steps):

1. the rungs' (rate, damage) points {(r(g), e(g))} reduced to their lower convex hull, slopes s_j = (e_j - e_{j+1}) / (r_{j+1} - r_j)
   (section 3.4, "Damage curve and hull");
2. block importance imp_b = abar_b * rho_{r(b)}, abar_b the mean of a_j over the
   block's 8 columns, both factors normalised to unit mean within the tensor
   (eq. (imp)); stored factors are fp32, evaluated in fp64 in a fixed order
   (appendix "Agreement");
3. floor: q = f-quantile of {imp_b}, imp_b <- max(imp_b, q) (section 3.3);
4. lambda by bisection so that the mean rate meets the target (eq. (lagrangian),
   Everett's theorem, appendix on ties), blocks ranked by the ladder
   j(b) = 1 + |{j : lambda / s_j <= imp_b}| (eq. (ladder));
5. tie pass: blocks of the tied group at the final threshold are lowered one
   rung, earliest first, until the total fits the budget (section 3.4;
   Algorithm 2 lowers T_t of them).

Readings where the paper is silent: the f-quantile is the inverted-CDF
(lower) empirical quantile over blocks; block order is the row-major block
index b = r * (ncols / 8) + g; the bisection runs over the bit patterns of the
non-negative double lambda, so it ends at two adjacent doubles.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def _rate_bits(K: int, P: int) -> int:
    # eq. (rate) with m = e = 4
    return K + 4 * P + 4


def hull(rates: np.ndarray, damage: np.ndarray) -> list[int]:
    """Indices (into the given rungs) of the lower convex hull vertices, by
    increasing rate. Collinear middle points and dominated rungs are dropped."""
    order = sorted(range(len(rates)), key=lambda i: (rates[i], damage[i], i))
    pts: list[int] = []
    for i in order:
        if pts and rates[pts[-1]] == rates[i]:
            continue  # same rate, larger damage (sorted): never on the lower hull
        while len(pts) >= 2:
            a, b = pts[-2], pts[-1]
            # cross product of (b - a) and (i - a); <= 0 means b is not strictly below
            cross = (rates[b] - rates[a]) * (damage[i] - damage[a]) - \
                (damage[b] - damage[a]) * (rates[i] - rates[a])
            if cross <= 0:
                pts.pop()
            else:
                break
        pts.append(i)
    # the allocation only uses the decreasing part (more rate must buy less damage)
    while len(pts) >= 2 and damage[pts[-1]] >= damage[pts[-2]]:
        pts.pop()
    return pts


def hull_slopes(H, rates_bits, damage) -> np.ndarray:
    """s_j = (e_j - e_{j+1}) / (r_{j+1} - r_j) with r in bits per weight
    (r = l / 8, eq. (rate)); one rounding each in fp64."""
    return np.array([(float(damage[H[j]]) - float(damage[H[j + 1]])) /
                     ((float(rates_bits[H[j + 1]]) - float(rates_bits[H[j]])) / 8.0)
                     for j in range(len(H) - 1)], dtype=np.float64)


@dataclass
class ScheduleResult:
    rung_of_block: np.ndarray   # uint8, index into the given rungs
    lam: float
    floor_q: float
    tie_count: int
    total_bits: int
    budget_bits: int
    hull: list
    imp: np.ndarray             # floored importance per block (fp64)


def block_importance(nrows: int, ncols: int, col_importance, row_importance=None) -> np.ndarray:
    """imp_b of eq. (imp), before the floor, row-major over blocks (fp64)."""
    a = np.asarray(col_importance, dtype=np.float32).astype(np.float64)
    G = ncols // 8
    abar = np.empty(G, dtype=np.float64)
    for g in range(G):
        s = 0.0
        for j in range(8):
            s = s + a[8 * g + j]
        abar[g] = s / 8.0
    tot = 0.0
    for g in range(G):
        tot = tot + abar[g]
    abar_n = abar / (tot / G)
    if row_importance is None:
        rho_n = np.ones(nrows, dtype=np.float64)
    else:
        rho = np.asarray(row_importance, dtype=np.float32).astype(np.float64)
        tr = 0.0
        for r in range(nrows):
            tr = tr + rho[r]
        rho_n = rho / (tr / nrows)
    return (rho_n[:, None] * abar_n[None, :]).reshape(-1)


def ladder(imp: np.ndarray, lam: float, slopes: np.ndarray) -> np.ndarray:
    """Hull position (0-based) of every block for multiplier lam, eq. (ladder)."""
    j = np.zeros(imp.shape, dtype=np.int64)
    for s in slopes:
        j += (lam / s <= imp)
    return j


def schedule(nrows: int, ncols: int, rungs, damage, target_bpw: float, col_importance,
             row_importance=None, floor_fraction: float = 0.06) -> ScheduleResult:
    rungs = [tuple(r) for r in rungs]
    nb = nrows * (ncols // 8)
    rates = np.array([_rate_bits(K, P) for K, P in rungs], dtype=np.float64)
    budget_f = 8.0 * target_bpw * nb
    budget = int(round(budget_f))
    if budget != budget_f:
        raise ValueError("budget 8 * target_bpw * nblocks is not an integer")
    imp = block_importance(nrows, ncols, col_importance, row_importance)
    q = float(np.quantile(imp, floor_fraction, method="inverted_cdf"))
    imp = np.maximum(imp, q)
    if len(rungs) == 1:
        H = [0]
    else:
        H = hull(rates, np.asarray(damage, dtype=np.float64))
    bits = np.array([int(rates[h]) for h in H], dtype=np.int64)
    slopes = hull_slopes(H, rates, damage)

    def total(lam):
        return int(bits[ladder(imp, lam, slopes)].sum())

    def to_result(jpos, lam, T):
        rob = np.array(H, dtype=np.uint8)[jpos]
        return ScheduleResult(rob, lam, q, T, int(bits[jpos].sum()), budget, H, imp)

    if len(H) == 1:
        if bits[0] * nb > budget:
            raise ValueError("budget below the single rung's rate")
        return to_result(np.zeros(nb, dtype=np.int64), 0.0, 0)
    if bits[0] * nb > budget:
        raise ValueError("budget below the lowest rung's rate")
    if total(0.0) <= budget:
        return to_result(ladder(imp, 0.0, slopes), 0.0, 0)
    hi = 2.0 * float(imp.max()) * float(slopes[0]) + 1.0
    assert total(hi) == bits[0] * nb
    lo_b = int(np.float64(0.0).view(np.int64))
    hi_b = int(np.float64(hi).view(np.int64))
    # invariant: total(lo) > budget >= total(hi)
    while hi_b - lo_b > 1:
        mid_b = (lo_b + hi_b) // 2
        mid = float(np.int64(mid_b).view(np.float64))
        if total(mid) > budget:
            lo_b = mid_b
        else:
            hi_b = mid_b
    lo = float(np.int64(lo_b).view(np.float64))
    hi = float(np.int64(hi_b).view(np.float64))
    j_hi = ladder(imp, hi, slopes)
    if int(bits[j_hi].sum()) == budget:
        return to_result(j_hi, hi, 0)
    # tie pass at lambda = lo: demote the tied group in block order
    j_lo = ladder(imp, lo, slopes)
    tied = np.nonzero(j_lo != j_hi)[0]         # ascending block index
    cur = int(bits[j_lo].sum())
    jpos = j_lo.copy()
    T = 0
    for b in tied:
        if cur <= budget:
            break
        cur -= int(bits[jpos[b]] - bits[j_hi[b]])
        jpos[b] = j_hi[b]
        T += 1
    if T == len(tied):
        return to_result(j_hi, hi, 0)
    return to_result(jpos, lo, T)


def decode_rungs(imp: np.ndarray, lam: float, T: int, hull_idx, slopes_from) -> np.ndarray:
    """Decoder side of Algorithm 2: the ladder at lam, the first T blocks at the
    threshold taking the lower rung. ``slopes_from`` = (rates, damage)."""
    rates, damage = slopes_from
    H = list(hull_idx)
    slopes = hull_slopes(H, rates, damage)
    jpos = ladder(imp, lam, slopes)
    if T:
        # blocks exactly at a threshold: promoted at lam but not just above it
        above = ladder(imp, float(np.nextafter(lam, np.inf)), slopes)
        tied = np.nonzero(jpos != above)[0][:T]
        jpos[tied] = above[tied]
    return np.array(H, dtype=np.uint8)[jpos]
