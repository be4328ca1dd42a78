"""Host logic of the rung-grid study (no GPU): rates against the paper's table,
and the ratio summary against closed forms."""
import os

import numpy as np
import pytest

from paper_2609_38477_amd import grid

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [l.split() for l in f if l.strip() and not l.startswith("#")]


def test_rates_match_table_grids():
    for K, P, rate in _rows("rung_grid_rates.txt"):
        assert grid.rate_bpw(int(K), int(P)) == float(rate)


def test_paper_grid_is_the_full_grid():
    assert len(grid.PAPER_GRID) == 45
    assert set(grid.PAPER_GRID) == {(S, k) for S in range(8, 17) for k in range(2, 7)}
    assert set(grid.RUNGSHAPE_RUNGS) | {grid.REFERENCE_RUNG} <= set(grid.PAPER_GRID)
    table = [tuple(int(v) for v in r[:2]) for r in _rows("rungshape_paper.txt")]
    assert tuple(table) == grid.RUNGSHAPE_RUNGS


def test_rungshape_constant_ratio():
    # every block's error at g is exactly c times its error at the reference:
    # median = quantiles = c and the log-ratio has zero spread
    rng = np.random.default_rng(0)
    e0 = rng.uniform(0.5, 2.0, 1000)
    err = {grid.REFERENCE_RUNG: e0}
    for i, r in enumerate(grid.RUNGSHAPE_RUNGS):
        err[r] = e0 * 2.0 ** (i - 2)
    for i, row in enumerate(grid.rungshape(err)):
        c = 2.0 ** (i - 2)
        assert row["blocks"] == 1000
        for k in ("median", "q10", "q90"):
            assert abs(row[k] - c) <= 1e-12 * c
        assert row["sd_log"] < 1e-12


def test_rungshape_lognormal_ratio_and_zero_blocks():
    # ratios exp(N(mu, s^2)): median -> e^mu, quantiles e^(mu +- 1.2816 s), sd of
    # log -> s; blocks with a zero error at either rung are left out
    rng = np.random.default_rng(1)
    n, mu, s = 200_000, np.log(1.5), 0.5
    e0 = rng.uniform(0.1, 1.0, n)
    e1 = e0 * np.exp(rng.normal(mu, s, n))
    e0[:10] = 0.0
    e1[10:20] = 0.0
    rows = grid.rungshape({(16, 3): e0, (14, 3): e1}, rungs=((14, 3),), ref=(16, 3))
    r = rows[0]
    assert r["blocks"] == n - 20
    assert abs(r["median"] / 1.5 - 1) < 0.01
    assert abs(r["q10"] / (1.5 * np.exp(-1.2815516 * s)) - 1) < 0.01
    assert abs(r["q90"] / (1.5 * np.exp(1.2815516 * s)) - 1) < 0.01
    assert abs(r["sd_log"] - s) < 0.005


def test_parse_rungs_names_and_lists():
    assert grid.parse_rungs("paper") == grid.PAPER_GRID
    assert set(grid.parse_rungs("rungshape")) == set(grid.RUNGSHAPE_RUNGS) | {grid.REFERENCE_RUNG}
    assert grid.parse_rungs("16,6;16,5;12,2") == ((16, 6), (16, 5), (12, 2))
    for bad in ("", "16", "16,6;16,6", "16,6,1", "a,b"):
        with pytest.raises(ValueError):
            grid.parse_rungs(bad)
