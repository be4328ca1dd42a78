"""Host parts of the importance front end in the library (no GPU): the
Gauss-Hermite rule, the channel sort and the outlier ranking against the oracle
and closed forms."""
import math
import os

import numpy as np
import pytest

from oracle import importance as oimp


@pytest.fixture(scope="module")
def sq():
    import paper_2609_38477_amd as sq
    if not os.path.exists(sq.LIB_PATH):
        from paper_2609_38477_amd import build
        build.build()
    return sq


@pytest.mark.parametrize("n", [1, 2, 3, 16, 64, 128, 255])
def test_gauss_hermite_matches_numpy_and_moments(sq, n):
    x, w = sq.seedq_gauss_hermite(n)
    with np.errstate(all="ignore"):
        xr, wr = np.polynomial.hermite.hermgauss(n)
    assert np.all(np.diff(x) > 0)
    assert np.allclose(x, xr, rtol=0, atol=1e-12 * max(1.0, np.abs(xr).max()))
    big = wr > 1e-280
    assert np.allclose(w[big], wr[big], rtol=1e-10, atol=0)
    # exact for polynomials of degree < 2n: sum w x^k = Gamma((k+1)/2) for even k
    for k in range(0, min(2 * n - 1, 40), 2):
        ref = math.gamma((k + 1) / 2)
        assert abs(np.sum(w * x ** k) - ref) <= 1e-11 * ref


def test_channel_order_matches_oracle(sq):
    rng = np.random.default_rng(4)
    a = np.round(rng.exponential(1.0, 5000) * 8).astype(np.float32)      # many ties
    assert np.array_equal(sq.seedq_channel_order(a), oimp.channel_order(a))


def test_select_outliers_matches_oracle(sq):
    rng = np.random.default_rng(1)
    W0, W1 = rng.normal(0, 1, (64, 400)), rng.normal(0, 1, (64, 400))
    W0[5, 7], W1[9, 3] = 1e6, 1e4
    a0, a1 = np.ones(400), np.ones(400)
    a1[30], a0[7] = 1e5, 1e4
    stats = [oimp.column_stats(W) for W in (W0, W1)]
    got = sq.seedq_select_outliers([s[0] for s in stats], [s[1] for s in stats], [a0, a1])
    assert got == oimp.outlier_columns([W0, W1], [a0, a1]) == [(0, 7), (1, 30), (1, 3)]
    # many candidates: the 32-per-rule cap and the keep count
    W = rng.normal(0, 1, (32, 100))
    for j in range(50):
        W[:, j] = 1.0
        W[j % 32, j] = 1e5 * (1 + j)
    st = oimp.column_stats(W)
    a = np.ones(100)
    assert sq.seedq_select_outliers([st[0]], [st[1]], [a], keep=4) == oimp.outlier_columns([W], [a])
    assert sq.seedq_select_outliers([st[0]], [st[1]], [a], keep=0) == []


def test_channel_order_rejects_non_finite_importance():
    import paper_2609_38477_amd as sq
    for bad in (np.nan, np.inf, -np.inf):
        a = np.array([1.0, bad, 0.5], dtype=np.float32)
        with pytest.raises(sq.SeedqError) as e:
            sq.seedq_channel_order(a)
        assert e.value.code == -1
