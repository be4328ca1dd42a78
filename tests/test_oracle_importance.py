"""Pins of the importance front-end oracle (oracle/importance.py) against
closed forms, independent quadrature and hand-made cases."""
import numpy as np
import pytest
from scipy import integrate

from oracle import importance as imp


@pytest.mark.parametrize("var,tol", [(1e-6, 1e-12), (0.01, 1e-12), (0.3, 1e-12), (1.0, 1e-12),
                                     (4.0, 1e-12), (25.0, 5e-6)])
def test_e_silu_sq_matches_adaptive_quadrature(var, tol):
    # 128-node Gauss-Hermite against an adaptive integral; the tolerance is the
    # quadrature's own error, which grows with the variance
    # E[silu(g)^2], g ~ N(0, var), by scipy's adaptive integral of the density
    s = np.sqrt(var)
    f = lambda x: (x / (1 + np.exp(-x))) ** 2 * np.exp(-x * x / (2 * var)) / (s * np.sqrt(2 * np.pi))
    ref, _ = integrate.quad(f, -40 * s, 40 * s, epsabs=0, epsrel=1e-13, limit=400)
    assert abs(imp.e_silu_sq(var) - ref) <= tol * ref


def test_e_silu_sq_small_variance_limit():
    # silu(x) = x/2 + x^2/4 + O(x^4): E[silu^2] = var/4 + 3 var^2/16 + O(var^3)
    v = 1e-4
    assert abs(imp.e_silu_sq(v) - (v / 4 + 3 * v * v / 16)) < 1e-11


def test_squared_matvec_hand_example():
    W = np.array([[1.0, -2.0, 0.0], [3.0, 0.5, -1.0]])
    a = np.array([1.0, 2.0, 4.0])
    assert np.array_equal(imp.sq_matvec(W, a), [1 + 8 + 0, 9 + 0.5 + 4])
    assert np.array_equal(imp.sq_matvec_t(W, np.array([1.0, 10.0])), [91.0, 6.5, 10.0])


def test_propagate_o_repeats_kv_heads():
    # 2 kv heads of dim 2, 4 query heads: channels [h0, h0, h1, h1] head-major
    W_v = np.diag([1.0, 2.0, 3.0, 4.0])
    a = np.ones(4)
    assert np.array_equal(imp.propagate_o(W_v, a, 4, 2), [1, 4, 1, 4, 9, 16, 9, 16])


def test_propagate_down_is_the_product_of_its_two_branches():
    rng = np.random.default_rng(0)
    Wg, Wu = rng.normal(0, 0.1, (5, 3)), rng.normal(0, 0.1, (5, 3))
    a = np.array([1.0, 0.5, 2.0])
    got = imp.propagate_down(Wg, Wu, a)
    var = (Wg ** 2) @ a
    assert np.allclose(got, imp.e_silu_sq(var) * ((Wu ** 2) @ a), rtol=1e-15, atol=0)


def test_rho_from_isotropic_logit_gradient():
    W_lm = np.array([[1.0, 2.0], [3.0, -1.0], [0.0, 2.0]])   # vocab 3, hidden 2
    assert np.array_equal(imp.rho_from_head(W_lm), [10.0, 9.0])


def test_channel_order_is_stable():
    assert imp.channel_order([3.0, 1.0, 3.0, 0.5, 1.0]).tolist() == [3, 1, 4, 0, 2]


def test_column_stats_and_dynamic_range():
    W = np.array([[0.0, 1.0, -4.0, 0.0],
                  [0.0, -3.0, 1.0, 0.0],
                  [0.0, 2.0, 2.0, 5.0],
                  [0.0, 4.0, 1.0, 0.0]])
    mx, med = imp.column_stats(W)
    assert mx.tolist() == [0, 4, 4, 5] and med.tolist() == [0, 2.5, 1.5, 0]
    dr = imp.dynamic_range(W)
    assert dr[0] == 0 and dr[3] == 2.0 ** 24
    assert abs(dr[1] - 4 / (2.5 + 4 * 2.0 ** -24)) < 1e-15


def test_outlier_ranking_by_better_position():
    rng = np.random.default_rng(1)
    W0 = rng.normal(0, 1, (64, 400))
    W1 = rng.normal(0, 1, (64, 400))
    # dynamic-range candidates: tensor 0 column 7 (huge), tensor 1 column 3 (large)
    W0[5, 7] = 1e6
    W1[9, 3] = 1e4
    a0 = np.ones(400)
    a1 = np.ones(400)
    # activation candidates (a_j >= 100 x the tensor mean): tensor 1 column 30
    # (largest a), tensor 0 column 7 (second)
    a1[30] = 1e5
    a0[7] = 1e4
    got = imp.outlier_columns([W0, W1], [a0, a1])
    # positions: (0,7): dr 0, act 1 -> 0; (1,30): act 0 -> 0; (1,3): dr 1 -> 1
    assert got == [(0, 7), (1, 30), (1, 3)]


def test_outliers_keep_four_and_at_most_32_per_rule():
    rng = np.random.default_rng(2)
    W = rng.normal(0, 1, (32, 100))
    for j in range(50):
        W[:, j] = 1.0                          # equal medians, so the spike orders the ratio
        W[j % 32, j] = 1e5 * (1 + j)          # 50 spike columns, larger for larger j
    got = imp.outlier_columns([W], [np.ones(100)])
    assert got == [(0, 49), (0, 48), (0, 47), (0, 46)]
