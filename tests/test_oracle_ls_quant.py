"""Pins for the oracle's least squares and shared-exponent quantiser
(section 3.1: least-squares coefficients, m-bit mantissas under one e-bit
exponent, m = e = 4)."""
import numpy as np
import pytest

import synthetic


def test_ls_p1_closed_form(oq):
    rng = np.random.default_rng(1)
    for s in rng.integers(1, 4096, size=20):
        U = oq.basis(12, 1, int(s))
        w = rng.normal(0, 0.02, 8)
        u = U[:, 0]
        t = oq.ls_solve(U, w)
        assert t[0] == pytest.approx(u @ w / (u @ u), rel=1e-13)


def test_ls_p2_cramer(oq):
    rng = np.random.default_rng(2)
    for s in rng.integers(1, 4096, size=20):
        U = oq.basis(12, 2, int(s))
        w = rng.normal(0, 0.02, 8)
        a, b = U[:, 0], U[:, 1]
        g11, g12, g22 = a @ a, a @ b, b @ b
        r1, r2 = a @ w, b @ w
        det = g11 * g22 - g12 * g12
        t_ref = np.array([(r1 * g22 - g12 * r2) / det, (g11 * r2 - g12 * r1) / det])
        assert np.allclose(oq.ls_solve(U, w), t_ref, rtol=1e-10, atol=1e-14)


@pytest.mark.parametrize("K,P", [(12, 3), (16, 3), (20, 4)])
def test_ls_residual_orthogonal_and_minimal(oq, K, P):
    rng = np.random.default_rng(K * 10 + P)
    for s in rng.integers(1, 1 << K, size=10):
        U = oq.basis(K, P, int(s))
        w = rng.normal(0, 0.02, 8)
        t = oq.ls_solve(U, w)
        r = w - U @ t
        assert np.abs(U.T @ r).max() < 1e-15
        base = r @ r
        for _ in range(20):
            d = rng.normal(0, 1e-3, P)
            rr = w - U @ (t + d)
            assert rr @ rr >= base


def test_ls_rank_deficient_min_norm(oq):
    # K = 11, P = 4, seed 0xFE: the four columns are linearly dependent
    Ui = oq.basis_int(11, 4, 0xFE)
    U = Ui.astype(np.float64) * 2.0 ** -10
    assert oq.rank_of(U) == 3
    _, sv, vt = np.linalg.svd(U)
    v = vt[-1]
    assert np.abs(U @ v).max() < 1e-12
    rng = np.random.default_rng(3)
    w = rng.normal(0, 0.02, 8)
    t = oq.ls_solve(U, w)
    # minimum norm: t has no component along the null space, residual orthogonal
    assert abs(t @ v) < 1e-12 * np.linalg.norm(t)
    assert np.abs(U.T @ (w - U @ t)).max() < 1e-14


def test_pinv_stack_matches_single(oq):
    A = oq.pinv_stack(10, 3)
    for s in [1, 100, 1023]:
        assert np.allclose(A[s - 1], np.linalg.pinv(oq.basis(10, 3, s)), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("t,e,q", [
    ([0.0, 0.0, 0.0], 15, [0, 0, 0]),            # zero block: finest exponent
    ([7.5], 0, [7]),                              # rne(7.5) = 8 does not fit: clamp at e = 0
    ([7.25], 0, [7]),
    ([-8.5], 0, [-8]),                            # rne(-8.5) = -8 fits
    ([-8.5000001], 0, [-8]),                      # does not fit at any e: clamp
    ([3.75], 0, [4]),                             # e = 1 gives rne(7.5) = 8
    ([3.7], 1, [7]),
    ([6.5, 7.0], 0, [6, 7]),                      # half to even
    ([5.5, 7.0], 0, [6, 7]),
    ([-6.5, 7.0], 0, [-6, 7]),
    ([7 * 2.0 ** -14], 14, [7]),
    ([1e-9], 15, [0]),
    ([-4.25 * 2.0 ** -9, 3.0 * 2.0 ** -9], 10, [-8, 6]),  # at e = 10: rne(-8.5) = -8 fits
    ([100.0, -3.0], 0, [7, -3]),
])
def test_quantiser_boundary_table(oq, t, e, q):
    got_e, got_q = oq.quantize(t)
    assert got_e == e and list(got_q) == q
    e2, q2 = oq.quantize_numpy(np.array(t))
    assert int(e2) == e and list(q2) == q


def test_quantiser_canonical_roundtrip(oq):
    for P in (2, 3, 4, 6):
        seeds, es, qs = synthetic.random_codes(200, 12, P, key=P, exps=tuple(range(16)))
        for e, q in zip(es, qs):
            t = np.ldexp(q.astype(np.float64), -int(e))
            ge, gq = oq.quantize(t)
            assert ge == int(e) and np.array_equal(gq, q)


def test_quantiser_c_matches_numpy(oq):
    rng = np.random.default_rng(4)
    t = rng.normal(0, 1, (2000, 3)) * np.exp(rng.uniform(-12, 3, (2000, 1)))
    e2, q2 = oq.quantize_numpy(t)
    for i in range(len(t)):
        e, q = oq.quantize(t[i])
        assert e == e2[i] and np.array_equal(q, q2[i])


def test_closed_form_exponent_equals_the_exponent_search(oq):
    # The kernels pick the shared exponent in closed form from frexp of every
    # coefficient; the definition (R6) searches e from 15 down. Check the two
    # agree at every boundary the closed form uses (mantissas 7.5 and -8.5
    # times 2^-e, one ulp either side) and on random coefficients.
    import math
    import numpy as np

    def closed(t):
        e = 15
        for v in t:
            if v != 0.0:
                f, E = math.frexp(abs(v))
                lim = (3 - E if f < 0.9375 else 2 - E) if v > 0 else (4 - E if f <= 0.53125 else 3 - E)
                e = min(e, lim)
        return max(e, 0)

    vals = []
    for e in range(-3, 18):
        for base in (7.5, -8.5, 7.0, -8.0, 3.75, -4.25):
            x = math.ldexp(base, -e)
            vals += [x, np.nextafter(x, np.inf), np.nextafter(x, -np.inf)]
    rng = np.random.default_rng(0)
    cases = [np.array([v, 0.0, 0.0]) for v in vals]
    cases += [rng.normal(0, 10.0 ** rng.uniform(-4, 1), 3) for _ in range(3000)]
    cases += [np.zeros(3)]
    for t in cases:
        e_ref, _ = oq.quantize(np.asarray(t, dtype=np.float64))
        assert closed(t) == e_ref, t
