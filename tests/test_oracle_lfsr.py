"""Pins for the oracle's LFSR basis (section 3.1, eq. (codec))."""
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "lfsr_k8_seed1.txt")


@pytest.mark.parametrize("K", list(range(8, 25)))
def test_maximal_length(oq, K):
    # maximal length (section 3.1): the period is 2^K - 1
    assert oq.period(K) == (1 << K) - 1
    m = oq.lfsr_mask(K)
    assert (m >> (K - 1)) == 1, "mask must keep the state K bits wide"


@pytest.mark.parametrize("K", [8, 11, 12, 16])
def test_visits_every_nonzero_state_once(oq, K):
    n = (1 << K) - 1
    u = oq.states(K, 1, n)
    x = u + (1 << (K - 1))
    assert x.min() == 1 and x.max() == n
    assert np.unique(x).size == n
    # centred states over a period sum to exactly zero, all in [-2^(K-1), 2^(K-1))
    assert int(u.sum()) == 0
    assert u.min() >= -(1 << (K - 1)) and u.max() < (1 << (K - 1))


def test_golden_k8_seed1(oq):
    rows = [l.split() for l in open(GOLDEN) if l.strip() and not l.startswith("#")]
    d = {r[0]: r[1:] for r in rows}
    K, seed = int(d["K"][0]), int(d["seed"][0])
    want = np.array([int(v) for v in d["u"]])
    assert np.array_equal(oq.states(K, seed, len(want)), want)
    U = oq.basis_int(K, 2, seed)
    assert np.array_equal(U[:, 0], want[:8])
    assert np.array_equal(U[:2, 1], want[8:10])


@pytest.mark.parametrize("K", [9, 16, 20])
def test_started_at_state_s(oq, K):
    # the basis of the successor seed is the same state sequence advanced by one
    rng = np.random.default_rng(K)
    for s in rng.integers(1, 1 << K, size=20):
        a = oq.states(K, int(s), 25)
        nxt = int(a[1]) + (1 << (K - 1))
        b = oq.states(K, nxt, 24)
        assert np.array_equal(a[1:], b)
        assert int(a[0]) + (1 << (K - 1)) == int(s)


@pytest.mark.parametrize("K,P", [(8, 3), (12, 2), (12, 3)])
def test_vectorised_states_match(oq, K, P):
    allU = oq.basis_int_all(K, P)
    for s in [1, 2, 77, (1 << K) - 1]:
        assert np.array_equal(allU[s - 1], oq.basis_int(K, P, s))
    U = oq.basis(K, P, 5)
    assert U.min() >= -1.0 and U.max() < 1.0


def test_bad_width_rejected(oq):
    with pytest.raises(ValueError):
        oq.states(7, 1, 8)
    with pytest.raises(ValueError):
        oq.states(8, 0, 8)
