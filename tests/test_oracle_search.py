"""Pins for the oracle's exhaustive seed search and decoder (section 3.1: the
encoder tries every nonzero seed and keeps the code of least quantised error;
Algorithm 2: w_hat = U(s) t_hat)."""
import numpy as np
import pytest

import synthetic


def _planted(oq, n, K, P, key):
    seeds, es, qs = synthetic.random_codes(n, K, P, key=key)
    w_hat, acc = oq.decompress(seeds, es, qs, K, P)
    return seeds, es, qs, w_hat, acc


@pytest.mark.parametrize("K,P", [(8, 3), (10, 2), (12, 3)])
def test_planted_blocks_recovered_exactly(oq, K, P):
    seeds, es, qs, w, acc = _planted(oq, 16, K, P, key=K + P)
    # planted weights are exact fp32 values acc * 2^-(K-1+e)
    assert np.array_equal(w.astype(np.float64), np.ldexp(acc.astype(np.float64),
                                                         -(K - 1 + es.astype(np.int64))[:, None]))
    r = oq.search(w, K, P)
    assert np.array_equal(r.seed, seeds)
    assert np.array_equal(r.e, es.astype(np.int32))
    assert np.array_equal(r.q, qs.astype(np.int32))
    assert np.all(r.err == 0.0)


@pytest.mark.parametrize("K,P", [(8, 3), (10, 2), (10, 4)])
def test_c_and_numpy_oracles_agree(oq, K, P):
    w = synthetic.weights(4, 32, 0.02, key=K * 7 + P, outlier_frac=0.02)
    a = oq.search(w, K, P)
    b = oq.search_numpy(w, K, P)
    assert np.array_equal(a.seed, b.seed)
    assert np.array_equal(a.e, b.e)
    assert np.array_equal(a.q, b.q)
    assert np.array_equal(a.err, b.err)


def test_search_is_minimum_over_all_seeds(oq):
    K, P = 8, 3
    w = synthetic.weights(2, 16, 0.02, key=5).reshape(-1, 8)
    r = oq.search(w, K, P)
    for b in range(len(w)):
        errs = []
        for s in range(1, 1 << K):
            t = oq.ls_solve(oq.basis(K, P, s), w[b].astype(np.float64))
            e, q = oq.quantize(t)
            errs.append(oq.code_error(w[b], K, P, s, e, q))
        errs = np.array(errs)
        assert r.err[b] == errs.min()
        assert r.seed[b] == int(np.argmin(errs)) + 1


def test_error_is_exact_and_bounded_below_by_ls_residual(oq):
    K, P = 12, 3
    w = synthetic.weights(1, 64, 0.02, key=6).reshape(-1, 8)
    r = oq.search(w, K, P)
    for b in range(len(w)):
        U = oq.basis(K, P, int(r.seed[b]))
        t_hat = np.ldexp(r.q[b].astype(np.float64), -int(r.e[b]))
        ref = np.sum((w[b].astype(np.float64) - U @ t_hat) ** 2)
        assert r.err[b] == pytest.approx(ref, rel=1e-12)
        t = oq.ls_solve(U, w[b].astype(np.float64))
        rls = np.sum((w[b] - U @ t) ** 2)
        assert r.err[b] >= rls * (1 - 1e-12)


def test_zero_block(oq):
    r = oq.search(np.zeros((1, 8), np.float32), 10, 3)
    assert r.seed[0] == 1 and r.e[0] == 15 and not r.q.any() and r.err[0] == 0.0


def test_power_of_two_scaling(oq):
    # doubling w doubles every t*, so the quantiser picks e - 1 with the same
    # mantissas and every error is multiplied by exactly 4
    K, P = 10, 3
    w = synthetic.weights(1, 64, 0.02, key=7).reshape(-1, 8)
    a = oq.search(w, K, P)
    b = oq.search(w * 2, K, P)
    assert np.array_equal(a.seed, b.seed)
    assert np.array_equal(a.e - 1, b.e)
    assert np.array_equal(a.q, b.q)
    assert np.array_equal(a.err * 4, b.err)


def test_decompress_matches_basis_product(oq):
    K, P = 16, 3
    seeds, es, qs = synthetic.random_codes(50, K, P, key=9, canonical=False)
    w_hat, acc = oq.decompress(seeds, es, qs, K, P)
    for i in range(50):
        Ui = oq.basis_int(K, P, int(seeds[i]))
        ref = Ui @ qs[i].astype(np.int64)
        assert np.array_equal(acc[i], ref)
        assert np.array_equal(w_hat[i], np.ldexp(ref.astype(np.float64), -(K - 1 + int(es[i]))).astype(np.float32))


def test_seed_fault_confined_to_block(oq):
    # a corrupted seed changes only its own block's weights (section 3.6)
    K, P = 16, 3
    seeds, es, qs = synthetic.random_codes(64, K, P, key=10)
    clean, _ = oq.decompress(seeds, es, qs, K, P)
    bad = seeds.copy()
    bad[17] ^= np.uint32(1 << 5)
    dirty, _ = oq.decompress(bad, es, qs, K, P)
    changed = np.nonzero((clean != dirty).any(axis=1))[0]
    assert list(changed) == [17]
    assert (clean[17] != dirty[17]).sum() <= 8
