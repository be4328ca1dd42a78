"""Pins for the oracle's rung schedule (sections 3.2-3.4, Algorithms 1-2)."""
import itertools

import numpy as np
import pytest

import synthetic
from oracle import allocation as sch

THREE = ((12, 2), (16, 3), (20, 4))
DAMAGE = (4.0, 1.0, 0.25)


def _bits(rungs):
    return np.array([K + 4 * P + 4 for K, P in rungs])


@pytest.mark.parametrize("name", ["mlp_up", "reduced", "l70b"])
def test_rate_identity(oq, name):
    wl = synthetic.WORKLOADS[name]
    a = synthetic.importance_profile(wl.ncols)
    r = oq.schedule(32, wl.ncols, wl.rungs, wl.damage, wl.target_bpw, a)
    nb = 32 * wl.ncols // 8
    bits = _bits(wl.rungs)[r.rung_of_block].sum()
    assert bits == r.total_bits == r.budget_bits == int(8 * wl.target_bpw * nb)


def test_uniform_single_rung(oq):
    a = synthetic.importance_profile(64)
    r = oq.schedule(8, 64, ((16, 3),), None, 4.0, a)
    assert not r.rung_of_block.any()
    assert r.total_bits == 32 * 64


def test_ladder_monotone(oq):
    a = synthetic.importance_profile(4096)
    r = oq.schedule(4, 4096, THREE, DAMAGE, 4.0, a)
    imp = r.imp
    order = np.argsort(imp, kind="stable")
    assert np.all(np.diff(r.rung_of_block[order].astype(int)) >= 0)


def test_floor(oq):
    a = synthetic.importance_profile(800)
    r = oq.schedule(5, 800, THREE, DAMAGE, 4.0, a, floor_fraction=0.06)
    assert np.sum(r.imp == r.floor_q) >= 0.06 * r.imp.size
    assert r.imp.min() == r.floor_q


def test_tie_pass_splits_group_in_block_order(oq):
    # 3 rows x 4 column groups: blocks of one group share their importance, so
    # a budget between group totals must split a group; the first T blocks (in
    # row-major block order) of the tied group take the lower rung.
    a = synthetic.importance_profile(32)
    nb = 12
    base = 24 * nb
    r = oq.schedule(3, 32, THREE, DAMAGE, (base + 8 * 5) / (8 * nb), a, floor_fraction=0.0)
    assert r.total_bits == base + 40
    assert r.tie_count > 0
    rob = r.rung_of_block.reshape(3, 4)
    # within every column group the rungs are non-decreasing down the rows
    assert np.all(np.diff(rob.astype(int), axis=0) >= 0)
    dec = sch.decode_rungs(r.imp, r.lam, r.tie_count, r.hull, (_bits(THREE), np.array(DAMAGE)))
    assert np.array_equal(dec, r.rung_of_block)


@pytest.mark.parametrize("trial", range(6))
def test_everett_optimality_brute_force(oq, trial):
    # random importances on 2 rows x 4 groups = 8 blocks, 3 rungs: the
    # allocation minimises sum imp_b e(g_b) over every allocation that spends
    # at most as many bits as it does (Everett's theorem, appendix on ties)
    rng = np.random.default_rng(trial)
    a = np.exp(rng.normal(0, 1, 32)).astype(np.float32)
    nb = 8
    target = rng.choice([3.25, 3.5, 3.75, 4.0, 4.5])
    r = oq.schedule(2, 32, THREE, DAMAGE, target, a, floor_fraction=0.0)
    bits = _bits(THREE)
    dmg = np.array(DAMAGE)
    mine = float(np.sum(r.imp * dmg[r.rung_of_block]))
    best = np.inf
    for alloc in itertools.product(range(3), repeat=nb):
        alloc = np.array(alloc)
        if bits[alloc].sum() <= r.total_bits:
            best = min(best, float(np.sum(r.imp * dmg[alloc])))
    assert mine <= best * (1 + 1e-12)
    assert r.total_bits <= r.budget_bits


def test_hull_drops_non_convex_rung(oq):
    rates = np.array([24.0, 28.0, 32.0])
    H = sch.hull(rates, np.array([4.0, 3.5, 1.0]))   # middle point above the chord
    assert H == [0, 2]
    H = sch.hull(rates, np.array([4.0, 1.5, 1.0]))
    assert H == [0, 1, 2]
    # a middle rung on the chord is no vertex of the hull (section 3.4: the
    # ladder runs over the hull's vertices; a collinear rung buys no better
    # damage per bit than mixing its neighbours)
    H = sch.hull(rates, np.array([4.0, 2.5, 1.0]))
    assert H == [0, 2]


def test_decoder_reproduces_allocation(oq):
    wl = synthetic.WORKLOADS["reduced"]
    a = synthetic.importance_profile(wl.ncols)
    r = oq.schedule(16, wl.ncols, wl.rungs, wl.damage, wl.target_bpw, a)
    dec = sch.decode_rungs(r.imp, r.lam, r.tie_count, r.hull, (_bits(THREE), np.array(DAMAGE)))
    assert np.array_equal(dec, r.rung_of_block)
