"""Pins of the stream oracle (oracle/stream.py) against a hand-derived payload,
the rate identity of eq. (rate) and round trips; and of the footprint metrics
of eq. (security_metrics) against hand counts."""
import os

import numpy as np
import pytest

from oracle import stream

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "stream_three_blocks.txt")


def _golden():
    rungs, rob, seed, exp, q, words = [], [], [], [], [], None
    for line in open(GOLDEN):
        t = line.split()
        if not t or t[0].startswith("#"):
            continue
        if t[0] == "rung":
            rungs.append((int(t[1]), int(t[2])))
        elif t[0] == "block":
            rob.append(int(t[1]))
            seed.append(int(t[2], 0))
            exp.append(int(t[3]))
            row = [int(v) for v in t[4:]]
            q.append(row + [0] * (8 - len(row)))
        elif t[0] == "words":
            words = [int(v, 0) for v in t[1:]]
    return rungs, np.array(rob), np.array(seed), np.array(exp), np.array(q), np.array(words, np.uint32)


def test_pack_matches_hand_derived_words():
    rungs, rob, seed, exp, q, words = _golden()
    assert np.array_equal(stream.pack(seed, exp, q, rob, rungs), words)


def test_unpack_hand_derived_words():
    rungs, rob, seed, exp, q, words = _golden()
    s, e, qq = stream.unpack(words, rob, rungs)
    assert np.array_equal(s, seed) and np.array_equal(e, exp) and np.array_equal(qq, q)


def test_unpack_rejects_a_short_stream():
    rungs, rob, seed, exp, q, words = _golden()
    with pytest.raises(ValueError):
        stream.unpack(words[:2], rob, rungs)


@pytest.mark.parametrize("trial", range(4))
def test_rate_identity_and_round_trip(trial):
    rng = np.random.default_rng(trial)
    rungs = [(8, 1), (12, 2), (16, 3), (20, 4), (24, 6)]
    nb = 200
    rob = rng.integers(0, len(rungs), nb)
    seed = np.array([int(rng.integers(1, 1 << rungs[r][0])) for r in rob])
    exp = rng.integers(0, 16, nb)
    q = np.zeros((nb, 8), dtype=np.int64)
    for b in range(nb):
        q[b, :rungs[rob[b]][1]] = rng.integers(-8, 8, rungs[rob[b]][1])
    words = stream.pack(seed, exp, q, rob, rungs)
    total = sum(K + 4 * P + 4 for K, P in (rungs[r] for r in rob))
    assert len(words) == (total + 31) // 32
    if total % 32:
        assert int(words[-1]) >> (total % 32) == 0        # zero padding
    s, e, qq = stream.unpack(words, rob, rungs)
    assert np.array_equal(s, seed) and np.array_equal(e, exp) and np.array_equal(qq, q)


def test_one_flipped_payload_bit_changes_one_block():
    rungs, rob, seed, exp, q, words = _golden()
    for n in range(65):
        w = words.copy()
        w[n // 32] ^= np.uint32(1 << (n % 32))
        s, e, qq = stream.unpack(w, rob, rungs)
        changed = (s != seed) | (e != exp) | np.any(qq != q, axis=1)
        assert changed.sum() == 1


def test_footprint_hand_counts():
    a = np.array([[1.0, 2.0], [3.0, 4.0]])
    b = a.copy()
    assert stream.footprint(a, b) == (0, 0.0, 0.0)
    b[0, 1] = 5.0                                   # one weight, |delta| = 3
    n, p, eta = stream.footprint(a, b)
    assert (n, p) == (1, 0.25) and abs(eta - 3.0 / np.sqrt(30.0)) < 1e-15
