"""Pins of the oracle's overlap, cost and argmin (snapshot scoring)."""
from fractions import Fraction

import numpy as np
import pytest

import brute


def _instance(rng, B, W, universe, max_len):
    chains, off = [], [0]
    for _ in range(B):
        L = int(rng.integers(0, max_len + 1))
        chains.extend(int(x) for x in rng.integers(1, universe, size=L))
        off.append(len(chains))
    keys, koff = [], [0]
    sets = []
    for _ in range(W):
        k = np.unique(rng.integers(1, universe, size=int(rng.integers(0, universe))))
        keys.extend(int(x) for x in k)
        koff.append(len(keys))
        sets.append(set(int(x) for x in k))
    active = rng.integers(0, 40, size=W).astype(np.int32)
    return (np.array(chains, np.uint64), np.array(off, np.int64), np.array(keys, np.uint64),
            np.array(koff, np.int64), active, sets)


@pytest.mark.parametrize("seed", range(6))
def test_score_batch_matches_bruteforce(orc, seed):
    rng = np.random.default_rng(seed)
    W = int(rng.integers(1, 7))
    chains, off, keys, koff, active, sets = _instance(rng, 40, W, 12, 10)
    w = (1.0, 0.5, 4.0) if seed % 2 == 0 else (0.75, 1.25, 2.5)
    cap = int(rng.integers(1, 30))
    ov, co, am = orc.score_batch(chains, off, keys, koff, active, *w, cap=cap)
    for i in range(len(off) - 1):
        ch = chains[off[i]:off[i + 1]]
        P = len(ch)
        costs = []
        for j in range(W):
            o = brute.overlap_set(ch, sets[j])
            assert ov[i, j] == o
            c = brute.cost_f32(*w, cap, P, o, int(active[j]))
            assert co[i, j].view(np.uint32) == np.float32(c).view(np.uint32)
            costs.append(c)
        best = 0
        for j in range(1, W):
            if costs[j] < costs[best]:
                best = j
        assert am[i] == best


def test_overlap_is_first_miss_not_count(orc):
    # blocks 2 and 3 are cached but block 1 is not: the cached prefix has length 1
    chains = np.array([5, 6, 7, 8], np.uint64)
    ov, _, _ = orc.score_batch(chains, np.array([0, 4]), np.array([5, 7, 8], np.uint64),
                               np.array([0, 3]), np.array([0], np.int32))
    assert ov[0, 0] == 1
    ov, _, _ = orc.score_batch(chains, np.array([0, 4]), np.array([6, 7, 8], np.uint64),
                               np.array([0, 3]), np.array([0], np.int32))
    assert ov[0, 0] == 0
    ov, _, _ = orc.score_batch(chains, np.array([0, 4]), np.array([5, 6, 7, 8], np.uint64),
                               np.array([0, 4]), np.array([0], np.int32))
    assert ov[0, 0] == 4


def _exact_cost(w_ov, w_act, w_sat, cap, P, o, A):
    r = Fraction(A + P, cap)
    x = max(r - 1, Fraction(0))
    return Fraction(w_ov) * (P - o) + Fraction(w_act) * A + Fraction(w_sat) * x * x


def test_cost_closed_forms(orc):
    rng = np.random.default_rng(11)
    for _ in range(500):
        cap = int(2 ** rng.integers(0, 16))
        P = int(rng.integers(0, 600))
        o = int(rng.integers(0, P + 1))
        A = int(rng.integers(0, 70000))
        c = float(orc.route_cost(1.0, 0.5, 4.0, cap, P, o, A))
        ex = _exact_cost(1.0, 0.5, 4.0, cap, P, o, A)
        assert c >= 0.0
        # t1, t2, r, x and t1+t2 are exact for dyadic weights and a power-of-two cap;
        # only x*x and the last addition may round (each by at most half an ulp)
        assert abs(Fraction(c) - ex) <= ex * Fraction(1, 2 ** 22) + Fraction(1, 2 ** 60)
        no_sat = float(orc.route_cost(1.0, 0.5, 0.0, cap, P, o, A))
        assert (c > no_sat) == (A + P > cap)
    # full cache hit on an idle, uncongested worker costs nothing
    assert float(orc.route_cost(1.0, 0.5, 4.0, 512, 32, 32, 0)) == 0.0
    # each weight scales its own term only
    assert float(orc.route_cost(2.0, 0.0, 0.0, 8, 10, 3, 100)) == 14.0
    assert float(orc.route_cost(0.0, 0.25, 0.0, 8, 10, 3, 100)) == 25.0
    assert float(orc.route_cost(0.0, 0.0, 1.0, 8, 4, 0, 12)) == 1.0     # x = 16/8 - 1


def test_argmin_special_cases(orc):
    rng = np.random.default_rng(5)
    chains, off, keys, koff, active, _ = _instance(rng, 30, 5, 10, 8)
    # one worker takes everything
    _, _, am = orc.score_batch(chains, off, keys[:koff[1]], koff[:2], active[:1])
    assert np.all(am == 0)
    # only load matters: least active blocks, lowest index among equals
    act = np.array([7, 3, 9, 3, 4], np.int32)
    _, _, am = orc.score_batch(chains, off, keys, koff, act, 0.0, 1.0, 0.0, cap=1)
    assert np.all(am == 1)
    # only overlap matters: longest cached prefix, lowest index among equals
    ov, _, am = orc.score_batch(chains, off, keys, koff, active, 1.0, 0.0, 0.0, cap=1)
    for i in range(len(off) - 1):
        assert am[i] == int(np.argmax(ov[i]))   # argmax returns the first maximum
    # empty caches and equal loads: worker 0
    _, _, am = orc.score_batch(chains, off, np.zeros(0, np.uint64), np.zeros(6, np.int64),
                               np.full(5, 4, np.int32))
    assert np.all(am == 0)


def test_empty_batch_and_empty_chains(orc):
    ov, co, am = orc.score_batch(np.zeros(0, np.uint64), np.array([0]), np.array([3], np.uint64),
                                 np.array([0, 1]), np.array([0], np.int32))
    assert ov.shape == (0, 1) and am.shape == (0,)
    ov, co, am = orc.score_batch(np.zeros(0, np.uint64), np.array([0, 0, 0]),
                                 np.array([3], np.uint64), np.array([0, 1]),
                                 np.array([0], np.int32))
    assert np.all(ov == 0) and np.all(co == 0.0)
