"""Pins of the oracle's PoA-hat: frozen matrix, Hungarian OPT, ratio."""
from fractions import Fraction

import numpy as np
import pytest
from scipy.optimize import linear_sum_assignment

import brute
from paper_2606_17081_amd.workload import POA_PARAMS

P_ = POA_PARAMS


def _window(rng, m, W, skew=0.0):
    p = np.ones(W) / W
    if skew:
        p = np.exp(-skew * np.arange(W))
        p /= p.sum()
    worker = rng.choice(W, size=m, p=p).astype(np.int32)
    blocks = rng.integers(1, 40, size=m).astype(np.int32)
    overlap = (rng.random((m, W)) * (blocks[:, None] + 1)).astype(np.int32)
    overlap = np.minimum(overlap, blocks[:, None])
    return worker, overlap, blocks


def test_matrix_closed_form(orc):
    rng = np.random.default_rng(0)
    worker, overlap, blocks = _window(rng, 30, 5, skew=0.5)
    c, n = orc.poa_matrix(worker, overlap, blocks, 5, **P_)
    assert n.tolist() == np.bincount(worker, minlength=5).tolist()
    for i in range(30):
        for j in range(5):
            gap = max(P_["C_cap"] - int(n[j]), 1)
            ex = (Fraction(P_["a"]) * int(n[j]) + Fraction(P_["b"]) + Fraction(P_["d"]) / gap ** 2
                  - Fraction(P_["w_c"]) * Fraction(int(overlap[i, j]), int(blocks[i])))
            assert abs(Fraction(float(c[i, j])) - ex) <= abs(ex) * Fraction(1, 2 ** 20)
    # the pole is guarded: a worker at or past C_j uses a gap of one
    worker = np.zeros(70, np.int32)
    c, n = orc.poa_matrix(worker, np.zeros((70, 2), np.int32), np.ones(70, np.int32), 2, **P_)
    assert abs(float(c[0, 0]) - (0.005 * 70 + 0.02 + 0.01)) < 1e-6


@pytest.mark.parametrize("seed", range(25))
def test_opt_matches_bruteforce(orc, seed):
    rng = np.random.default_rng(seed)
    W = int(rng.integers(1, 5))
    m = int(rng.integers(1, 9 if W <= 2 else 8))
    worker, overlap, blocks = _window(rng, m, W, skew=float(rng.choice([0.0, 1.0])))
    c, _ = orc.poa_matrix(worker, overlap, blocks, W, **P_)
    K = (m + W - 1) // W
    s, o, ow = orc.poa_window(worker, overlap, blocks, W, **P_)
    assert o == pytest.approx(brute.opt_bruteforce(c, K), rel=1e-12, abs=1e-15)
    assert s == pytest.approx(sum(float(c[i, worker[i]]) for i in range(m)), rel=1e-15)
    assert np.bincount(ow, minlength=W).max() <= K
    assert o == pytest.approx(sum(float(c[i, ow[i]]) for i in range(m)), rel=1e-12)


@pytest.mark.parametrize("m,W", [(16, 3), (64, 6), (100, 7), (96, 16), (40, 40)])
def test_opt_matches_scipy_assignment(orc, m, W):
    rng = np.random.default_rng(m * 100 + W)
    worker, overlap, blocks = _window(rng, m, W, skew=0.3)
    c, _ = orc.poa_matrix(worker, overlap, blocks, W, **P_)
    K = (m + W - 1) // W
    rep = np.repeat(c.astype(np.float64), K, axis=1)          # column j*K+r replicates worker j
    r, col = linear_sum_assignment(rep)
    ref = float(rep[r, col].sum())
    _, o, _ = orc.poa_window(worker, overlap, blocks, W, **P_)
    assert o == pytest.approx(ref, rel=1e-12)


def test_poa_is_one_without_congestion_or_cache_terms(orc):
    rng = np.random.default_rng(4)
    worker, overlap, blocks = _window(rng, 50, 4, skew=1.0)
    s, o, _ = orc.poa_window(worker, overlap, blocks, 4, a=0.0, b=0.02, d=0.0, beta=2, C_cap=64,
                             w_c=0.0)
    assert s == o


def test_opt_closed_form_without_cache_term(orc):
    # w_c = 0: every row costs base_j on worker j, so OPT fills the cheapest workers first
    rng = np.random.default_rng(9)
    for _ in range(10):
        W = int(rng.integers(2, 7))
        m = int(rng.integers(1, 60))
        worker, overlap, blocks = _window(rng, m, W, skew=1.5)
        c, n = orc.poa_matrix(worker, overlap, blocks, W, a=P_["a"], b=P_["b"], d=P_["d"],
                              beta=2, C_cap=P_["C_cap"], w_c=0.0)
        base = c[0].astype(np.float64)
        K = (m + W - 1) // W
        left, expect = m, 0.0
        for j in np.argsort(base, kind="stable"):
            take = min(K, left)
            expect += take * base[j]
            left -= take
        _, o, _ = orc.poa_window(worker, overlap, blocks, W, a=P_["a"], b=P_["b"], d=P_["d"],
                                 beta=2, C_cap=P_["C_cap"], w_c=0.0)
        assert o == pytest.approx(expect, rel=1e-12)


def test_poa_at_least_one_when_greedy_is_feasible(orc):
    rng = np.random.default_rng(12)
    hit = 0
    for _ in range(200):
        W = int(rng.integers(1, 6))
        m = int(rng.integers(1, 40))
        worker, overlap, blocks = _window(rng, m, W)
        K = (m + W - 1) // W
        if np.bincount(worker, minlength=W).max() > K:
            continue
        hit += 1
        s, o, _ = orc.poa_window(worker, overlap, blocks, W, **P_)
        assert s >= o * (1 - 1e-12)
    assert hit > 10


def test_hand_window(orc):
    # four requests, all greedily on worker 0 where they are fully cached; worker 1 idle.
    # n = (4, 0); c_i0 = 4a + b + d/60^2 - w_c, c_i1 = b + d/64^2; OPT puts two on each.
    worker = np.zeros(4, np.int32)
    blocks = np.full(4, 8, np.int32)
    overlap = np.array([[8, 0]] * 4, np.int32)
    s, o, _ = orc.poa_window(worker, overlap, blocks, 2, **P_)
    a, b, d, wc = (Fraction(P_[k]) for k in ("a", "b", "d", "w_c"))
    c0 = 4 * a + b + d / 3600 - wc
    c1 = b + d / 4096
    assert s == pytest.approx(float(4 * c0), rel=1e-6)
    assert o == pytest.approx(float(2 * c0 + 2 * c1), rel=1e-6)
    assert s / o == pytest.approx(float((4 * c0) / (2 * c0 + 2 * c1)), rel=1e-6)


def test_windows_split_and_empty(orc):
    rng = np.random.default_rng(1)
    worker, overlap, blocks = _window(rng, 23, 3)
    s, o = orc.poa_windows(worker, overlap, blocks, 3, 8, **P_)
    assert s.shape == (3,)
    s2, o2, _ = orc.poa_window(worker[16:], overlap[16:], blocks[16:], 3, **P_)
    assert s[2] == s2 and o[2] == o2
    s, o, _ = orc.poa_window(worker[:0], overlap[:0], blocks[:0], 3, **P_)
    assert s == 0.0 and o == 0.0
