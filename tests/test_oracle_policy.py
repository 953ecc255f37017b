"""Pins of the oracle's worker-selection policies: the softmax of
Eq. router-softmax at temperature tau > 0 (with its float exp), and the static
counterfactual policies of the discussion section (round robin, uniform
random, power of two choices).  Distributions are checked on exact grids of
the random words against probabilities computed independently in fp64."""
import math

import numpy as np
import pytest

import brute
from paper_2606_17081_amd import workload as wl

ARGMIN, SOFTMAX, RR, RANDOM, P2C = (wl.POLICY_ARGMIN, wl.POLICY_SOFTMAX, wl.POLICY_ROUND_ROBIN,
                                    wl.POLICY_RANDOM, wl.POLICY_P2C)
GRID = [k << 16 for k in range(1 << 16)]          # r0 with u = k / 2^16 exactly


def test_exp_against_libm(orc):
    xs = np.concatenate([np.linspace(-87.0, 0.0, 20001, dtype=np.float32),
                         -np.logspace(-8, 1.9, 2000).astype(np.float32)])
    for x in xs:
        ref = math.exp(float(x))
        assert abs(orc.exp_neg(float(x)) - ref) <= 2.5e-7 * ref, float(x)
    assert orc.exp_neg(0.0) == 1.0
    assert orc.exp_neg(-87.5) == 0.0 and orc.exp_neg(-1e30) == 0.0
    v = [orc.exp_neg(float(x)) for x in np.linspace(-20.0, 0.0, 4001, dtype=np.float32)]
    assert all(a <= b for a, b in zip(v, v[1:]))           # monotone


def _freq(orc, policy, tau, costs, rs0, rs1=(0,)):
    W = len(costs)
    cnt = np.zeros(W, np.int64)
    for r0 in rs0:
        for r1 in rs1:
            cnt[orc.select(policy, tau, costs, 0, r0, r1)] += 1
    return cnt / cnt.sum()


@pytest.mark.parametrize("costs,tau", [([3.0, 1.0, 1.0, 2.0], 1.0), ([10.0, 12.5, 11.0], 2.0),
                                       ([100.0, 101.0, 140.0, 100.5, 99.0], 16.0), ([5.0], 3.0),
                                       ([0.0, 0.0, 0.0, 0.0, 0.0, 0.0], 0.7)])
def test_softmax_frequencies_match_probabilities(orc, costs, tau):
    c = np.array(costs, np.float64)
    p = np.exp(-c / tau)
    p /= p.sum()
    f = _freq(orc, SOFTMAX, tau, costs, GRID)
    np.testing.assert_allclose(f, p, atol=2.0 ** -16 * len(costs) + 2e-6)


def test_softmax_limits(orc):
    rng = np.random.default_rng(5)
    for _ in range(20):
        costs = rng.uniform(0, 100, size=int(rng.integers(2, 9))).astype(np.float32).tolist()
        am = orc.select(ARGMIN, 0.0, costs)
        assert am == int(np.argmin(costs))
        # a temperature far below the cost gaps: only the least cost has weight
        gap = np.diff(np.sort(costs)).min()
        if gap > 0:
            tau = float(gap) / 200.0
            assert set(orc.select(SOFTMAX, tau, costs, 0, r0, 0) for r0 in GRID[::257]) == {am}
        # a temperature far above the costs: uniform
        f = _freq(orc, SOFTMAX, 1e12, costs, GRID)
        np.testing.assert_allclose(f, 1.0 / len(costs), atol=2.0 ** -16 * len(costs))
    # the draw's extremes stay in range
    assert orc.select(SOFTMAX, 1.0, [1.0, 2.0], 0, 0, 0) == 0
    assert orc.select(SOFTMAX, 1.0, [1.0, 2.0], 0, 0xFFFFFFFF, 0) == 1


def test_round_robin_and_random(orc):
    for W in (1, 2, 5, 6, 64):
        assert [orc.select(RR, 0.0, [0.0] * W, t) for t in range(3 * W + 2)] == [t % W for t in range(3 * W + 2)]
        cnt = np.bincount([orc.select(RANDOM, 0.0, [0.0] * W, 0, r0) for r0 in GRID], minlength=W)
        assert cnt.size == W and cnt.max() - cnt.min() <= 1
        assert orc.select(RANDOM, 0.0, [0.0] * W, 0, 0xFFFFFFFF) == W - 1


@pytest.mark.parametrize("W", [2, 3, 6, 7])
def test_power_of_two_choices(orc, W):
    # strictly increasing costs: worker j wins when it is drawn with a costlier one,
    # P = 2 (W - 1 - j) / (W (W - 1))
    costs = [float(10 + 3 * j) for j in range(W)]
    rs = [k << 24 for k in range(256)]
    f = _freq(orc, P2C, 0.0, costs, rs, rs)
    p = np.array([2.0 * (W - 1 - j) / (W * (W - 1)) for j in range(W)])
    np.testing.assert_allclose(f, p, atol=2.0 / 256)
    # equal costs: the lower index of the two
    f = _freq(orc, P2C, 0.0, [1.0] * W, rs, rs)
    np.testing.assert_allclose(f, p, atol=2.0 / 256)
    assert orc.select(P2C, 0.0, [4.0], 0, 123, 456) == 0


def test_bad_policies_rejected(orc):
    assert orc.select(9, 0.0, [1.0, 2.0]) == -1
    tr = wl.tiny_trace(0)
    with pytest.raises(ValueError):
        orc.simulate_trace(4, 256, wl.EpisodeSpec(seed=0, concurrency=8, policy=SOFTMAX, tau=0.0), tr)
    with pytest.raises(ValueError):
        orc.simulate_trace(4, 256, wl.EpisodeSpec(seed=0, concurrency=8, policy=7), tr)


@pytest.mark.parametrize("field,value", [("w_ov", -1.0), ("w_act", -0.5), ("w_sat", float("nan")),
                                         ("ctrl_w_ov", -0.25)])
def test_negative_or_nan_weights_rejected(orc, field, value):
    tr = wl.tiny_trace(0)
    with pytest.raises(ValueError):
        orc.simulate_trace(4, 256, wl.EpisodeSpec(seed=0, concurrency=8, **{field: value}), tr)


@pytest.mark.parametrize("policy,tau", [(SOFTMAX, 0.5), (SOFTMAX, 4.0), (RR, 0.0), (RANDOM, 0.0), (P2C, 0.0)])
@pytest.mark.parametrize("seed", range(6))
def test_episode_policies_match_twin(orc, policy, tau, seed):
    """The episode loop hands route t its costs and words (rand[2t], rand[2t+1]):
    checked against the OrderedDict twin driving the same selection rule."""
    from test_oracle_episode import _flat_chains, _random_case
    rng = np.random.default_rng(7000 + seed)
    W, cache, spec, turn_off, turn_blocks, chains = _random_case(rng, multiturn=seed % 2 == 1)
    spec.policy, spec.tau = policy, tau
    n = int(turn_off[-1])
    rand = rng.integers(0, 1 << 32, size=2 * n, dtype=np.uint64).astype(np.uint32)
    flat, off = _flat_chains(chains)
    out = orc.simulate_episode(W, cache, spec, turn_off, turn_blocks, off, flat, rand=rand)
    sel = lambda costs, t: orc.select(policy, tau, np.array(costs, np.float32), t, int(rand[2 * t]),
                                      int(rand[2 * t + 1]))
    routes, _ = brute.episode(W, cache, spec.hold_steps, spec.routes_per_step, spec.w_ov, spec.w_act,
                              spec.w_sat, spec.cap, turn_off, turn_blocks, chains, spec.controller,
                              spec.ctrl_w_ov, spec.ctrl_window, spec.ctrl_num, spec.ctrl_den, select=sel)
    assert [r["worker"] for r in routes] == out["route_worker"].tolist()
    assert [r["overlap"] for r in routes] == out["overlap"].tolist()
    assert [len(r["evicted"]) for r in routes] == out["evict_count"].tolist()


def test_route_rand_is_seeded():
    sp = wl.EpisodeSpec(seed=3, concurrency=64, policy=RANDOM)
    a, b = wl.route_rand(sp, 100), wl.route_rand(sp, 100)
    assert a.dtype == np.uint32 and a.shape == (200,) and np.array_equal(a, b)
    assert not np.array_equal(a, wl.route_rand(wl.EpisodeSpec(seed=4, concurrency=64, policy=RANDOM), 100))
