"""Pins of the oracle's memory tiers (Section 4.2, Eq. kv-cost): under LRU a
worker's k1 most recently used blocks form G1, the next k2 G2 and the rest G3,
and the router's prefill term charges a cached block by its tier.  Checked by a
brute-force twin, reductions to the untiered cost and hand-worked cases."""
import numpy as np
import pytest

import brute
from paper_2606_17081_amd import workload as wl
from test_oracle_episode import _flat_chains, _random_case


def _tiered(spec, k1, k2, tw):
    return wl.EpisodeSpec(**{**spec.__dict__, "tier_g1": k1, "tier_g2": k2, "tier_w": tuple(tw)})


def _tier_sizes(rng, cache, small=False):
    k1 = int(rng.integers(1, max(1, cache // 3) + 1))     # small G1, so prefixes straddle tiers
    k2 = int(rng.integers(1, max(1, cache // 4) + 1)) if small else int(rng.integers(0, cache - k1 + 1))
    return k1, k2


def _twin(orc, rng, W, cache, spec, turn_off, turn_blocks, chains, small=False):
    k1, k2 = _tier_sizes(rng, cache, small)
    tw = [float(x) for x in rng.choice([0.0, 0.125, 0.3, 0.5, 1.0, 2.0], size=3)]
    spec = _tiered(spec, k1, k2, tw)
    flat, off = _flat_chains(chains)
    out = orc.simulate_episode(W, cache, spec, turn_off, turn_blocks, off, flat, dump=True, evicted_cap=100000)
    routes, final = brute.episode(W, cache, spec.hold_steps, spec.routes_per_step, spec.w_ov, spec.w_act,
                                  spec.w_sat, spec.cap, turn_off, turn_blocks, chains, spec.controller,
                                  spec.ctrl_w_ov, spec.ctrl_window, spec.ctrl_num, spec.ctrl_den,
                                  tiers=(k1, k2, tw))
    for t, r in enumerate(routes):
        assert out["route_worker"][t] == r["worker"], t
        assert out["overlap"][t].tolist() == r["overlap"], t
        assert [tuple(x) for x in out["tier_overlap"][t].tolist()] == r["tier_overlap"], t
        assert out["cost"][t].view(np.uint32).tolist() == [np.float32(c).view(np.uint32) for c in r["cost"]], t
    assert out["evicted_keys"].tolist() == [k for r in routes for k in r["evicted"]]
    assert [k.tolist() for k in out["final_keys"]] == final
    o = out["overlap"]
    o1, o12 = out["tier_overlap"][..., 0], out["tier_overlap"][..., 1]
    assert np.all(o1 <= o12) and np.all(o12 <= o)


@pytest.mark.parametrize("seed", range(40))
def test_matches_bruteforce_twin(orc, seed):
    rng = np.random.default_rng(11000 + seed)
    W, cache, spec, turn_off, turn_blocks, chains = _random_case(rng, multiturn=seed % 2 == 1)
    _twin(orc, rng, W, cache, spec, turn_off, turn_blocks, chains)


@pytest.mark.parametrize("seed", range(12))
def test_matches_bruteforce_twin_arbitrary_keys(orc, seed):
    # keys from a tiny alphabet: the tiers need not be prefixes of a chain's cached blocks
    rng = np.random.default_rng(13000 + seed)
    W, cache, spec, turn_off, turn_blocks, chains = _random_case(rng, multiturn=seed % 2 == 1)
    chains = [list(dict.fromkeys(int(x) for x in rng.integers(1, 6, size=len(c)))) for c in chains]
    tb = [min(turn_blocks[t], len(chains[c])) for c in range(len(chains)) for t in range(turn_off[c], turn_off[c + 1])]
    _twin(orc, rng, W, cache, spec, turn_off, tb, chains)


@pytest.mark.parametrize("seed", range(6))
def test_single_tier_reduces_to_untiered(orc, seed):
    # G1 = the whole cache at weight 0: every cached block is free, as without tiers
    rng = np.random.default_rng(300 + seed)
    W, cache, spec, turn_off, turn_blocks, chains = _random_case(rng, multiturn=True)
    flat, off = _flat_chains(chains)
    base = orc.simulate_episode(W, cache, spec, turn_off, turn_blocks, off, flat, dump=True, evicted_cap=10 ** 5)
    tiered = orc.simulate_episode(W, cache, _tiered(spec, cache, 0, (0.0, 0.7, 0.9)), turn_off, turn_blocks, off,
                                  flat, dump=True, evicted_cap=10 ** 5)
    for k in ("route_worker", "overlap", "evict_count", "evicted_keys", "totals"):
        assert np.array_equal(base[k], tiered[k]), k
    assert np.array_equal(base["cost"].view(np.uint32), tiered["cost"].view(np.uint32))
    assert np.array_equal(tiered["tier_overlap"][..., 0], base["overlap"])
    assert np.array_equal(tiered["tier_overlap"][..., 1], base["overlap"])


def test_full_weight_tiers_cost_like_no_cache(orc):
    # every tier at weight 1: a cached block costs what recomputing it does, so the prefill
    # term is P on every worker (exact: integers below 2^24)
    rng = np.random.default_rng(5)
    W, cache, spec, turn_off, turn_blocks, chains = _random_case(rng, multiturn=True)
    spec = wl.EpisodeSpec(**{**spec.__dict__, "w_act": 0.0, "w_sat": 0.0})
    flat, off = _flat_chains(chains)
    out = orc.simulate_episode(W, cache, _tiered(spec, max(1, cache // 3), cache // 3, (1.0, 1.0, 1.0)),
                               turn_off, turn_blocks, off, flat)
    P = out["route_blocks"].astype(np.float32)
    want = (np.float32(spec.w_ov) * P)[:, None] * np.ones((1, W), np.float32)
    assert np.array_equal(out["cost"], want)


def test_hand_worked_tiers(orc):
    # one worker, 6-block cache, G1 = 2 blocks, G2 = 2, G3 = 2; one route per step.
    # A = [1, 2], B = [3, 4]: recency (newest first) 3 4 1 2, so G1 = {3, 4}, G2 = {1, 2}.
    # A' = [1, 2, 7]: o = 2, none in G1, both in G1 u G2 -> (o1, o12) = (0, 2);
    #   prefill (3 - 2) + 0.25 * 2 = 1.5.  Recency now 1 2 7 3 4: G1 = {1, 2}, G2 = {7, 3}.
    # C = [3, 4, 8]: o = 2, block 3 in G2, block 4 in G3 -> (0, 1);
    #   prefill 1 + 0.25 * 1 + 0.5 * 1 = 1.75.
    chains = [[1, 2], [3, 4], [1, 2, 7], [3, 4, 8]]
    flat, off = _flat_chains(chains)
    spec = wl.EpisodeSpec(seed=0, concurrency=1, hold_steps=1, w_ov=1.0, w_act=0.0, w_sat=0.0, cap=1 << 20,
                          tier_g1=2, tier_g2=2, tier_w=(0.0, 0.25, 0.5))
    out = orc.simulate_episode(1, 6, spec, [0, 1, 2, 3, 4], [2, 2, 3, 3], off, flat)
    assert out["overlap"][:, 0].tolist() == [0, 0, 2, 2]
    assert out["tier_overlap"][:, 0].tolist() == [[0, 0], [0, 0], [0, 2], [0, 1]]
    assert out["cost"][:, 0].tolist() == [2.0, 2.0, 1.5, 1.75]


def test_rejects_bad_parameters(orc):
    flat, off = _flat_chains([[1]])
    for kw in (dict(tier_g1=3, tier_g2=2), dict(tier_g1=-1), dict(tier_g1=1, tier_g2=-1),
               dict(tier_g1=1, evict_policy=wl.EVICT_FREQ, decay_steps=1), dict(tier_g1=1, tier_w=(0.0, -1.0, 0.0))):
        spec = wl.EpisodeSpec(**{**wl.EpisodeSpec(seed=0, concurrency=1, hold_steps=1).__dict__, **kw})
        with pytest.raises(ValueError):
            orc.simulate_episode(1, 4, spec, [0, 1], [1], off, flat)


def _straddle_case(rng):
    # conversations whose turns extend one chain, caches a few prompts deep: cached prefixes
    # run through all three tiers
    W, cache = int(rng.integers(1, 4)), int(rng.integers(24, 48))
    n_conv = int(rng.integers(6, 16))
    chains, turn_blocks, turn_off, nxt = [], [], [0], 1
    shared = [list(range(1000 * (g + 1), 1000 * (g + 1) + 12)) for g in range(3)]
    for _ in range(n_conv):
        g = int(rng.integers(0, 3))
        L = int(rng.integers(14, 30))
        head = shared[g][: int(rng.integers(2, 12))]
        ch = head + list(range(nxt, nxt + L - len(head)))
        nxt += L
        chains.append(ch)
        tb = sorted(int(x) for x in rng.integers(len(head), L + 1, size=int(rng.integers(1, 4))))
        turn_blocks.extend(tb)
        turn_off.append(len(turn_blocks))
    H, rps = int(rng.integers(1, 4)), int(rng.integers(1, 3))
    spec = wl.EpisodeSpec(seed=0, concurrency=H * rps, hold_steps=H, w_ov=1.0, w_act=float(rng.choice([0.0, 0.5])),
                          w_sat=0.0, cap=64)
    return W, cache, spec, turn_off, turn_blocks, chains


@pytest.mark.parametrize("seed", range(16))
def test_matches_bruteforce_twin_straddling(orc, seed):
    rng = np.random.default_rng(17000 + seed)
    W, cache, spec, turn_off, turn_blocks, chains = _straddle_case(rng)
    _twin(orc, rng, W, cache, spec, turn_off, turn_blocks, chains, small=True)


def test_straddling_cases_cover_every_tier(orc):
    # the straddling twin cases do put cached prefixes across G1, G2 and G3
    n3 = 0
    for seed in range(16):
        rng = np.random.default_rng(17000 + seed)
        W, cache, spec, turn_off, turn_blocks, chains = _straddle_case(rng)
        k1, k2 = _tier_sizes(rng, cache, small=True)
        tw = [float(x) for x in rng.choice([0.0, 0.125, 0.3, 0.5, 1.0, 2.0], size=3)]
        flat, off = _flat_chains(chains)
        out = orc.simulate_episode(W, cache, _tiered(spec, k1, k2, tw), turn_off, turn_blocks, off, flat)
        t, o = out["tier_overlap"], out["overlap"]
        n3 += int(((0 < t[..., 0]) & (t[..., 0] < t[..., 1]) & (t[..., 1] < o)).sum())
    assert n3 >= 15
