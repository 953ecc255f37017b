"""Pins of the oracle's frequency eviction (the KV block manager's policy of
Section 2.2: frequency 1 on insert, doubled on a hit, minus 1 per time-decay
step and never below 1; least frequent block first, least recently used among
equals): a brute-force twin, a reduction to LRU, hand-worked eviction orders
and invariants."""
import numpy as np
import pytest

import brute
from paper_2606_17081_amd import workload as wl
from test_oracle_episode import _flat_chains, _parent_map, _random_case

CAP = 1 << 20


def _freq(spec, T):
    return wl.EpisodeSpec(**{**spec.__dict__, "evict_policy": wl.EVICT_FREQ, "decay_steps": T})


def _brute(W, cache, spec, turn_off, turn_blocks, chains, T):
    return brute.episode(W, cache, spec.hold_steps, spec.routes_per_step, spec.w_ov, spec.w_act, spec.w_sat,
                         spec.cap, turn_off, turn_blocks, chains, spec.controller, spec.ctrl_w_ov,
                         spec.ctrl_window, spec.ctrl_num, spec.ctrl_den, freq=(T, CAP))


@pytest.mark.parametrize("seed", range(48))
def test_matches_bruteforce_twin(orc, seed):
    rng = np.random.default_rng(7000 + seed)
    W, cache, spec, turn_off, turn_blocks, chains = _random_case(rng, multiturn=seed % 2 == 1)
    T = int(rng.choice([1, 2, 3, 5, 1000]))
    spec = _freq(spec, T)
    flat, off = _flat_chains(chains)
    out = orc.simulate_episode(W, cache, spec, turn_off, turn_blocks, off, flat, dump=True, evicted_cap=100000)
    routes, final = _brute(W, cache, spec, turn_off, turn_blocks, chains, T)
    ev = []
    for t, r in enumerate(routes):
        assert out["route_worker"][t] == r["worker"]
        assert out["route_step"][t] == r["step"]
        assert out["overlap"][t].tolist() == r["overlap"]
        assert out["evict_count"][t] == len(r["evicted"])
        ev.extend(r["evicted"])
    assert out["evicted_keys"].tolist() == ev
    assert [k.tolist() for k in out["final_keys"]] == final


@pytest.mark.parametrize("seed", range(12))
def test_matches_bruteforce_twin_arbitrary_keys(orc, seed):
    # keys from a tiny alphabet: caches are not prefix-closed and hits land past the first miss
    rng = np.random.default_rng(9000 + seed)
    W, cache, spec, turn_off, turn_blocks, chains = _random_case(rng, multiturn=seed % 2 == 1)
    chains = [list(dict.fromkeys(int(x) for x in rng.integers(1, 6, size=len(c)))) for c in chains]
    tb = [min(turn_blocks[t], len(chains[c])) for c in range(len(chains)) for t in range(turn_off[c], turn_off[c + 1])]
    T = int(rng.choice([1, 2, 4]))
    spec = _freq(spec, T)
    flat, off = _flat_chains(chains)
    out = orc.simulate_episode(W, cache, spec, turn_off, tb, off, flat, dump=True, evicted_cap=100000)
    routes, final = _brute(W, cache, spec, turn_off, tb, chains, T)
    assert [r["worker"] for r in routes] == out["route_worker"].tolist()
    assert [r["overlap"] for r in routes] == out["overlap"].tolist()
    assert out["evicted_keys"].tolist() == [k for r in routes for k in r["evicted"]]
    assert [k.tolist() for k in out["final_keys"]] == final


@pytest.mark.parametrize("seed", range(6))
def test_reduces_to_lru_without_hits(orc, seed):
    # every block is touched once (distinct chains, one turn each): every frequency stays 1,
    # so frequency eviction is least-recently-used eviction, for any decay period
    rng = np.random.default_rng(100 + seed)
    n, W, cache = 40, int(rng.integers(1, 4)), int(rng.integers(3, 30))
    lens = rng.integers(1, 9, size=n)
    chains, nxt = [], 1
    for L in lens:
        chains.append(list(range(nxt, nxt + int(L))))
        nxt += int(L)
    flat, off = _flat_chains(chains)
    turn_off = list(range(n + 1))
    spec = wl.EpisodeSpec(seed=0, concurrency=4, hold_steps=2, cap=8)
    lru = orc.simulate_episode(W, cache, spec, turn_off, lens, off, flat, dump=True, evicted_cap=10 ** 5)
    for T in (1, 3, 100):
        fr = orc.simulate_episode(W, cache, _freq(spec, T), turn_off, lens, off, flat, dump=True,
                                  evicted_cap=10 ** 5)
        for k in ("route_worker", "overlap", "evict_count", "evicted_keys"):
            assert np.array_equal(fr[k], lru[k]), k
        assert [k.tolist() for k in fr["final_keys"]] == [k.tolist() for k in lru["final_keys"]]
    assert int(lru["totals"][1]) > 0


def _one_worker(orc, chains, cache, T, evict_policy):
    # one worker, one route per step: route t runs at step t
    flat, off = _flat_chains(chains)
    spec = wl.EpisodeSpec(seed=0, concurrency=1, hold_steps=1, cap=1 << 20, evict_policy=evict_policy,
                          decay_steps=T)
    n = len(chains)
    return orc.simulate_episode(1, cache, spec, list(range(n + 1)), [len(c) for c in chains], off, flat,
                                dump=True, evicted_cap=1000)


def test_hot_prefix_survives_where_lru_drops_it(orc):
    # prompt A = [1, 2] is sent three times (frequencies 1 -> 2 -> 4), then cold prompts
    # [10, 11], [20, 21], [30, 31] fill a 6-block cache.  LRU evicts A's blocks, the oldest;
    # frequency eviction (no decay within the episode) evicts each cold prompt's blocks
    # instead, the deeper block first (it has the older touch).
    chains = [[1, 2], [1, 2], [1, 2], [10, 11], [20, 21], [30, 31]]
    lru = _one_worker(orc, chains, 6, 1, wl.EVICT_LRU)
    fr = _one_worker(orc, chains, 6, 1000, wl.EVICT_FREQ)
    assert lru["evicted_keys"].tolist() == [2, 1]
    assert fr["evicted_keys"].tolist() == [11, 10]
    assert fr["final_keys"][0].tolist() == [2, 1, 21, 20, 31, 30]
    assert fr["evict_count"].tolist() == [0, 0, 0, 0, 0, 2]


def test_decay_lets_a_hot_prefix_go(orc):
    # same prompts with a decay step before every step: A's frequency goes 1, 2 (after a
    # decay to 1), 2, then back to 1 at step 3; at step 5 every block is at 1 and A's blocks
    # are the oldest
    chains = [[1, 2], [1, 2], [1, 2], [10, 11], [20, 21], [30, 31]]
    fr = _one_worker(orc, chains, 6, 1, wl.EVICT_FREQ)
    assert fr["evicted_keys"].tolist() == [2, 1]
    # a decay step every 2 steps (steps 2 and 4): A goes 1, 2, 2, 2, 1 -- gone again
    fr2 = _one_worker(orc, chains, 6, 2, wl.EVICT_FREQ)
    assert fr2["evicted_keys"].tolist() == [2, 1]
    # every 3 steps (step 3 only, before step 5): A goes 1, 2, 4, 3 and survives
    fr3 = _one_worker(orc, chains, 6, 3, wl.EVICT_FREQ)
    assert fr3["evicted_keys"].tolist() == [11, 10]


def test_many_hits_then_cold_blocks(orc):
    # 30 hits take the frequency to the cap (2^20, reached after 20); a block there still
    # outlives the blocks at frequency 1, of which the older goes first
    chains = [[1]] * 31 + [[5], [6]]
    fr = _one_worker(orc, chains, 2, 10 ** 6, wl.EVICT_FREQ)
    assert fr["evicted_keys"].tolist() == [5]
    assert fr["final_keys"][0].tolist() == [1, 6]


@pytest.mark.parametrize("T", [1, 4, 32])
def test_invariants_under_pressure(orc, T):
    # the tiny workload with 64-block caches: capacity, prefix closure (a parent is at least as
    # frequent as its child and touched later), and insert - evict = cached
    w = wl.tiny_workload()
    tr = w.traces[0]
    chains = orc.trace_chains(tr)
    per_conv = [chains[tr.chain_off[c]:tr.chain_off[c + 1]] for c in range(tr.n_conv)]
    out = orc.simulate_trace(w.W, 64, _freq(w.episodes[0], T), tr, chains, dump=True, evicted_cap=10 ** 6)
    assert int(out["totals"][1]) > 0
    assert int(out["totals"][0]) - int(out["totals"][1]) == int(out["totals"][7])
    parent = _parent_map(per_conv)
    for keys in out["final_keys"]:
        assert len(keys) <= 64
        s = set(int(k) for k in keys)
        assert all(parent[k] in s for k in s if k in parent)
    assert np.all(out["overlap"] <= out["route_blocks"][:, None])


def test_rejects_bad_parameters(orc):
    flat, off = _flat_chains([[1]])
    spec = wl.EpisodeSpec(seed=0, concurrency=1, hold_steps=1, evict_policy=wl.EVICT_FREQ, decay_steps=0)
    with pytest.raises(ValueError):
        orc.simulate_episode(1, 4, spec, [0, 1], [1], off, flat)
    spec = wl.EpisodeSpec(seed=0, concurrency=1, hold_steps=1, evict_policy=2, decay_steps=1)
    with pytest.raises(ValueError):
        orc.simulate_episode(1, 4, spec, [0, 1], [1], off, flat)
