"""Pins of the oracle's routing episodes: hand fixtures, a brute-force twin, invariants."""
import json
import os

import numpy as np
import pytest

import brute
from paper_2606_17081_amd import workload as wl

GOLD = os.path.join(os.path.dirname(__file__), "golden", "episode_hand.json")


def _spec(case):
    return wl.EpisodeSpec(seed=0, concurrency=case["routes_per_step"] * case["H"],
                          hold_steps=case["H"], w_ov=case["w_ov"], w_act=case["w_act"],
                          w_sat=case["w_sat"], cap=case["cap"], controller=case["controller"],
                          ctrl_w_ov=case.get("ctrl_w_ov", 0.25), ctrl_window=case.get("ctrl_window", 128),
                          ctrl_num=case.get("ctrl_num", 9), ctrl_den=case.get("ctrl_den", 10))


def _flat_chains(chains):
    off = np.zeros(len(chains) + 1, np.int64)
    np.cumsum([len(c) for c in chains], out=off[1:])
    flat = np.array([k for c in chains for k in c], np.uint64)
    return flat, off


@pytest.mark.parametrize("idx", range(3))
def test_hand_fixtures(orc, idx):
    with open(GOLD) as f:
        case = json.load(f)["cases"][idx]
    flat, off = _flat_chains(case["chains"])
    out = orc.simulate_episode(case["W"], case["cache_blocks"], _spec(case), case["turn_off"],
                               case["turn_blocks"], off, flat, dump=True, evicted_cap=64)
    ex = case["expect"]
    for k in ("route_turn", "route_worker", "route_step", "evict_count", "last_hash"):
        assert out[k].tolist() == ex[k], k
    assert out["overlap"].tolist() == ex["overlap"]
    assert out["cost"].tolist() == ex["cost"]
    assert out["evicted_keys"].tolist() == ex["evicted_keys"]
    t = out["totals"]
    assert t[0] == ex["totals"]["prefill"] and t[1] == ex["totals"]["evicted"]
    assert t[2] == ex["totals"]["sum_P"] and t[5] == ex["totals"]["steps"]
    assert t[6] == ex["totals"]["sum_overlap"] and t[7] == ex["totals"]["cached"]
    if "ctrl_routes" in ex["totals"]:
        assert t[3] == ex["totals"]["ctrl_routes"] and t[4] == ex["totals"]["ctrl_activations"]
    assert [k.tolist() for k in out["final_keys"]] == ex["final"]


def _random_case(rng, multiturn):
    W = int(rng.integers(1, 5))
    cache = int(rng.integers(2, 12))
    H = int(rng.integers(1, 4))
    rps = int(rng.integers(1, 4))
    n_conv = int(rng.integers(1, 14))
    # chains over a small alphabet of "tokens" so prefixes are shared; keys are
    # prefix identifiers (as chained hashes are)
    chains, turn_blocks, turn_off = [], [], [0]
    prefix_id = {}
    for _ in range(n_conv):
        L = int(rng.integers(1, 9))
        path = tuple(int(x) for x in rng.integers(0, 3, size=L))
        ch = []
        for k in range(1, L + 1):
            ch.append(prefix_id.setdefault(path[:k], len(prefix_id) + 1))
        chains.append(ch)
        if multiturn:
            nt = int(rng.integers(1, 4))
            tb = sorted(int(x) for x in rng.integers(0, L + 1, size=nt))
        else:
            tb = [L]
        turn_blocks.extend(tb)
        turn_off.append(len(turn_blocks))
    ctrl = int(rng.integers(0, 2))
    spec = wl.EpisodeSpec(seed=0, concurrency=rps * H, hold_steps=H,
                          w_ov=float(rng.choice([0.0, 0.25, 1.0, 2.0])), w_act=float(rng.choice([0.0, 0.5, 1.0])),
                          w_sat=float(rng.choice([0.0, 4.0])), cap=int(rng.integers(1, 20)),
                          controller=ctrl, ctrl_window=int(rng.integers(1, 5)),
                          ctrl_num=int(rng.integers(0, 10)), ctrl_den=10)
    return W, cache, spec, turn_off, turn_blocks, chains


@pytest.mark.parametrize("seed", range(40))
def test_matches_bruteforce_twin(orc, seed):
    rng = np.random.default_rng(1000 + seed)
    W, cache, spec, turn_off, turn_blocks, chains = _random_case(rng, multiturn=seed % 2 == 1)
    flat, off = _flat_chains(chains)
    out = orc.simulate_episode(W, cache, spec, turn_off, turn_blocks, off, flat, dump=True,
                               evicted_cap=100000)
    routes, final = brute.episode(W, cache, spec.hold_steps, spec.routes_per_step, spec.w_ov,
                                  spec.w_act, spec.w_sat, spec.cap, turn_off, turn_blocks, chains,
                                  spec.controller, spec.ctrl_w_ov, spec.ctrl_window, spec.ctrl_num,
                                  spec.ctrl_den)
    assert len(routes) == len(out["route_worker"]) == turn_off[-1]
    ev = []
    for t, r in enumerate(routes):
        assert out["route_turn"][t] == r["turn"]
        assert out["route_worker"][t] == r["worker"]
        assert out["route_step"][t] == r["step"]
        assert out["route_blocks"][t] == r["P"]
        assert out["overlap"][t].tolist() == r["overlap"]
        assert out["cost"][t].view(np.uint32).tolist() == \
            [np.float32(c).view(np.uint32) for c in r["cost"]]
        assert out["evict_count"][t] == len(r["evicted"])
        ev.extend(r["evicted"])
    assert out["evicted_keys"].tolist() == ev
    assert [k.tolist() for k in out["final_keys"]] == final
    assert out["totals"][3] == sum(r["active"] for r in routes)
    assert out["totals"][4] == sum(r["first_active"] for r in routes)


def _parent_map(chains):
    parent = {}
    for ch in chains:
        for k in range(1, len(ch)):
            parent[int(ch[k])] = int(ch[k - 1])
    return parent


def test_tiny_workload_invariants(orc):
    w = wl.tiny_workload()
    tr = w.traces[0]
    spec = w.episodes[0]
    chains = orc.trace_chains(tr)
    per_conv = [chains[tr.chain_off[c]:tr.chain_off[c + 1]] for c in range(tr.n_conv)]
    out = orc.simulate_trace(w.W, w.cache_blocks, spec, tr, chains, dump=True, evicted_cap=10 ** 6)
    n = tr.n_turns
    R = spec.routes_per_step
    # single-turn: requests are routed in index order, C/H per step
    assert out["route_turn"].tolist() == list(range(n))
    assert out["route_step"].tolist() == [t // R for t in range(n)]
    assert np.all(out["overlap"] >= 0)
    assert np.all(out["overlap"] <= out["route_blocks"][:, None])
    # occupancy never exceeds capacity, and caches stay prefix-closed
    parent = _parent_map(per_conv)
    for keys in out["final_keys"]:
        assert len(keys) <= w.cache_blocks
        s = set(int(k) for k in keys)
        for k in s:
            if k in parent:
                assert parent[k] in s
    # conservation: blocks inserted - evicted = blocks still cached
    inserted = int(out["totals"][0])      # misses on the chosen worker are inserted
    assert inserted - int(out["totals"][1]) == int(out["totals"][7])
    assert out["last_hash"].tolist() == [int(c[-1]) for c in per_conv]


def test_eviction_pressure_invariants(orc):
    # the tiny trace with 64-block caches: eviction happens, capacity and prefix closure hold
    w = wl.tiny_workload()
    tr = w.traces[0]
    chains = orc.trace_chains(tr)
    per_conv = [chains[tr.chain_off[c]:tr.chain_off[c + 1]] for c in range(tr.n_conv)]
    out = orc.simulate_trace(w.W, 64, w.episodes[0], tr, chains, dump=True, evicted_cap=10 ** 6)
    assert int(out["totals"][1]) > 0
    assert int(out["totals"][0]) - int(out["totals"][1]) == int(out["totals"][7])
    parent = _parent_map(per_conv)
    for keys in out["final_keys"]:
        assert len(keys) <= 64
        s = set(int(k) for k in keys)
        assert all(parent[k] in s for k in s if k in parent)
    assert int(out["evict_count"].sum()) == int(out["totals"][1])


def test_overlap_is_first_miss_in_episodes(orc):
    # key 2 is cached by the first request, but the second request's block 0 (key 3) is not:
    # the cached prefix of [3, 2] is empty although one of its blocks is cached
    flat, off = _flat_chains([[1, 2], [3, 2], [1, 5, 2]])
    spec = wl.EpisodeSpec(seed=0, concurrency=1, hold_steps=1, w_ov=1.0, w_act=0.0, w_sat=0.0,
                          cap=8)
    out = orc.simulate_episode(1, 16, spec, [0, 1, 2, 3], [2, 2, 3], off, flat)
    assert out["overlap"][:, 0].tolist() == [0, 0, 1]


@pytest.mark.parametrize("seed", range(12))
def test_matches_bruteforce_twin_arbitrary_keys(orc, seed):
    # keys drawn from a tiny alphabet, so caches are not prefix-closed along chains
    rng = np.random.default_rng(5000 + seed)
    W, cache, spec, turn_off, turn_blocks, chains = _random_case(rng, multiturn=seed % 2 == 1)
    chains = [[int(x) for x in rng.integers(1, 6, size=len(c))] for c in chains]
    chains = [list(dict.fromkeys(c)) for c in chains]        # distinct keys within a chain
    tb = []
    for c in range(len(chains)):
        for t in range(turn_off[c], turn_off[c + 1]):
            tb.append(min(turn_blocks[t], len(chains[c])))
    flat, off = _flat_chains(chains)
    out = orc.simulate_episode(W, cache, spec, turn_off, tb, off, flat, dump=True)
    routes, final = brute.episode(W, cache, spec.hold_steps, spec.routes_per_step, spec.w_ov,
                                  spec.w_act, spec.w_sat, spec.cap, turn_off, tb, chains,
                                  spec.controller, spec.ctrl_w_ov, spec.ctrl_window, spec.ctrl_num,
                                  spec.ctrl_den)
    assert [r["worker"] for r in routes] == out["route_worker"].tolist()
    assert [r["overlap"] for r in routes] == out["overlap"].tolist()
    assert [k.tolist() for k in out["final_keys"]] == final


def test_cache_hit_after_route(orc):
    # re-sending a prompt right after it was routed finds it fully cached on that worker
    rng = np.random.default_rng(2)
    chains = [list(range(10 * c + 1, 10 * c + 1 + int(rng.integers(1, 8)))) for c in range(6)]
    chains = chains + chains
    flat, off = _flat_chains(chains)
    n = len(chains)
    spec = wl.EpisodeSpec(seed=0, concurrency=1, hold_steps=1, w_ov=1.0, w_act=0.0, w_sat=0.0, cap=8)
    out = orc.simulate_episode(3, 64, spec, np.arange(n + 1), [len(c) for c in chains], off, flat)
    for t in range(6, 12):
        first = out["route_worker"][t - 6]
        assert out["overlap"][t][first] == len(chains[t])
        assert out["route_worker"][t] == first


def test_single_worker_and_jsq(orc):
    w = wl.tiny_workload()
    tr = w.traces[0]
    chains = orc.trace_chains(tr)
    spec = wl.EpisodeSpec(seed=0, concurrency=8, cap=512)
    out = orc.simulate_trace(1, 256, spec, tr, chains)
    assert np.all(out["route_worker"] == 0)
    # overlap weight and overload term off: join the worker with the fewest active blocks
    spec = wl.EpisodeSpec(seed=0, concurrency=8, w_ov=0.0, w_sat=0.0, cap=512)
    out = orc.simulate_trace(4, 256, spec, tr, chains)
    A = np.zeros(4, np.int64)
    steps = {}
    for t in range(tr.n_turns):
        s = int(out["route_step"][t])
        if s not in steps:
            for r in range(t):
                if int(out["route_step"][r]) == s - spec.hold_steps:
                    A[out["route_worker"][r]] -= out["route_blocks"][r]
            steps[s] = True
        assert out["route_worker"][t] == int(np.argmin(A))
        A[out["route_worker"][t]] += out["route_blocks"][t]


def test_controller_never_fires_without_load(orc):
    w = wl.tiny_workload()
    tr = w.traces[0]
    chains = orc.trace_chains(tr)
    spec = wl.EpisodeSpec(seed=0, concurrency=8, cap=1 << 30, controller=1, ctrl_window=4)
    out = orc.simulate_trace(4, 256, spec, tr, chains)
    assert out["totals"][3] == 0 and out["totals"][4] == 0
    spec0 = wl.EpisodeSpec(seed=0, concurrency=8, cap=1 << 30)
    out0 = orc.simulate_trace(4, 256, spec0, tr, chains)
    assert np.array_equal(out["route_worker"], out0["route_worker"])


def test_multiturn_inflight_bounded(orc):
    tr = wl.multiturn_trace(3, n_conv=24, max_turns=5, add_lo=16, add_hi=64, ctx_max=300)
    chains = orc.trace_chains(tr)
    spec = wl.EpisodeSpec(seed=3, concurrency=8, cap=64)
    out = orc.simulate_trace(3, 40, spec, tr, chains)
    steps = out["route_step"]
    H = spec.hold_steps
    for s in range(int(steps.max()) + 1):
        inflight = int(np.sum((steps > s - H) & (steps <= s)))
        assert inflight <= spec.concurrency
    # every turn is routed exactly once, and a turn never precedes its predecessor
    assert sorted(out["route_turn"].tolist()) == list(range(tr.n_turns))
    pos = {int(t): i for i, t in enumerate(out["route_turn"])}
    for c in range(tr.n_conv):
        ts = list(range(int(tr.turn_off[c]), int(tr.turn_off[c + 1])))
        for a, b in zip(ts, ts[1:]):
            assert steps[pos[b]] >= steps[pos[a]] + H
