"""GPU parity of memory tiers (Section 4.2, Eq. kv-cost: a worker's k1 most
recently used blocks in G1, the next k2 in G2, the rest in G3; the routing
cost charges a cached block by its tier) against the CPU oracle: routes,
overlaps, tier overlaps, costs and evictions bit for bit, PoA-hat within 1e-9."""
import sys

import numpy as np
import pytest

from paper_2606_17081_amd import workload as wl
from test_gpu_parity import _compare_episode, _oracle_episode, _prefix_closed_case, _run, _status_clean

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2606_17081_amd import rkroute as rk
    rk.lib()
    assert rk.device_status(reset=True) == 0
    return torch, rk


def _tiered(sp, k1, k2, tw=(0.0, 0.25, 0.5)):
    return wl.EpisodeSpec(**{**sp.__dict__, "tier_g1": k1, "tier_g2": k2, "tier_w": tuple(tw)})


def _compare(g, o, W, window, label):
    assert np.array_equal(g["tier_overlap"], o["tier_overlap"]), label
    _compare_episode(g, o, W, window=window, label=label)


def _chains_workload(name, W, cache, cases, specs):
    """Workload over explicit block-key chains (one trace per case)."""
    traces, flat = {}, []
    for seed, (chains, turn_off, turn_blocks) in enumerate(cases):
        lens = np.array([len(c) for c in chains], np.int32)
        chain_off = np.zeros(len(chains) + 1, np.int64)
        np.cumsum(lens, out=chain_off[1:])
        traces[seed] = wl.Trace(seed=seed, tokens=np.zeros(16, np.int32), tok_off=chain_off * 0,
                                chain_blocks=lens, chain_off=chain_off, turn_off=np.asarray(turn_off, np.int64),
                                turn_blocks=np.asarray(turn_blocks, np.int32), group=np.zeros(len(chains), np.int32),
                                shared=np.zeros(len(chains), np.int32))
        flat.append(np.array([k for c in chains for k in c], np.uint64))
    return wl.Workload(name, W=W, cache_blocks=cache, traces=traces, episodes=specs), np.concatenate(flat)


def test_hand_worked(gpu, orc):
    # one worker, 6-block cache, G1 = G2 = G3 = 2 blocks: (o1, o12) = (0, 2) then (0, 1)
    chains = [[1, 2], [3, 4], [1, 2, 7], [3, 4, 8]]
    spec = wl.EpisodeSpec(seed=0, concurrency=1, hold_steps=1, w_ov=1.0, w_act=0.0, w_sat=0.0, cap=1 << 20,
                          tier_g1=2, tier_g2=2, tier_w=(0.0, 0.25, 0.5))
    w, flat = _chains_workload("hand", 1, 6, [(chains, [0, 1, 2, 3, 4], [2, 2, 3, 3])], [spec])
    for mode in (0, 1):
        r = _run(gpu, w, mode=mode, chains=flat)
        g = r.episode_results(0)
        assert g["tier_overlap"][:, 0].tolist() == [[0, 0], [0, 0], [0, 2], [0, 1]]
        assert g["cost"][:, 0].tolist() == [2.0, 2.0, 1.5, 1.75]


def _straddle_case(rng):
    n_conv = int(rng.integers(8, 24))
    chains, turn_blocks, turn_off, nxt = [], [], [0], 1
    shared = [list(range(100000 * (g + 1), 100000 * (g + 1) + 40)) for g in range(4)]
    for _ in range(n_conv):
        g = int(rng.integers(0, 4))
        head = shared[g][: int(rng.integers(2, 40))]
        L = len(head) + int(rng.integers(1, 60))
        ch = head + list(range(nxt, nxt + L - len(head)))
        nxt += L
        chains.append(ch)
        tb = sorted(int(x) for x in rng.integers(len(head), L + 1, size=int(rng.integers(1, 4))))
        turn_blocks.extend(tb)
        turn_off.append(len(turn_blocks))
    return chains, turn_off, turn_blocks


def test_random_small_episodes(gpu, orc):
    """40 episodes with tiers (multi-turn, shared heads, eviction), both probe modes."""
    rng = np.random.default_rng(4242)
    W, cache = 3, 160
    cases, specs = [], []
    for seed in range(40):
        cases.append(_straddle_case(rng) if seed % 2 else _prefix_closed_case(rng, W, cache, multiturn=True))
        H, rps = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        k1 = int(rng.integers(1, 60))
        k2 = int(rng.integers(0, cache - k1 + 1)) if seed % 3 else int(rng.integers(1, 40))
        tw = [float(x) for x in rng.choice([0.0, 0.125, 0.3, 0.5, 1.0], size=3)]
        specs.append(wl.EpisodeSpec(seed=seed, concurrency=H * rps, hold_steps=H, w_ov=1.0,
                                    w_act=float(rng.choice([0.0, 0.5])), w_sat=float(rng.choice([0.0, 4.0])),
                                    cap=int(rng.integers(8, 300)), tier_g1=k1, tier_g2=k2, tier_w=tuple(tw)))
    w, flat = _chains_workload("tiers", W, cache, cases, specs)
    straddles = 0
    for mode in (0, 1):
        say("40 episodes with memory tiers, probe mode", mode)
        r = _run(gpu, w, mode=mode, chains=flat)
        for e, sp in enumerate(specs):
            tr = w.traces[sp.seed]
            keys = np.array([k for c in cases[sp.seed][0] for k in c], np.uint64)
            o = orc.simulate_episode(W, cache, sp, tr.turn_off, tr.turn_blocks, tr.chain_off, keys)
            _compare(r.episode_results(e), o, W, sp.concurrency, f"episode {e} mode {mode}")
            t = o["tier_overlap"]
            straddles += int(((0 < t[..., 0]) & (t[..., 0] < t[..., 1]) & (t[..., 1] < o["overlap"])).sum())
    assert straddles > 0


def test_whole_cache_g1_matches_untiered(gpu):
    """G1 = the whole cache at weight 0 gives the untiered episode, bit for bit."""
    base = wl.tiny_workload()
    sp = base.episodes[0]
    w = wl.Workload("tiny-tiers", W=base.W, cache_blocks=64, traces=base.traces,
                    episodes=[sp, _tiered(sp, 64, 0, (0.0, 0.9, 0.9))])
    r = _run(gpu, w)
    a, b = r.episode_results(0), r.episode_results(1)
    for k in ("route_worker", "overlap", "evict_count", "evict_digest", "totals"):
        assert np.array_equal(a[k], b[k]), k
    assert np.array_equal(a["cost"].view(np.uint32), b["cost"].view(np.uint32))


def test_multiturn_shape(gpu, orc):
    """Multi-turn traces (64 conversations, 32 workers, 2,048-block caches, heavy eviction) with
    G1 = 512 and G2 = 512 blocks."""
    base = wl.multiturn_workload(seeds=range(2), n_conv=64)
    eps = [_tiered(sp, 512, 512) for sp in base.episodes]
    w = wl.Workload("multiturn-tiers", W=base.W, cache_blocks=2048, traces=base.traces, episodes=eps)
    say("running", len(eps), "multi-turn episodes with tiers")
    r = _run(gpu, w)
    cache = {}
    for e in range(len(eps)):
        o = _oracle_episode(orc, w, eps[e], cache)
        assert o["totals"][1] > 0
        _compare(r.episode_results(e), o, w.W, 256, f"multiturn tiers e{e}")


def test_sweep_shape(gpu, orc):
    """A 1P/5D-shaped trace (4,096 requests, 6 workers, 65,536-block caches) with G1 = 4,096 and
    G2 = 8,192 blocks, at C = 64."""
    base = wl.sweep70b_workload(seeds=range(1), concurrency=(64,))
    eps = [_tiered(sp, 4096, 8192) for sp in base.episodes]
    w = wl.Workload("sweep-tiers", W=base.W, cache_blocks=base.cache_blocks, traces=base.traces, episodes=eps)
    r = _run(gpu, w)
    o = _oracle_episode(orc, w, eps[0], {})
    _compare(r.episode_results(0), o, w.W, 64, "sweep tiers")
    t = o["tier_overlap"]
    assert np.any(t[..., 0] < o["overlap"])


def test_bad_parameters_flagged(gpu):
    torch, rk = gpu
    from paper_2606_17081_amd.episodes import EpisodeRunner
    base = wl.tiny_workload()
    for kw in (dict(tier_g1=200, tier_g2=100), dict(tier_g1=1, tier_g2=-1),
               dict(tier_g1=8, evict_policy=wl.EVICT_FREQ, decay_steps=2), dict(tier_g1=8, tier_w=(0.0, -1.0, 0.0))):
        sp = wl.EpisodeSpec(**{**base.episodes[0].__dict__, **kw})
        r = EpisodeRunner(base, [sp])
        r.simulate()
        torch.cuda.synchronize()
        st = rk.device_status(reset=True)
        assert st & 0x40, (kw, st)          # bad parameters
    # tiers asked for by an episode of a launch that did not reserve them
    sp = wl.EpisodeSpec(**{**base.episodes[0].__dict__, "tier_g1": 8})
    r = EpisodeRunner(base, [sp])
    r.batch.tiers = 0
    r.simulate()
    torch.cuda.synchronize()
    assert rk.device_status(reset=True) & 0x40
    _status_clean(rk)
