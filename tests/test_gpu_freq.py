"""GPU parity of frequency eviction (the KV block manager's policy: frequency 1
on insert, doubled per hit up to 2^20, minus 1 per time-decay step with a floor
of 1; least frequent block first, least recently used among equals) against the
CPU oracle: routes, overlaps, costs, eviction counts and digests bit for bit,
PoA-hat within 1e-9."""
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


def _freq(sp, T):
    return wl.EpisodeSpec(**{**sp.__dict__, "evict_policy": wl.EVICT_FREQ, "decay_steps": T})


def test_tiny_under_pressure(gpu, orc):
    """The tiny trace with 64-block caches, decay every 1, 4 and 1000 steps, next to LRU."""
    base = wl.tiny_workload()
    sp0 = base.episodes[0]
    eps = [sp0] + [_freq(sp0, T) for T in (1, 4, 1000)]
    w = wl.Workload("tiny-freq", W=base.W, cache_blocks=64, traces=base.traces, episodes=eps)
    for mode in (0, 1):
        say("tiny, frequency eviction, probe mode", mode)
        r = _run(gpu, w, mode=mode)
        for e, sp in enumerate(eps):
            o = _oracle_episode(orc, w, sp, {})
            assert o["totals"][1] > 0
            _compare_episode(r.episode_results(e), o, w.W, window=sp.concurrency, label=f"T {sp.decay_steps}")


def test_random_small_episodes(gpu, orc):
    """48 small episodes (prefix-closed keys, heavy eviction, multi-turn), LRU and frequency
    eviction with decay periods 1..8, in one launch, both probe modes."""
    rng = np.random.default_rng(313)
    W, cache = 4, 28
    traces, specs, all_chains = {}, [], {}
    for seed in range(48):
        chains, turn_off, turn_blocks = _prefix_closed_case(rng, W, cache, multiturn=seed % 2 == 1)
        lens = np.array([len(c) for c in chains], np.int32)
        chain_off = np.zeros(len(chains) + 1, np.int64)
        np.cumsum(lens, out=chain_off[1:])
        traces[seed] = wl.Trace(seed=seed, tokens=np.zeros(16, np.int32), tok_off=chain_off * 0,
                                chain_blocks=lens, chain_off=chain_off, turn_off=turn_off,
                                turn_blocks=turn_blocks, group=np.zeros(len(chains), np.int32),
                                shared=np.zeros(len(chains), np.int32))
        all_chains[seed] = np.array([k for c in chains for k in c], np.uint64)
        H, rps = int(rng.integers(1, 5)), int(rng.integers(1, 6))
        T = int(rng.integers(1, 9))
        specs.append(wl.EpisodeSpec(seed=seed, concurrency=H * rps, hold_steps=H, w_ov=float(rng.choice([0.25, 1.0])),
                                    w_act=0.5, w_sat=float(rng.choice([0.0, 4.0])), cap=int(rng.integers(1, 200)),
                                    controller=int(rng.integers(0, 2)), ctrl_window=int(rng.integers(1, 6)),
                                    evict_policy=wl.EVICT_FREQ if seed % 4 else wl.EVICT_LRU,
                                    decay_steps=T if seed % 4 else 0))
    work = wl.Workload("random-freq", W=W, cache_blocks=cache, traces=traces, episodes=specs)
    flat = np.concatenate([all_chains[s] for s in sorted(traces)])
    differs = 0
    for mode in (0, 1):
        say("48 random episodes, frequency eviction, probe mode", mode)
        r = _run(gpu, work, mode=mode, chains=flat)
        for e, sp in enumerate(specs):
            tr = traces[sp.seed]
            o = orc.simulate_episode(W, cache, sp, tr.turn_off, tr.turn_blocks, tr.chain_off, all_chains[sp.seed])
            _compare_episode(r.episode_results(e), o, W, window=sp.concurrency,
                             label=f"episode {e} T {sp.decay_steps}")
            if mode == 0 and sp.evict_policy == wl.EVICT_FREQ:
                sp_lru = wl.EpisodeSpec(**{**sp.__dict__, "evict_policy": wl.EVICT_LRU, "decay_steps": 0})
                lru = orc.simulate_episode(W, cache, sp_lru, tr.turn_off, tr.turn_blocks, tr.chain_off,
                                           all_chains[sp.seed])
                differs += int(not np.array_equal(lru["evict_digest"], o["evict_digest"]))
    assert differs > 0         # the cases do tell the two policies apart


def test_multiturn_full_size(gpu, orc):
    """Long-context multi-turn episodes at full size (512 conversations, 16,384-block caches)
    under frequency eviction with decay every 4 and 64 steps."""
    say("generating 4 multi-turn traces")
    base = wl.multiturn_workload(seeds=range(4))
    eps = [_freq(sp, T) for sp in base.episodes for T in (4, 64)]
    w = wl.Workload("multiturn-freq", W=base.W, cache_blocks=base.cache_blocks, traces=base.traces, episodes=eps)
    say("running", len(eps), "episodes on the GPU")
    r = _run(gpu, w)
    cache = {}
    for e in (0, 3, 6):
        say("oracle episode", e, "T", eps[e].decay_steps)
        o = _oracle_episode(orc, w, eps[e], cache)
        assert o["totals"][1] > 0
        _compare_episode(r.episode_results(e), o, w.W, window=256, label=f"multiturn freq e{e}")


def test_sweep_shape_with_decay(gpu, orc):
    """1P/5D-shaped traces with small caches (heavy pressure) under frequency eviction."""
    base = wl.sweep70b_workload(seeds=range(2), concurrency=(32, 256))
    eps = [_freq(sp, 8) for sp in base.episodes]
    w = wl.Workload("sweep-freq", W=base.W, cache_blocks=2048, traces=base.traces, episodes=eps)
    say("running", len(eps), "sweep-shaped episodes with 2,048-block caches")
    r = _run(gpu, w)
    cache = {}
    for e in range(len(eps)):
        o = _oracle_episode(orc, w, eps[e], cache)
        assert o["totals"][1] > 0
        _compare_episode(r.episode_results(e), o, w.W, window=eps[e].concurrency, label=f"sweep freq e{e}")


def test_eviction_extremes(gpu, orc):
    """Caches smaller than one prompt, single worker, decay every step."""
    tr = wl.tiny_trace(4)
    for W, cache in [(4, 1), (2, 7), (1, 40)]:
        for T in (1, 3):
            say("frequency eviction extremes W", W, "cache", cache, "T", T)
            spec = wl.EpisodeSpec(seed=4, concurrency=8, cap=64, evict_policy=wl.EVICT_FREQ, decay_steps=T)
            work = wl.Workload("x", W=W, cache_blocks=cache, traces={4: tr}, episodes=[spec])
            for mode in (0, 1):
                r = _run(gpu, work, mode=mode)
                o = orc.simulate_trace(W, cache, spec, tr)
                _compare_episode(r.episode_results(0), o, W, window=8, label=f"W{W} cache{cache} T{T}")


def test_bad_parameters_flagged(gpu):
    torch, rk = gpu
    from paper_2606_17081_amd.episodes import EpisodeRunner
    base = wl.tiny_workload()
    for kw in (dict(evict_policy=2, decay_steps=1), dict(evict_policy=wl.EVICT_FREQ, decay_steps=0)):
        sp = wl.EpisodeSpec(**{**base.episodes[0].__dict__, **kw})
        r = EpisodeRunner(base, [sp])
        r.simulate()
        torch.cuda.synchronize()
        st = rk.device_status(reset=True)
        assert st & 0x40, (kw, st)          # bad parameters
    _status_clean(rk)
