"""GPU parity of the worker-selection policies (softmax at temperature tau,
round robin, uniform random, power of two choices) against the CPU oracle:
routes, overlaps, costs and evictions bit for bit, PoA-hat within 1e-9."""
import sys

import numpy as np
import pytest

from paper_2606_17081_amd import workload as wl
from test_gpu_parity import _compare_episode, _oracle_episode, _prefix_closed_case, _run, _status_clean

pytestmark = pytest.mark.gpu
POLICIES = [(wl.POLICY_SOFTMAX, 4.0), (wl.POLICY_SOFTMAX, 0.5), (wl.POLICY_ROUND_ROBIN, 0.0),
            (wl.POLICY_RANDOM, 0.0), (wl.POLICY_P2C, 0.0), (wl.POLICY_ARGMIN, 0.0)]


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


def test_tiny_every_policy(gpu, orc):
    base = wl.tiny_workload()
    eps = [wl.EpisodeSpec(seed=0, concurrency=8, cap=512, policy=p, tau=tau) for p, tau in POLICIES]
    w = wl.Workload("tiny-policies", W=base.W, cache_blocks=base.cache_blocks, traces=base.traces, episodes=eps)
    for mode in (0, 1):
        say("tiny, every policy, probe mode", mode)
        r = _run(gpu, w, mode=mode)
        for e, sp in enumerate(eps):
            o = _oracle_episode(orc, w, sp, {})
            _compare_episode(r.episode_results(e), o, w.W, window=sp.concurrency, label=f"policy {sp.policy}")


def test_random_small_episodes_mixed_policies(gpu, orc):
    """48 small episodes with every policy, heavy eviction and multi-turn, in one launch."""
    rng = np.random.default_rng(91)
    W, cache = 5, 30
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
        p, tau = POLICIES[seed % len(POLICIES)]
        specs.append(wl.EpisodeSpec(seed=seed, concurrency=H * rps, hold_steps=H, w_ov=float(rng.choice([0.25, 1.0])),
                                    w_act=0.5, w_sat=float(rng.choice([0.0, 4.0])), cap=int(rng.integers(1, 200)),
                                    controller=int(rng.integers(0, 2)), ctrl_window=int(rng.integers(1, 6)),
                                    policy=p, tau=tau))
    work = wl.Workload("random-policies", W=W, cache_blocks=cache, traces=traces, episodes=specs)
    flat = np.concatenate([all_chains[s] for s in sorted(traces)])
    for mode in (0, 1):
        say("48 random episodes with policies, probe mode", mode)
        r = _run(gpu, work, mode=mode, chains=flat)
        for e, sp in enumerate(specs):
            tr = traces[sp.seed]
            o = orc.simulate_episode(W, cache, sp, tr.turn_off, tr.turn_blocks, tr.chain_off, all_chains[sp.seed])
            _compare_episode(r.episode_results(e), o, W, window=sp.concurrency, label=f"episode {e} policy {sp.policy}")


def test_policy_sweep_full_size_sampled(gpu, orc):
    """The 1P/5D-shaped traces under every policy (2 seeds x 5 C x 5 policies) in one launch;
    one sampled episode per policy against the oracle; PoA-hat finite."""
    w = wl.policy_workload(seeds=range(2))
    say("running", len(w.episodes), "policy episodes")
    r = _run(gpu, w)
    cache = {}
    for k in range(len(wl.POLICY_SWEEP)):
        e = k * 10 + (k * 3) % 10
        sp = r.episodes[e]
        say("oracle episode", e, "policy", sp.policy, "C", sp.concurrency, "seed", sp.seed)
        o = _oracle_episode(orc, w, sp, cache)
        _compare_episode(r.episode_results(e), o, w.W, window=sp.concurrency, label=f"policy e{e}")
    poa = r.poa_hat.cpu().numpy()[: len(r.episodes)]
    assert np.all(np.isfinite(poa)) and np.all(poa > 0)


def test_bad_policy_parameters_flagged(gpu):
    torch, rk = gpu
    base = wl.tiny_workload()
    from paper_2606_17081_amd.episodes import EpisodeRunner
    for p, tau in ((9, 0.0), (wl.POLICY_SOFTMAX, 0.0), (wl.POLICY_SOFTMAX, -1.0)):
        sp = wl.EpisodeSpec(seed=0, concurrency=8, cap=512, policy=p, tau=tau)
        r = EpisodeRunner(base, [sp])
        r.simulate()
        torch.cuda.synchronize()
        bits = rk.device_status(reset=True)
        assert bits & 0x40, (p, tau, bits)
    # negative or NaN weights (the argmin orders costs by their bits, which needs costs >= 0)
    for field, value in (("w_ov", -1.0), ("w_act", -0.5), ("w_sat", float("nan")), ("ctrl_w_ov", -0.25)):
        sp = wl.EpisodeSpec(seed=0, concurrency=8, cap=512, **{field: value})
        r = EpisodeRunner(base, [sp])
        r.simulate()
        torch.cuda.synchronize()
        assert rk.device_status(reset=True) & 0x40, field
        assert int(r.totals[0, 2]) == 0, field          # outputs left unwritten
    # a policy that draws, launched without draws
    sp = wl.EpisodeSpec(seed=0, concurrency=8, cap=512, policy=wl.POLICY_RANDOM)
    r = EpisodeRunner(base, [sp])
    r.batch.route_rand = None
    r.simulate()
    torch.cuda.synchronize()
    assert rk.device_status(reset=True) & 0x40
    _status_clean(rk)


def _regime_compare(g, o, label):
    assert np.array_equal(g["route_regime"], o["route_regime"]), label


def test_regime_controller_small_episodes(gpu, orc):
    """40 small episodes under the regime controller, with a latency model that saturates at a
    few requests so that every regime is visited, in one launch."""
    rng = np.random.default_rng(123)
    W, cache = 4, 40
    reg = dict(wl.REGIME_PARAMS, a=0.2, b=0.0, d=0.5, n_sat=4, theta1=0.4, theta2=0.9, eps=0.1, k=2,
               tau=(0.0, 0.7, 3.0), w_ov=(1.0, 0.5, 0.1))
    traces, specs, all_chains = {}, [], {}
    for seed in range(40):
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
        specs.append(wl.EpisodeSpec(seed=seed, concurrency=H * rps, hold_steps=H, w_act=0.5,
                                    w_sat=float(rng.choice([0.0, 4.0])), cap=int(rng.integers(1, 200)), controller=2))
    work = wl.Workload("regime", W=W, cache_blocks=cache, traces=traces, episodes=specs, regime=reg)
    flat = np.concatenate([all_chains[s] for s in sorted(traces)])
    seen = set()
    for mode in (0, 1):
        say("40 regime-controller episodes, probe mode", mode)
        r = _run(gpu, work, mode=mode, chains=flat)
        for e, sp in enumerate(specs):
            tr = traces[sp.seed]
            o = orc.simulate_episode(W, cache, sp, tr.turn_off, tr.turn_blocks, tr.chain_off, all_chains[sp.seed],
                                     regime=reg)
            g = r.episode_results(e)
            _compare_episode(g, o, W, window=sp.concurrency, label=f"regime episode {e}")
            _regime_compare(g, o, f"regime episode {e}")
            seen |= set(o["route_regime"].tolist())
    assert seen == {0, 1, 2}


def test_regime_controller_sweep_sampled(gpu, orc):
    """The 1P/5D-shaped traces (4 seeds x 5 C) under the regime controller with the paper's
    parameters; three sampled episodes against the oracle."""
    base = wl.sweep70b_workload(seeds=range(4))
    eps = [wl.EpisodeSpec(seed=sp.seed, concurrency=sp.concurrency, cap=sp.cap, controller=2) for sp in base.episodes]
    w = wl.Workload("sweep-regime", W=base.W, cache_blocks=base.cache_blocks, traces=base.traces, episodes=eps)
    r = _run(gpu, w)
    cache = {}
    for e in (1, 9, 19):
        sp = r.episodes[e]
        say("oracle regime episode", e, "C", sp.concurrency)
        o = _oracle_episode(orc, w, sp, cache)
        g = r.episode_results(e)
        _compare_episode(g, o, w.W, window=sp.concurrency, label=f"sweep regime e{e}")
        _regime_compare(g, o, f"sweep regime e{e}")
