"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Integer results (hashes, overlaps, routes, steps, evictions, digests, argmins)
must match bit for bit; fp32 costs must match bit for bit as well (both sides
evaluate the same IEEE operations in the same order, which is tighter than the
1e-5 relative bound the method needs); PoA sums use a 1e-9 relative bound
(fp64 sums of identical fp32 terms, possibly of a different optimal
assignment).  Large workloads run at their full per-episode sizes in the same
launch configuration as the benchmark and are checked on sampled episodes.
"""
import json
import os
import sys

import numpy as np
import pytest

from paper_2606_17081_amd import workload as wl

pytestmark = pytest.mark.gpu
REL = 1e-9
GOLD = os.path.join(os.path.dirname(__file__), "golden", "episode_hand.json")


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


def _status_clean(rk):
    bits = rk.device_status(reset=True)
    assert bits == 0, [v for k, v in rk.DEV_BITS.items() if bits & k]


def _compare_episode(g, o, W, poa_params=wl.POA_PARAMS, window=None, label=""):
    n = len(o["route_worker"])
    assert len(g["route_worker"]) == n, label
    for k in ("route_turn", "route_worker", "route_step", "route_blocks", "evict_count", "evict_digest",
              "last_hash"):
        bad = np.nonzero(np.asarray(g[k]) != np.asarray(o[k]))[0]
        assert bad.size == 0, f"{label} {k} differs first at route {bad[:5]}"
    assert np.array_equal(g["overlap"], o["overlap"]), label
    if "cost" in g:
        assert np.array_equal(g["cost"].view(np.uint32), o["cost"].view(np.uint32)), label
    assert np.array_equal(g["totals"], o["totals"]), (label, g["totals"], o["totals"])
    if window is not None:
        from oracle import oracle as O
        ref = O.episode_poa(o, W, window, poa_params)
        np.testing.assert_allclose(g["selfish"], ref["selfish"], rtol=REL)
        np.testing.assert_allclose(g["coordinated"], ref["coordinated"], rtol=REL)
        assert g["poa_hat"] == pytest.approx(ref["poa_hat"], rel=REL)


# ------------------------------------------------------------------ hashing

def test_hash_chains_parity(gpu, orc):
    torch, rk = gpu
    traces = [wl.tiny_trace(0), wl.sweep70b_trace(5), wl.multiturn_trace(2, n_conv=64)]
    for tr in traces:
        say("hash parity, seed", tr.seed, "sequences", tr.n_conv, "blocks", tr.n_blocks)
        up = rk.to_device
        ch = rk.hash_chains(up(tr.tokens), up(tr.tok_off), up(tr.chain_off))
        torch.cuda.synchronize()
        got = rk.to_host_u64(ch[: tr.n_blocks])
        assert np.array_equal(got, orc.trace_chains(tr))
    # empty sequences, a trailing partial block, zero sequences
    toks = np.arange(16 * 3 + 5, dtype=np.int32)
    tok_off = np.array([0, 0, 16 * 3 + 5], np.int64)
    chain_off = np.array([0, 0, 3], np.int64)
    ch = rk.hash_chains(torch.from_numpy(toks).cuda(), torch.from_numpy(tok_off).cuda(),
                        torch.from_numpy(chain_off).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(rk.to_host_u64(ch[:3]), orc.hash_chains(toks, tok_off, [0, 3], chain_off))
    _status_clean(rk)


def test_hash_short_tokens_flagged(gpu):
    torch, rk = gpu
    toks = torch.zeros(20, dtype=torch.int32, device="cuda")
    ch = rk.hash_chains(toks, torch.tensor([0, 20], device="cuda"), torch.tensor([0, 2], device="cuda"))
    torch.cuda.synchronize()
    assert rk.device_status(reset=True) & 0x2
    assert int(rk.to_host_u64(ch[1:2])[0]) == 0


# ------------------------------------------------------------------ snapshot scoring

def _score(rk, torch, inst, mode, tables=None):
    up = rk.to_device
    if tables is None:
        tables = rk.table_build(up(inst.keys), inst.key_off, inst.log2_slots)
    ov, co, am = rk.route_score_batch(up(inst.chains), up(inst.chain_off), tables, inst.log2_slots,
                                      up(inst.active), inst.w_ov, inst.w_act, inst.w_sat, inst.cap,
                                      probe_mode=mode)
    torch.cuda.synchronize()
    return ov.cpu().numpy(), co.cpu().numpy(), am.cpu().numpy(), tables


@pytest.mark.parametrize("W", [64, 5, 70])
def test_score_small_both_modes(gpu, orc, W):
    torch, rk = gpu
    inst = wl.scoring_instance(seed=W, B=1500, W=W, log2_slots=11, len_lo=1, len_hi=70)
    ref = orc.score_batch(inst.chains, inst.chain_off, inst.keys, inst.key_off, inst.active,
                          inst.w_ov, inst.w_act, inst.w_sat, inst.cap)
    for mode in (rk.RK_PROBE_PREFIX, rk.RK_PROBE_SCAN):
        say("score small W", W, "mode", mode)
        ov, co, am, _ = _score(rk, torch, inst, mode)
        assert np.array_equal(ov, ref[0])
        assert np.array_equal(co.view(np.uint32), ref[1].view(np.uint32))
        assert np.array_equal(am, ref[2])
    _status_clean(rk)


def test_score_scan_mode_arbitrary_tables(gpu, orc):
    # keys from a tiny alphabet: tables are not prefix-closed along chains
    torch, rk = gpu
    rng = np.random.default_rng(3)
    W, B = 9, 800
    L = rng.integers(0, 40, size=B)
    chain_off = np.zeros(B + 1, np.int64)
    np.cumsum(L, out=chain_off[1:])
    chains = rng.integers(1, 30, size=int(chain_off[-1])).astype(np.uint64)
    keys = [np.unique(rng.integers(1, 30, size=int(rng.integers(0, 25)))).astype(np.uint64) for _ in range(W)]
    key_off = np.zeros(W + 1, np.int64)
    np.cumsum([k.size for k in keys], out=key_off[1:])
    inst = wl.ScoringInstance(W=W, B=B, keys=np.concatenate(keys), key_off=key_off, chains=chains,
                              chain_off=chain_off, active=rng.integers(0, 50, W).astype(np.int32), cap=16,
                              log2_slots=6)
    ref = orc.score_batch(inst.chains, inst.chain_off, inst.keys, inst.key_off, inst.active,
                          inst.w_ov, inst.w_act, inst.w_sat, inst.cap)
    ov, co, am, _ = _score(rk, torch, inst, rk.RK_PROBE_SCAN)
    assert np.array_equal(ov, ref[0]) and np.array_equal(am, ref[2])
    assert np.array_equal(co.view(np.uint32), ref[1].view(np.uint32))
    _status_clean(rk)


def test_score_full_size_sampled(gpu, orc):
    """65,536 requests x 64 workers, 2^20-slot tables; 300 sampled requests vs the oracle."""
    torch, rk = gpu
    say("generating the 65,536 x 64 scoring instance")
    inst = wl.scoring_instance(seed=0)
    say("scoring on the GPU")
    ov, co, am, tables = _score(rk, torch, inst, rk.RK_PROBE_PREFIX)
    _status_clean(rk)
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([[0, inst.B - 1], rng.integers(0, inst.B, 298)]))
    say("oracle on", rows.size, "sampled requests")
    r_ov, r_co, r_am = orc.score_batch(inst.chains, inst.chain_off, inst.keys, inst.key_off, inst.active,
                                       inst.w_ov, inst.w_act, inst.w_sat, inst.cap, rows=rows)
    assert np.array_equal(ov[rows], r_ov)
    assert np.array_equal(co[rows].view(np.uint32), r_co.view(np.uint32))
    assert np.array_equal(am[rows], r_am)
    # properties over every request: overlap within the prompt, argmin is the first minimum
    P = np.diff(inst.chain_off)
    assert np.all(ov >= 0) and np.all(ov <= P[:, None])
    assert np.array_equal(am, np.argmin(co, axis=1))
    # the scan mode agrees on the same tables (prefix-closed by construction)
    ov2, _, am2, _ = _score(rk, torch, inst, rk.RK_PROBE_SCAN, tables=tables)
    assert np.array_equal(ov2, ov) and np.array_equal(am2, am)
    _status_clean(rk)


def test_score_empty_and_degenerate(gpu, orc):
    torch, rk = gpu
    inst = wl.scoring_instance(seed=9, B=40, W=3, log2_slots=6, len_lo=1, len_hi=8)
    n4 = int(inst.chain_off[5] - inst.chain_off[4])                       # make request 4 empty
    inst.chains = np.delete(inst.chains, np.s_[inst.chain_off[4]:inst.chain_off[5]])
    inst.chain_off[5:] -= n4
    ref = orc.score_batch(inst.chains, inst.chain_off, inst.keys, inst.key_off, inst.active,
                          inst.w_ov, inst.w_act, inst.w_sat, inst.cap)
    ov, co, am, _ = _score(rk, torch, inst, rk.RK_PROBE_PREFIX)
    assert np.array_equal(ov, ref[0]) and np.array_equal(am, ref[2])
    assert np.array_equal(co.view(np.uint32), ref[1].view(np.uint32))
    z = torch.zeros(1, dtype=torch.int64, device="cuda")
    o, c, a = rk.route_score_batch(torch.zeros(1, dtype=torch.int64, device="cuda"), z,
                                   torch.zeros(3 << 6, dtype=torch.int64, device="cuda"), 6,
                                   torch.zeros(3, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    assert a.numel() == 0
    _status_clean(rk)


# ------------------------------------------------------------------ episodes

def _run(gpu, workload, episodes=None, mode=0, chains=None):
    torch, rk = gpu
    from paper_2606_17081_amd.episodes import EpisodeRunner
    r = EpisodeRunner(workload, episodes, probe_mode=mode, chains=chains)
    r.step()
    torch.cuda.synchronize()
    _status_clean(rk)
    return r


def _oracle_episode(orc, workload, spec, chains_cache):
    tr = workload.traces[spec.seed]
    if spec.seed not in chains_cache:
        chains_cache[spec.seed] = orc.trace_chains(tr)
    return orc.simulate_trace(workload.W, workload.cache_blocks, spec, tr, chains_cache[spec.seed])


@pytest.mark.parametrize("mode", [0, 1])
def test_tiny_episode_parity(gpu, orc, mode):
    w = wl.tiny_workload()
    say("tiny episode, probe mode", mode)
    r = _run(gpu, w, mode=mode)
    o = _oracle_episode(orc, w, w.episodes[0], {})
    _compare_episode(r.episode_results(0), o, w.W, window=w.episodes[0].concurrency, label="tiny")


def test_hand_fixtures_gpu(gpu):
    with open(GOLD) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        say("hand fixture", case["name"])
        chains = case["chains"]
        n = len(chains)
        lens = np.array([len(c) for c in chains], np.int32)
        chain_off = np.zeros(n + 1, np.int64)
        np.cumsum(lens, out=chain_off[1:])
        tok_off = chain_off * 16
        tr = wl.Trace(seed=0, tokens=np.zeros(int(tok_off[-1]) or 16, np.int32), tok_off=tok_off,
                      chain_blocks=lens, chain_off=chain_off, turn_off=np.array(case["turn_off"], np.int64),
                      turn_blocks=np.array(case["turn_blocks"], np.int32), group=np.zeros(n, np.int32),
                      shared=np.zeros(n, np.int32))
        spec = wl.EpisodeSpec(seed=0, concurrency=case["routes_per_step"] * case["H"], hold_steps=case["H"],
                              w_ov=case["w_ov"], w_act=case["w_act"], w_sat=case["w_sat"], cap=case["cap"],
                              controller=case["controller"], ctrl_w_ov=case.get("ctrl_w_ov", 0.25),
                              ctrl_window=case.get("ctrl_window", 128), ctrl_num=case.get("ctrl_num", 9),
                              ctrl_den=case.get("ctrl_den", 10))
        work = wl.Workload("hand", W=case["W"], cache_blocks=case["cache_blocks"], traces={0: tr}, episodes=[spec])
        flat_chains = np.array([k for c in chains for k in c], np.uint64)
        for mode in (0, 1):
            g = _run(gpu, work, mode=mode, chains=flat_chains).episode_results(0)
            ex = case["expect"]
            assert g["route_turn"].tolist() == ex["route_turn"]
            assert g["route_worker"].tolist() == ex["route_worker"]
            assert g["route_step"].tolist() == ex["route_step"]
            assert g["overlap"].tolist() == ex["overlap"]
            assert g["cost"].tolist() == ex["cost"]
            assert g["evict_count"].tolist() == ex["evict_count"]
            assert g["last_hash"].tolist() == ex["last_hash"]
            t = g["totals"]
            assert t[0] == ex["totals"]["prefill"] and t[1] == ex["totals"]["evicted"]
            assert t[5] == ex["totals"]["steps"] and t[7] == ex["totals"]["cached"]


def _prefix_closed_case(rng, W, cache, multiturn):
    n_conv = int(rng.integers(1, 40))
    chains, turn_blocks, turn_off = [], [], [0]
    prefix_id = {}
    for _ in range(n_conv):
        L = int(rng.integers(1, 150))
        path = tuple(int(x) for x in rng.integers(0, 2 if L < 20 else 4, size=L))
        chains.append([prefix_id.setdefault(path[:k], len(prefix_id) + 1) for k in range(1, L + 1)])
        tb = sorted(int(x) for x in rng.integers(0, L + 1, size=int(rng.integers(1, 4)))) if multiturn else [L]
        turn_blocks.extend(tb)
        turn_off.append(len(turn_blocks))
    return chains, np.array(turn_off, np.int64), np.array(turn_blocks, np.int32)


def test_random_small_episodes_batched(gpu, orc):
    """60 small episodes (prefix-closed keys, heavy eviction, controller, multi-turn) in one launch."""
    torch, rk = gpu
    rng = np.random.default_rng(77)
    W, cache = 3, 24
    traces, specs, all_chains = {}, [], {}
    for seed in range(60):
        chains, turn_off, turn_blocks = _prefix_closed_case(rng, W, cache, multiturn=seed % 2 == 1)
        lens = np.array([len(c) for c in chains], np.int32)
        chain_off = np.zeros(len(chains) + 1, np.int64)
        np.cumsum(lens, out=chain_off[1:])
        traces[seed] = wl.Trace(seed=seed, tokens=np.zeros(16, np.int32), tok_off=chain_off * 0,
                                chain_blocks=lens, chain_off=chain_off, turn_off=turn_off,
                                turn_blocks=turn_blocks, group=np.zeros(len(chains), np.int32),
                                shared=np.zeros(len(chains), np.int32))
        all_chains[seed] = np.array([k for c in chains for k in c], np.uint64)
        H = int(rng.integers(1, 5))
        rps = int(rng.integers(1, 6))
        specs.append(wl.EpisodeSpec(seed=seed, concurrency=H * rps, hold_steps=H,
                                    w_ov=float(rng.choice([0.0, 0.25, 1.0, 2.0])),
                                    w_act=float(rng.choice([0.0, 0.5, 1.0])), w_sat=float(rng.choice([0.0, 4.0])),
                                    cap=int(rng.integers(1, 200)), controller=int(rng.integers(0, 2)),
                                    ctrl_window=int(rng.integers(1, 6)), ctrl_num=int(rng.integers(0, 10))))
    work = wl.Workload("random", W=W, cache_blocks=cache, traces=traces, episodes=specs)
    flat = np.concatenate([all_chains[s] for s in sorted(traces)])
    for mode in (0, 1):
        say("60 random episodes, probe mode", mode)
        r = _run(gpu, work, mode=mode, chains=flat)
        for e, sp in enumerate(specs):
            tr = traces[sp.seed]
            o = orc.simulate_episode(W, cache, sp, tr.turn_off, tr.turn_blocks, tr.chain_off, all_chains[sp.seed])
            _compare_episode(r.episode_results(e), o, W, window=sp.concurrency, label=f"episode {e}")


def test_sweep70b_full_launch_sampled(gpu, orc):
    """All 320 episodes of the 1P/5D-shaped sweep in one launch; 3 sampled episodes vs the oracle."""
    say("generating 64 traces of 4,096 requests")
    w = wl.sweep70b_workload()
    say("running 320 episodes on the GPU")
    r = _run(gpu, w)
    cache = {}
    for e in (0, 64 * 2 + 17, 64 * 5 - 1):
        sp = r.episodes[e]
        say("oracle episode", e, "seed", sp.seed, "C", sp.concurrency)
        o = _oracle_episode(orc, w, sp, cache)
        _compare_episode(r.episode_results(e), o, w.W, window=sp.concurrency, label=f"sweep70b e{e}")
    poa = r.poa_hat.cpu().numpy()[: len(r.episodes)]
    assert np.all(np.isfinite(poa)) and np.all(poa > 0)


def test_saturation_subset(gpu, orc):
    """8 seeds x 8 concurrency levels x 5 overlap weights with the controller; 5 sampled episodes."""
    say("generating 8 saturation traces")
    w = wl.saturation_workload(seeds=range(8))
    say("running", len(w.episodes), "episodes on the GPU")
    r = _run(gpu, w)
    cache = {}
    idx = {(sp.seed, sp.concurrency, sp.w_ov): e for e, sp in enumerate(r.episodes)}
    for key in [(0, 8, 1.0), (1, 128, 1.0), (2, 256, 0.0), (3, 1024, 2.0), (7, 64, 0.25)]:
        e = idx[key]
        say("oracle episode", key)
        o = _oracle_episode(orc, w, r.episodes[e], cache)
        _compare_episode(r.episode_results(e), o, w.W, window=key[1], label=f"saturation {key}")
    tot = r.totals.cpu().numpy()[: len(r.episodes)]
    assert tot[:, 3].sum() > 0        # the controller fires somewhere in the sweep


def test_multiturn_subset(gpu, orc):
    """Long-context multi-turn episodes at full size (512 conversations, 16,384-block caches)."""
    say("generating 12 multi-turn traces")
    w = wl.multiturn_workload(seeds=range(12))
    say("running 12 episodes on the GPU")
    r = _run(gpu, w)
    cache = {}
    for e in (0, 11):
        say("oracle episode", e)
        o = _oracle_episode(orc, w, r.episodes[e], cache)
        _compare_episode(r.episode_results(e), o, w.W, window=256, label=f"multiturn e{e}")
        assert o["totals"][1] > 0


def test_eviction_extremes(gpu, orc):
    """Caches smaller than one prompt (a route evicts part of its own prompt), single worker."""
    tr = wl.tiny_trace(4)
    for W, cache in [(4, 1), (2, 7), (1, 40)]:
        say("eviction extremes W", W, "cache", cache)
        spec = wl.EpisodeSpec(seed=4, concurrency=8, cap=64)
        work = wl.Workload("x", W=W, cache_blocks=cache, traces={4: tr}, episodes=[spec])
        for mode in (0, 1):
            r = _run(gpu, work, mode=mode)
            o = orc.simulate_trace(W, cache, spec, tr)
            _compare_episode(r.episode_results(0), o, W, window=8, label=f"W{W} cache{cache}")


def test_determinism(gpu):
    torch, rk = gpu
    w = wl.sweep70b_workload(seeds=range(4), concurrency=(64, 256))
    from paper_2606_17081_amd.episodes import EpisodeRunner
    r = EpisodeRunner(w)
    r.step()
    a = [t.clone() for t in (r.route_worker, r.overlap, r.evict_digest, r.coord)]
    r.step()
    torch.cuda.synchronize()
    b = (r.route_worker, r.overlap, r.evict_digest, r.coord)
    for x, y in zip(a, b):
        assert torch.equal(x.cpu(), y.cpu())
    _status_clean(rk)


def test_snapshot_poa(gpu, orc):
    """PoA-hat of the snapshot workload: windows of 512 requests, K = 8 replicas per worker."""
    torch, rk = gpu
    inst = wl.scoring_instance(seed=2, B=4096, W=64, log2_slots=14, len_lo=16, len_hi=128)
    ov, co, am, _ = _score(rk, torch, inst, rk.RK_PROBE_PREFIX)
    P = np.diff(inst.chain_off).astype(np.int32)
    win = np.arange(0, inst.B + 1, 512, dtype=np.int64)
    up = rk.to_device
    sel = torch.zeros(win.size - 1, dtype=torch.float64, device="cuda")
    coo = torch.zeros_like(sel)
    hat = torch.zeros(1, dtype=torch.float64, device="cuda")
    pp = dict(wl.POA_PARAMS)
    params = rk.PoaParams(pp["a"], pp["b"], pp["d"], pp["beta"], pp["C_cap"], pp["w_c"], 8)
    ws = torch.empty(rk.poa_workspace_size(inst.B, 64), dtype=torch.uint8, device="cuda")
    rk.poa_estimate(up(win), up(np.array([0, win.size - 1], np.int64)), inst.B, 512, 64, up(am), up(ov), up(P),
                    params, sel, coo, hat, ws)
    torch.cuda.synchronize()
    _status_clean(rk)
    sel, coo = sel.cpu().numpy(), coo.cpu().numpy()
    for w in (0, 3, 7):
        s, c, _ = orc.poa_window(am[512 * w:512 * (w + 1)], ov[512 * w:512 * (w + 1)], P[512 * w:512 * (w + 1)],
                                 64, K=8, **pp)
        assert sel[w] == pytest.approx(s, rel=REL) and coo[w] == pytest.approx(c, rel=REL)
    assert float(hat[0]) == pytest.approx(sel.sum() / coo.sum(), rel=1e-12)


@pytest.mark.parametrize("W", [1, 2, 5, 8, 9, 12, 15, 16, 17, 24, 32, 40, 64])
def test_poa_worker_counts(gpu, orc, W):
    """Windows of 1..160 rows at worker counts on both sides of the kernel's lane layouts (rows of
    16 lanes for W <= 16, one lane per worker above), with overlaps from a few levels so that many
    costs tie and a moved row often held several edge minima; every window against the oracle."""
    torch, rk = gpu
    rng = np.random.default_rng(1000 + W)
    sizes = [1, 2, 3, W, W + 1, 2 * W, 5 * W + 3] + [int(x) for x in rng.integers(1, 161, 12)]
    sizes = [m for m in sizes if m >= 1]
    win = np.zeros(len(sizes) + 1, np.int64)
    np.cumsum(sizes, out=win[1:])
    n = int(win[-1])
    P = rng.integers(1, 300, n).astype(np.int32)
    am = rng.integers(0, W, n).astype(np.int32)
    lev = rng.choice([0.0, 0.25, 0.5, 1.0], size=(n, W), p=[0.4, 0.2, 0.2, 0.2])
    ov = np.floor(lev * P[:, None]).astype(np.int32)
    up = rk.to_device
    sel = torch.zeros(len(sizes), dtype=torch.float64, device="cuda")
    coo = torch.zeros_like(sel)
    hat = torch.zeros(1, dtype=torch.float64, device="cuda")
    pp = dict(wl.POA_PARAMS)
    params = rk.PoaParams(pp["a"], pp["b"], pp["d"], pp["beta"], pp["C_cap"], pp["w_c"], 0)
    mw = max(sizes)
    ws = torch.empty(rk.poa_workspace_size(n, W), dtype=torch.uint8, device="cuda")
    say("PoA parity, W", W, "windows", len(sizes), "rows", n)
    rk.poa_estimate(up(win), up(np.array([0, len(sizes)], np.int64)), n, mw, W, up(am), up(ov), up(P),
                    params, sel, coo, hat, ws)
    torch.cuda.synchronize()
    _status_clean(rk)
    sel, coo = sel.cpu().numpy(), coo.cpu().numpy()
    for w in range(len(sizes)):
        r0, r1 = int(win[w]), int(win[w + 1])
        s, c, _ = orc.poa_window(am[r0:r1], ov[r0:r1], P[r0:r1], W, **pp)
        assert sel[w] == pytest.approx(s, rel=REL), (W, w, sizes[w])
        assert coo[w] == pytest.approx(c, rel=REL), (W, w, sizes[w])


def test_lazy_recency_late_first_eviction(gpu, orc):
    """1P/5D-shaped traces with caches that fill only late in the episode (under LRU the kernel
    keeps no recency until a worker first evicts, then rebuilds it from the whole history of
    that worker's routes): every route, eviction count and digest against the oracle."""
    base = wl.sweep70b_workload(seeds=range(2), concurrency=(32, 512))
    late = 0
    for cache in (12288, 24000, 40000):
        w = wl.Workload("late-evict", W=base.W, cache_blocks=cache, traces=base.traces, episodes=base.episodes)
        say("sweep-shaped episodes with", cache, "-block caches")
        r = _run(gpu, w)
        oc = {}
        for e, sp in enumerate(base.episodes):
            o = _oracle_episode(orc, w, sp, oc)
            ev = np.nonzero(o["evict_count"])[0]
            late += int(ev.size > 0 and ev[0] > len(o["evict_count"]) // 4)   # a long history before it
            _compare_episode(r.episode_results(e), o, w.W, window=sp.concurrency, label=f"cache {cache} e{e}")
    assert late >= 8


def _repeated_turns_case(rng, n_conv, monotone):
    """Prefix-closed conversations of 1-5 turns; each turn reads the first turn_blocks of its
    conversation's chain, growing from turn to turn (monotone) or in any order."""
    chains, turn_blocks, turn_off, prefix_id = [], [], [0], {}
    for _ in range(n_conv):
        L = int(rng.integers(4, 48))
        path = tuple(int(x) for x in rng.integers(0, 3, size=L))
        chains.append([prefix_id.setdefault(path[:k], len(prefix_id) + 1) for k in range(1, L + 1)])
        tb = [int(x) for x in rng.integers(1, L + 1, size=int(rng.integers(1, 6)))]
        if monotone:
            tb.sort()
        turn_blocks.extend(tb)
        turn_off.append(len(turn_blocks))
    return chains, np.array(turn_off, np.int64), np.array(turn_blocks, np.int32)


def test_recency_rebuild_repeated_turns(gpu, orc):
    """Multi-turn episodes whose workers first evict after hundreds of routes, so the recency
    rebuilt from a worker's history spans several chunks of 256 routes, with later turns of a
    conversation on the same worker rereading its chain (the rebuild skips the touches they
    repeat), turn lengths growing or in any order: every route, overlap, eviction count and
    digest against the oracle."""
    rng = np.random.default_rng(2024)
    W = 3
    traces, all_chains = {}, {}
    for seed in range(6):
        chains, turn_off, turn_blocks = _repeated_turns_case(rng, 600, monotone=seed % 2 == 0)
        lens = np.array([len(c) for c in chains], np.int32)
        chain_off = np.zeros(len(chains) + 1, np.int64)
        np.cumsum(lens, out=chain_off[1:])
        traces[seed] = wl.Trace(seed=seed, tokens=np.zeros(16, np.int32), tok_off=chain_off * 0,
                                chain_blocks=lens, chain_off=chain_off, turn_off=turn_off,
                                turn_blocks=turn_blocks, group=np.zeros(len(chains), np.int32),
                                shared=np.zeros(len(chains), np.int32))
        all_chains[seed] = np.array([k for c in chains for k in c], np.uint64)
    flat = np.concatenate([all_chains[s] for s in sorted(traces)])
    specs = [wl.EpisodeSpec(seed=s, concurrency=8, hold_steps=2, w_ov=w, w_act=0.5, w_sat=4.0, cap=200)
             for s in sorted(traces) for w in (1.0, 2.0)]
    spanned = 0
    for cache in (1200, 2400):
        work = wl.Workload("repeated-turns", W=W, cache_blocks=cache, traces=traces, episodes=specs)
        say("repeated-turn episodes with", cache, "-block caches")
        r = _run(gpu, work, chains=flat)
        for e, sp in enumerate(specs):
            tr = traces[sp.seed]
            o = orc.simulate_episode(W, cache, sp, tr.turn_off, tr.turn_blocks, tr.chain_off, all_chains[sp.seed])
            _compare_episode(r.episode_results(e), o, W, window=sp.concurrency, label=f"cache {cache} e{e}")
            # routes before their worker's first eviction whose conversation comes back to that
            # worker in a later chunk of 256 routes, also before it
            rw = np.asarray(o["route_worker"])
            conv = np.searchsorted(tr.turn_off, np.asarray(o["route_turn"]), side="right") - 1
            ev = np.nonzero(o["evict_count"])[0]
            for j in range(W):
                evj = ev[rw[ev] == j]
                t_end = int(evj[0]) if evj.size else 0
                last = {}
                for t in range(t_end - 1, -1, -1):
                    if rw[t] != j:
                        continue
                    if conv[t] in last and last[conv[t]] // 256 != t // 256:
                        spanned += 1
                    last.setdefault(conv[t], t)
    assert spanned >= 100, spanned


def test_workspace_contents_never_read(gpu, orc):
    """An episode clears the parts of its workspace it uses (the run index at
    its start; a worker's block table at its start under frequency eviction,
    else at the worker's first eviction): launches on a workspace filled with
    random bytes give the same routes, overlaps, costs, evictions and totals
    as the first launch, for LRU episodes that evict and for frequency
    eviction, in one launch."""
    torch, rk = gpu
    from paper_2606_17081_amd.episodes import EpisodeRunner
    w = wl.multiturn_workload(seeds=range(2), n_conv=96)
    eps = [wl.EpisodeSpec(**{**sp.__dict__, "cap": 512}) for sp in w.episodes]
    eps += [wl.EpisodeSpec(**{**sp.__dict__, "cap": 512, "evict_policy": wl.EVICT_FREQ, "decay_steps": 3})
            for sp in w.episodes]
    w2 = wl.Workload(w.name, W=w.W, cache_blocks=1024, traces=w.traces, episodes=eps)
    r = EpisodeRunner(w2)
    r.hash()
    r.simulate()
    torch.cuda.synchronize()
    _status_clean(rk)
    outs = (r.route_worker, r.overlap, r.cost, r.evict_digest, r.totals)
    ref = [t.clone() for t in outs]
    assert int(ref[4][:, 1].sum()) > 0, "the case must evict"
    gen = torch.Generator(device="cuda")
    for rep in range(3):
        gen.manual_seed(rep)
        r.workspace.copy_(torch.randint(0, 256, r.workspace.shape, dtype=torch.uint8, device="cuda",
                                        generator=gen))
        for t in outs:
            t.zero_()
        r.simulate()
        torch.cuda.synchronize()
        _status_clean(rk)
        for k, (v, x) in enumerate(zip(outs, ref)):
            assert torch.equal(v, x), f"output {k} differs after filling the workspace (pass {rep})"
    for e in (0, 3):
        sp = r.episodes[e]
        say("oracle episode", e, "eviction policy", sp.evict_policy)
        o = orc.simulate_trace(w2.W, w2.cache_blocks, sp, w2.traces[sp.seed])
        _compare_episode(r.episode_results(e), o, w2.W, label=f"random workspace e{e}")


@pytest.mark.parametrize("name", ["sweep", "multiturn"])
def test_lean_decision_loop_matches_full(gpu, name):
    """Episodes routed by argmin under LRU without a controller run the lean
    copy of the decision loop; the same episodes with the overlap-weight
    controller switched on at a load it can never reach run the lean copy with
    the controller, and with the regime controller held in its first regime
    (thresholds never reached, that regime's weight and temperature those of
    the episode) the full copy; all three must route identically (routes,
    overlaps, costs, evictions, totals)."""
    from dataclasses import replace
    torch, rk = gpu
    base = (wl.sweep70b_workload(seeds=range(4), concurrency=(32, 512)) if name == "sweep"
            else wl.multiturn_workload(seeds=range(2)))
    ctrl = wl.Workload(base.name, W=base.W, cache_blocks=base.cache_blocks, traces=base.traces,
                       episodes=[replace(sp, controller=1, ctrl_num=1 << 30, ctrl_den=1) for sp in base.episodes])
    assert all(sp.w_ov == 1.0 for sp in base.episodes)
    full = wl.Workload(base.name, W=base.W, cache_blocks=base.cache_blocks, traces=base.traces,
                       episodes=[replace(sp, controller=2) for sp in base.episodes],
                       regime=dict(wl.REGIME_PARAMS, theta1=1e30, theta2=1e30, tau=(0.0, 0.7, 0.8),
                                   w_ov=(1.0, 1.0, 0.1)))
    outs = []
    for w in (base, ctrl, full):
        say(name, "episodes", len(w.episodes), "controller", w.episodes[0].controller)
        r = _run(gpu, w)
        n = r.n_rows
        outs.append([r.route_worker[:n].cpu().numpy(), r.overlap[:n].cpu().numpy(),
                     r.cost[:n].cpu().numpy().view(np.uint32), r.evict_digest[:n].cpu().numpy(),
                     r.totals.cpu().numpy()])
        assert rk.device_status(reset=True) == 0
    for v in (1, 2):
        for k, (a, b) in enumerate(zip(outs[0], outs[v])):
            if k == 4:        # totals: the controllers count their own activity in columns 3 and 4
                a, b = np.delete(a, [3, 4], axis=1), np.delete(b, [3, 4], axis=1)
            assert np.array_equal(a, b), f"output {k} differs between the lean loop and copy {v}"


def test_queued_workspaces_match(gpu, orc):
    """Fewer episode workspaces than episodes: 7 workgroups take 160 saturation
    episodes in turn, each episode clearing what it uses of its workspace (the
    last pass starts on a workspace filled with random bytes).  Every output
    equals the launch with one workspace per episode, and episodes run before
    and after a workspace changed hands (the first 7 and the last ones of the
    queue) match the oracle."""
    torch, rk = gpu
    from paper_2606_17081_amd.episodes import EpisodeRunner
    w = wl.saturation_workload(seeds=range(4))
    say("saturation, one workspace per episode:", len(w.episodes), "episodes")
    ref = _run(gpu, w)
    n, E = ref.n_rows, len(w.episodes)
    want = [t[:n].cpu().numpy() for t in (ref.route_worker, ref.overlap, ref.evict_count, ref.evict_digest,
                                          ref.last_hash)]
    want += [ref.cost[:n].cpu().numpy().view(np.uint32), ref.totals[:E].cpu().numpy(), ref.poa_hat[:E].cpu().numpy()]
    r = EpisodeRunner(w, ws_slots=7)
    assert r.workspace.numel() == rk.simulate_workspace_size(7, w.W, w.cache_blocks, r.max_blocks, r.max_conv,
                                                             r.max_routes)
    r.hash()
    for rep in range(3):
        say("7 workspaces, pass", rep)
        for t in (r.route_worker, r.overlap, r.cost, r.evict_digest, r.totals, r.poa_hat):
            t.zero_()
        if rep == 2:
            r.workspace.copy_(torch.randint(0, 256, r.workspace.shape, dtype=torch.uint8, device="cuda"))
        r.simulate()
        r.poa()
        torch.cuda.synchronize()
        _status_clean(rk)
        got = [t[:n].cpu().numpy() for t in (r.route_worker, r.overlap, r.evict_count, r.evict_digest,
                                             r.last_hash)]
        got += [r.cost[:n].cpu().numpy().view(np.uint32), r.totals[:E].cpu().numpy(), r.poa_hat[:E].cpu().numpy()]
        for k, (a, b) in enumerate(zip(want, got)):
            assert np.array_equal(a, b), f"output {k} differs with 7 workspaces (pass {rep})"
    cache = {}
    for e in list(range(7)) + [E - 41, E - 1]:
        sp = r.episodes[e]
        say("oracle episode", e, "C", sp.concurrency, "w_ov", sp.w_ov)
        o = _oracle_episode(orc, w, sp, cache)
        _compare_episode(r.episode_results(e), o, w.W, window=sp.concurrency, label=f"queued e{e}")


def test_saturation_full_launch_sampled(gpu, orc):
    """All 10,240 saturation / controller episodes in one launch on 512 episode
    workspaces (the benchmark's configuration); sampled episodes of every
    concurrency level against the oracle, the first and the last of the queue
    among them."""
    torch, rk = gpu
    from paper_2606_17081_amd.episodes import EpisodeRunner
    say("generating 256 saturation traces")
    w = wl.saturation_workload()
    say("running", len(w.episodes), "episodes on 512 workspaces")
    r = EpisodeRunner(w, ws_slots=512)
    r.step()
    torch.cuda.synchronize()
    _status_clean(rk)
    E = len(r.episodes)
    idx = {(sp.seed, sp.concurrency, sp.w_ov): e for e, sp in enumerate(r.episodes)}
    keys = [(0, 8, 0.0), (200, 8, 1.0), (255, 16, 2.0), (17, 32, 0.25), (99, 64, 0.5), (128, 128, 1.0),
            (64, 256, 0.0), (3, 512, 2.0), (255, 1024, 2.0)]
    cache = {}
    for key in keys:
        e = idx[key]
        say("oracle episode", e, key)
        o = _oracle_episode(orc, w, r.episodes[e], cache)
        _compare_episode(r.episode_results(e), o, w.W, window=key[1], label=f"saturation {key}")
    assert idx[(255, 1024, 2.0)] == E - 1
    P = r.route_blocks[: r.n_rows].cpu().numpy()
    ov = r.overlap[: r.n_rows].cpu().numpy()
    assert np.all(ov >= 0) and np.all(ov <= P[:, None])
    tot = r.totals[:E].cpu().numpy()
    assert tot[:, 3].sum() > 0 and tot[:, 1].sum() > 0     # the controller fires, some episodes evict
