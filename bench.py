"""Benchmark of the KV-aware routing hot path on one MI355X.

One step = one pass of the whole path over the 1P/5D-shaped sweep: block-hash
chains of 64 traces of 4,096 requests, 320 routing episodes (W = 6 workers,
C in {32, 64, 128, 256, 512} x 64 seeds), and the PoA-hat windows and ratios.
Inputs (tokens, offsets, parameters) are resident in HBM before timing.
Consecutive steps overlap on two streams (two sets of buffers take turns): a
step's episodes run while the other stream finishes the previous step's
PoA-hat and hashes and clears the tables for the next step; every step still
does all of its work inside the timed region, and its results are checked
against a sequential step.

Also measured in the same run: the batched scoring kernel on 65,536 requests x
64 workers with 2^20-slot tables, and the CPU oracle on a bounded sample of
the sweep (reported as cpu_baseline).

Prints one JSON line.  Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "request×worker route scorings/sec + routing episodes/sec; % HBM roofline"
HBM_PEAK_GBS = 8000.0
PROFILE_DIR = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = {
    "episode_kernel": ["paper_2606_17081_amd/csrc/episode.hip", "paper_2606_17081_amd/csrc/rk_internal.h"],
    "score_kernel": ["paper_2606_17081_amd/csrc/score.hip", "paper_2606_17081_amd/csrc/rk_internal.h"],
    "score_index_kernel": ["paper_2606_17081_amd/csrc/index.hip", "paper_2606_17081_amd/csrc/rk_internal.h"],
    "poa_window_kernel": ["paper_2606_17081_amd/csrc/poa.hip", "paper_2606_17081_amd/csrc/rk_internal.h"],
    "block_fnv_kernel": ["paper_2606_17081_amd/csrc/abi.hip", "paper_2606_17081_amd/csrc/rk_internal.h"],
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_digest(kernel: str) -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source; else None."""
    path = os.path.join(PROFILE_DIR, f"traffic_{kernel}_{workload}.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, v = line.split("=", 1)
                vals[k.strip()] = v.strip()
    if vals.get("source_sha256_16") != source_digest(kernel):
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


# ---------------------------------------------------------------- algorithmic bytes

def table_clear_bytes(runner) -> float:
    """Bytes the tables' clear must write per launch: every 16-byte slot of
    the W tables of every episode."""
    live_max = runner.cache_blocks + runner.max_blocks
    S = 1 << int(np.ceil(np.log2(2 * live_max)))
    return float(len(runner.episodes) * runner.W * S * 16)


def episode_algorithmic_bytes(runner) -> float:
    """Bytes the episode kernel must move per launch, each access counted
    once at its natural width (no cache-line rounding):
      per route:   per worker the keys a binary search for the first miss
                   reads, ceil(log2(P + 1)) probes of 8 B; 8 B of outputs per
                   worker (overlap, cost) and 28 B per route; the first chain
                   hash of the route compared with those of the other routes
                   of its batch of 64 (8 B each);
                   on a worker that evicts at some point of the episode, the
                   touch of P blocks (chain hash read 8, key read 8, stamp
                   write 4, log write 4) and insert of P - o keys (8 each);
                   on a worker that never evicts, recency decides nothing, so
                   only the P - o missing blocks: chain hash read 8, key
                   write 8;
      per eviction: log read 4, stamp read 4 and write 4, key read 8."""
    W = runner.W
    n = runner.n_rows
    P = runner.route_blocks[:n].cpu().numpy().astype(np.float64)
    sig = runner.route_worker[:n].cpu().numpy()
    ov = runner.overlap[:n].cpu().numpy()
    o_sig = ov[np.arange(n), sig].astype(np.float64)
    ev = runner.evict_count[:n].cpu().numpy().astype(np.float64)
    probes = np.ceil(np.log2(P + 1.0))
    # routes on (episode, worker) pairs that evict at some point
    evicting = np.zeros(n, bool)
    for (r0, nr, _, _) in runner.rows:
        sl = slice(r0, r0 + nr)
        ws = np.unique(sig[sl][ev[sl] > 0])
        evicting[sl] = np.isin(sig[sl], ws)
    b = np.sum(8 * W * probes + 8 * W + 28 + 8 * 63)
    b += np.sum(np.where(evicting, 28 * P + 8 * (P - o_sig), 16 * (P - o_sig)))
    b += np.sum(20 * ev)
    return float(b)


def score_algorithmic_bytes(inst) -> float:
    """Compulsory bytes of one batched-scoring launch: every table slot once,
    every chain hash once, the offsets, and the outputs (overlap and cost per
    pair, argmin per request)."""
    B, W = inst.B, inst.W
    tables = W * (1 << inst.log2_slots) * 8
    chains = inst.chains.size * 8
    offs = (B + 1) * 8 + W * 4
    outs = B * W * (4 + 4) + B * 4
    return float(tables + chains + offs + outs)


def score_index_algorithmic_bytes(inst, overlap: np.ndarray) -> float:
    """Bytes the global-index scorer needs per launch, each access counted once
    at its natural width: every chain hash once, the offsets and loads, the
    outputs, and one 16-byte index slot per position a first-miss scan of the
    union must see: M_i + [M_i < P_i] positions, M_i = max_j o_ij (positions
    past M_i are cached nowhere, one all-miss probe closes the scan)."""
    B, W = inst.B, inst.W
    P = np.diff(inst.chain_off).astype(np.float64)
    M = overlap.max(axis=1).astype(np.float64) if W > 0 else np.zeros(B)
    index = 16.0 * np.sum(M + (M < P))
    chains = inst.chains.size * 8
    offs = (B + 1) * 8 + W * 4
    outs = B * W * (4 + 4) + B * 4
    return float(index + chains + offs + outs)


# ---------------------------------------------------------------- timing helpers

class KernelTimer:
    """HIP events around one stage, recorded on the stream the stage runs on."""

    def __init__(self, torch, stream):
        self.torch, self.stream, self.pairs = torch, stream, []

    def __enter__(self):
        self.a = self.torch.cuda.Event(enable_timing=True)
        self.b = self.torch.cuda.Event(enable_timing=True)
        self.a.record(self.stream)
        return self

    def __exit__(self, *exc):
        self.b.record(self.stream)
        self.pairs.append((self.a, self.b))

    def mean_ms(self):
        self.torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in self.pairs])) if self.pairs else 0.0


def burst_ms(torch, stream, fn, n):
    """Mean duration of n back-to-back launches of fn, from one pair of HIP
    events on the launching stream around all of them (for launches of tens
    of microseconds, where an event pair per launch would add its own
    overhead to each)."""
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(n):
        fn()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / n


def cpu_baseline(workload, seeds, threads):
    """The CPU oracle on a bounded sample: hash the sampled traces, run every
    episode of those seeds (all five concurrency levels) and its PoA-hat."""
    from concurrent.futures import ThreadPoolExecutor
    from oracle import oracle as O
    from paper_2606_17081_amd.workload import POA_PARAMS
    specs = [e for e in workload.episodes if e.seed in seeds]
    t0 = time.perf_counter()
    with ThreadPoolExecutor(max_workers=threads) as ex:
        chains = dict(zip(seeds, ex.map(lambda s: O.trace_chains(workload.traces[s]), seeds)))

        def one(sp):
            out = O.simulate_trace(workload.W, workload.cache_blocks, sp, workload.traces[sp.seed], chains[sp.seed])
            O.episode_poa(out, workload.W, sp.concurrency, POA_PARAMS)
            return len(out["route_worker"])
        routes = sum(ex.map(one, specs))
    dt = time.perf_counter() - t0
    return dict(value=routes * workload.W / dt, unit="scorings/s", cores=threads, kind="oracle",
                sample=f"{len(specs)} episodes (seeds {min(seeds)}..{max(seeds)} x C in 32..512) of the "
                       f"1P/5D-shaped sweep incl. hashing and PoA-hat; {routes} routes in {dt:.2f} s",
                episodes_per_s=len(specs) / dt, seconds=dt)


def index_log2_slots(n_keys: int) -> int:
    """Index slots for n_keys insertions at load <= 0.25: short probe walks
    (2^27 slots, 2 GiB, for the 65,536 x 64 instance)."""
    b = 4
    while (1 << b) < 4 * n_keys:
        b += 1
    return b


def scoring_bench(torch, rk, wl, stream, steps):
    """Time the 65,536 x 64 snapshot scoring on the per-worker tables
    (rk_route_score_batch) and on the global block index
    (rk_route_score_index) built from the same key sets."""
    log("generating the 65,536 x 64 scoring instance")
    inst = wl.scoring_instance(seed=0)
    up = rk.to_device
    keys = up(inst.keys)
    tables = rk.table_build(keys, inst.key_off, inst.log2_slots)
    chains, chain_off, active = up(inst.chains), up(inst.chain_off), up(inst.active)
    ov = torch.empty((inst.B, inst.W), dtype=torch.int32, device="cuda")
    co = torch.empty((inst.B, inst.W), dtype=torch.float32, device="cuda")
    am = torch.empty(inst.B, dtype=torch.int32, device="cuda")
    for _ in range(3):
        rk.route_score_batch(chains, chain_off, tables, inst.log2_slots, active, overlap=ov, cost=co, argmin=am)
    ms = burst_ms(torch, stream, lambda: rk.route_score_batch(chains, chain_off, tables, inst.log2_slots, active,
                                                              overlap=ov, cost=co, argmin=am), max(steps, 10))
    assert rk.device_status(reset=True) == 0
    salg = score_algorithmic_bytes(inst)
    ach = salg / (ms * 1e-3) / 1e9
    log(f"scoring (tables): {ms:.4f} ms, {inst.B * inst.W / (ms * 1e-3):.4g} scorings/s, {ach:.1f} GB/s algorithmic")
    ov_ref = ov.cpu().numpy()
    del tables
    torch.cuda.empty_cache()

    lg = index_log2_slots(int(inst.key_off[-1]))
    tb = KernelTimer(torch, stream)
    index = torch.empty(2 << lg, dtype=torch.int64, device="cuda")
    for _ in range(3):
        with tb:
            rk.index_build(keys, inst.key_off, lg, index=index)
    for _ in range(3):
        rk.route_score_index(chains, chain_off, index, lg, active, overlap=ov, cost=co, argmin=am)
    ms_i = burst_ms(torch, stream, lambda: rk.route_score_index(chains, chain_off, index, lg, active, overlap=ov,
                                                                cost=co, argmin=am), max(steps, 10))
    assert rk.device_status(reset=True) == 0
    ov_i = ov.cpu().numpy()
    assert np.array_equal(ov_i, ov_ref), "index and table scorers disagree"
    ialg = score_index_algorithmic_bytes(inst, ov_i)
    ach_i = ialg / (ms_i * 1e-3) / 1e9
    log(f"scoring (index): {ms_i:.4f} ms, {inst.B * inst.W / (ms_i * 1e-3):.4g} scorings/s, "
        f"{ach_i:.1f} GB/s algorithmic; index build {tb.mean_ms():.3f} ms")
    wl_name = "scoring 65536 requests x 64 workers, 2^20-slot tables at load 0.5, chains of 16..512"
    return {"workload": wl_name,
            "scorings_per_s": inst.B * inst.W / (ms * 1e-3), "avg_ms": round(ms, 4),
            "roofline": {"kernel": "score_kernel", "bound": "hbm", "achieved": round(ach, 3),
                         "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 6),
                         "traffic": measured_traffic("score_kernel", "scoring"),
                         "algorithmic_bytes": salg},
            "index": {"workload": wl_name + "; the same key sets in one global block index of "
                                            f"2^{lg} 16-byte slots",
                      "scorings_per_s": inst.B * inst.W / (ms_i * 1e-3), "avg_ms": round(ms_i, 4),
                      "index_build_ms": round(tb.mean_ms(), 4),
                      "roofline": {"kernel": "score_index_kernel", "bound": "hbm", "achieved": round(ach_i, 3),
                                   "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ach_i / HBM_PEAK_GBS, 6),
                                   "traffic": measured_traffic("score_index_kernel", "scoring"),
                                   "algorithmic_bytes": ialg}}}


def policy_bench(torch, rk, wl, stream, steps):
    """The 1P/5D-shaped traces under every selection policy (the router's
    argmin and softmax, and the static round-robin, random and power-of-two
    policies): 16 seeds x 5 concurrency levels x 5 policies in one launch;
    PoA-hat per policy and concurrency level."""
    from paper_2606_17081_amd.episodes import EpisodeRunner
    log("generating the policy sweep (16 traces, 480 episodes)")
    w = wl.policy_workload()
    r = EpisodeRunner(w, keep_cost=False)
    r.hash()
    r.simulate()
    r.poa()
    torch.cuda.synchronize()
    ts, tp = KernelTimer(torch, stream), KernelTimer(torch, stream)
    for _ in range(max(1, steps // 2)):
        with ts:
            r.simulate()
        with tp:
            r.poa()
    torch.cuda.synchronize()
    assert rk.device_status(reset=True) == 0
    poa = r.poa_hat[: len(r.episodes)].cpu().numpy()
    out = {}
    for p, tau in wl.POLICY_SWEEP:
        name = wl.POLICY_NAMES[p] + (f" tau={tau:g}" if p == wl.POLICY_SOFTMAX else "")
        by_c = {}
        for C in wl.SWEEP70B_C:
            v = np.array([poa[e] for e, sp in enumerate(r.episodes) if sp.policy == p and sp.concurrency == C])
            by_c[str(C)] = [round(float(v.mean()), 6), round(float(v.std()), 6)]
        out[name] = by_c
    by_c, share = {}, {}
    reg = r.route_regime[: r.n_rows].cpu().numpy()
    for C in wl.SWEEP70B_C:
        es = [e for e, sp in enumerate(r.episodes) if sp.controller == 2 and sp.concurrency == C]
        if es:
            v = poa[es]
            by_c[str(C)] = [round(float(v.mean()), 6), round(float(v.std()), 6)]
            rows = np.concatenate([np.arange(r.rows[e][0], r.rows[e][0] + r.rows[e][1]) for e in es])
            share[str(C)] = [round(float(np.mean(reg[rows] == k)), 4) for k in range(3)]
    if by_c:
        out["regime controller"] = by_c
        out["regime controller: share of routes Below/Transition/Saturated"] = share
    E = len(r.episodes)
    log(f"policies: {E} episodes, simulate {ts.mean_ms():.3f} ms, PoA {tp.mean_ms():.3f} ms")
    return {"workload": "1P/5D-shaped traces, W=6, 4096 requests, C in {32..512} x 16 seeds x "
                        "(5 policies + the regime controller)",
            "episodes": E, "simulate_ms": round(ts.mean_ms(), 4), "poa_ms": round(tp.mean_ms(), 4),
            "episodes_per_s": E / (ts.mean_ms() * 1e-3), "poa_hat_by_policy_and_C": out}


def cache_bench(torch, rk, wl, stream, steps, seeds=16):
    """The long-context multi-turn traces (32 workers, 512 conversations,
    16,384-block caches, C = 256) under LRU, frequency eviction (decay every 4
    and 64 steps) and LRU with memory tiers (G1 = G2 = 4,096 blocks, G3 the
    other 8,192; weights 0, 0.25, 0.5): PoA-hat, recomputed prefill blocks,
    evictions and, with tiers, where the reused blocks came from."""
    from paper_2606_17081_amd.episodes import EpisodeRunner
    log(f"generating {seeds} multi-turn traces")
    base = wl.multiturn_workload(seeds=range(seeds))
    variants = [("lru", {}), ("frequency, decay every 4 steps", dict(evict_policy=wl.EVICT_FREQ, decay_steps=4)),
                ("frequency, decay every 64 steps", dict(evict_policy=wl.EVICT_FREQ, decay_steps=64)),
                ("lru, tiers G1/G2/G3 = 4096/4096/8192", dict(tier_g1=4096, tier_g2=4096))]
    out = {}
    for name, kw in variants:
        eps = [wl.EpisodeSpec(**{**sp.__dict__, **kw}) for sp in base.episodes]
        w = wl.Workload(base.name, W=base.W, cache_blocks=base.cache_blocks, traces=base.traces, episodes=eps)
        r = EpisodeRunner(w, keep_cost=False)
        r.hash()
        r.simulate()
        r.poa()
        torch.cuda.synchronize()
        ts = KernelTimer(torch, stream)
        for _ in range(max(1, steps // 4)):
            with ts:
                r.simulate()
        r.poa()
        torch.cuda.synchronize()
        assert rk.device_status(reset=True) == 0
        E = len(eps)
        tot = r.totals[:E].cpu().numpy()
        poa = r.poa_hat[:E].cpu().numpy()
        res = {"episodes": E, "simulate_ms": round(ts.mean_ms(), 3), "episodes_per_s": round(E / (ts.mean_ms() * 1e-3), 1),
               "routes_per_s": float(r.n_rows / (ts.mean_ms() * 1e-3)),
               "poa_hat": [round(float(poa.mean()), 6), round(float(poa.std()), 6)],
               "recomputed_blocks_per_episode": round(float(tot[:, 0].mean()), 1),
               "reused_blocks_per_episode": round(float(tot[:, 6].mean()), 1),
               "evicted_blocks_per_episode": round(float(tot[:, 1].mean()), 1)}
        if r.tier_overlap is not None:
            n = r.n_rows
            sig = r.route_worker[:n].long()
            rows = torch.arange(n, device=sig.device)
            t = r.tier_overlap[:n][rows, sig].long().cpu().numpy()
            o = r.overlap[:n][rows, sig].long().cpu().numpy()
            g1, g2, g3 = t[:, 0].sum(), (t[:, 1] - t[:, 0]).sum(), (o - t[:, 1]).sum()
            res["reused_blocks_share_G1_G2_G3"] = [round(float(x / max(o.sum(), 1)), 4) for x in (g1, g2, g3)]
        log(f"cache policies: {name}: {res}")
        out[name] = res
    return {"workload": f"long-context multi-turn traces, W=32, 512 conversations, 16384-block caches, C=256, "
                        f"{seeds} seeds per variant", "variants": out}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-scoring", action="store_true")
    ap.add_argument("--cpu-seeds", type=int, default=64)
    ap.add_argument("--no-policies", action="store_true")
    ap.add_argument("--no-cache-policies", action="store_true")
    ap.add_argument("--only", choices=("all", "sweep", "scoring", "policies", "cache"), default="all",
                    help="profiling passes: run only the sweep step or only the scoring kernel")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain device copy of this size (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: episodes shard across GPUs with no exchange, "
              "and runs on several GPUs are not provided", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_17081_amd import rkroute as rk
    from paper_2606_17081_amd import workload as wl
    from paper_2606_17081_amd.episodes import EpisodeRunner
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)

    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copied {n} bytes 5 times")
        return

    if args.only == "scoring":
        score = scoring_bench(torch, rk, wl, torch.cuda.current_stream(), args.steps)
        print(json.dumps({"score_batch": score}), flush=True)
        return
    if args.only == "policies":
        pol = policy_bench(torch, rk, wl, torch.cuda.current_stream(), args.steps)
        print(json.dumps({"policies": pol}), flush=True)
        return
    if args.only == "cache":
        cp = cache_bench(torch, rk, wl, torch.cuda.current_stream(), args.steps)
        print(json.dumps({"cache_policies": cp}), flush=True)
        return
    log("generating the sweep (64 traces of 4,096 requests)")
    w = wl.sweep70b_workload()
    # Two runners (each with its own chains, outputs and workspace) take turns, so that consecutive
    # steps can overlap: step k's episodes run on the main stream while the second stream computes
    # step k-1's PoA-hat and hashes and clears the tables for step k+1.  Each step still does all of
    # its work (hash, clear, episodes, PoA-hat) inside the timed region.
    runners = [EpisodeRunner(w, keep_cost=True) for _ in range(2)]
    runner = runners[0]
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    log(f"{len(runner.episodes)} episodes, {runner.n_rows} routes, {runner.n_windows} PoA windows; warmup {args.warmup}")
    for _ in range(max(1, args.warmup)):      # at least one untimed sequential step: the reference
        for r in runners:
            r.step()
    torch.cuda.synchronize()
    assert rk.device_status(reset=True) == 0
    # the sequential result every pipelined step must reproduce
    E0, n0 = len(runner.episodes), runner.n_rows
    ref_poa = runner.poa_hat[:E0].clone()
    ref_route = runner.route_worker[:n0].clone()

    side = torch.cuda.Stream()
    t_sim = KernelTimer(torch, stream)
    t_hash, t_clear, t_poa = KernelTimer(torch, side), KernelTimer(torch, side), KernelTimer(torch, side)
    e_sim = [None] * args.steps

    def prepare(k):
        """Hash and clear the tables for step k on the second stream, once the episodes of the
        runner's previous step (k - 2) are done."""
        r = runners[k % 2]
        if k >= 2:
            side.wait_event(e_sim[k - 2])
        with t_hash:
            r.hash(stream=side)
        with t_clear:
            r.clear_tables(stream=side)
        ready = torch.cuda.Event()
        ready.record(side)
        return ready

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ready = prepare(0)
    for k in range(args.steps):
        r = runners[k % 2]
        stream.wait_event(ready)
        with t_sim:
            r.simulate(stream=stream, tables_clear=True)
        done = torch.cuda.Event()
        done.record(stream)
        e_sim[k] = done
        if k + 1 < args.steps:
            ready = prepare(k + 1)
        side.wait_event(done)
        with t_poa:
            r.poa(stream=side)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    assert rk.device_status(reset=True) == 0
    for r in runners[: min(2, args.steps)]:
        assert torch.equal(r.poa_hat[:E0], ref_poa), "pipelined steps differ from the sequential step (PoA-hat)"
        assert torch.equal(r.route_worker[:n0], ref_route), "pipelined steps differ from the sequential step (routes)"
    ms_step = wall * 1e3 / args.steps
    E = len(runner.episodes)
    scorings = runner.n_rows * runner.W
    stage_ms = dict(hash=t_hash.mean_ms(), simulate=t_sim.mean_ms(), poa=t_poa.mean_ms())
    clear_ms = t_clear.mean_ms()
    clear_bytes = table_clear_bytes(runner)
    log(f"step {ms_step:.3f} ms; stages {stage_ms} (hash and PoA-hat on the second stream); "
        f"table clear {clear_ms:.3f} ms on the second stream")
    poa_hat = runner.poa_hat[:E].cpu().numpy()
    per_C = {}
    for C in wl.SWEEP70B_C:
        v = np.array([poa_hat[e] for e, sp in enumerate(runner.episodes) if sp.concurrency == C])
        per_C[str(C)] = [round(float(v.mean()), 6), round(float(v.std()), 6)]

    dom = max(stage_ms, key=stage_ms.get)
    dom_kernel = {"hash": "block_fnv_kernel", "simulate": "episode_kernel", "poa": "poa_window_kernel"}[dom]
    dom_label = dom_kernel
    if dom_kernel == "episode_kernel":
        alg = episode_algorithmic_bytes(runner)
    else:
        alg = None
    roofline = None
    if alg is not None:
        achieved = alg / (stage_ms[dom] * 1e-3) / 1e9
        traffic = measured_traffic(dom_kernel, "sweep70b")
        roofline = {"kernel": dom_label, "bound": "hbm", "achieved": round(achieved, 3), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 6),
                    "traffic": traffic, "algorithmic_bytes": alg, "avg_ms": round(stage_ms[dom], 4)}
    else:
        roofline = {"kernel": dom_kernel, "bound": "alu", "achieved": None, "peak": None, "unit": None,
                    "frac": None, "traffic": None, "avg_ms": round(stage_ms[dom], 4)}

    score = None
    if not args.no_scoring and args.only == "all":
        del runner, runners
        torch.cuda.empty_cache()
        score = scoring_bench(torch, rk, wl, stream, args.steps)

    pol = None
    if not args.no_policies and args.only == "all":
        torch.cuda.empty_cache()
        pol = policy_bench(torch, rk, wl, stream, args.steps)

    cache_pol = None
    if not args.no_cache_policies and args.only == "all":
        torch.cuda.empty_cache()
        cache_pol = cache_bench(torch, rk, wl, stream, args.steps)

    cpu = None
    if not args.no_cpu_baseline and args.only == "all":
        threads = max(1, min(16, os.cpu_count() or 1))
        log(f"oracle on {args.cpu_seeds} seeds x 5 concurrency levels with {threads} threads")
        cpu = cpu_baseline(w, list(range(args.cpu_seeds)), threads)
        log(f"oracle: {cpu['value']:.4g} scorings/s in {cpu['seconds']:.2f} s")

    line = {
        "metric": METRIC,
        "value": scorings / (ms_step * 1e-3),
        "unit": "scorings/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64/i32 hashing and probes, f32 cost, f64 PoA sums",
        "data": "synthetic",
        "config": {"workload": "sweep70b: 70B-1P/5D-shaped sweep, W=6 workers, 4096 requests per episode, "
                               "C in {32,64,128,256,512} x 64 seeds = 320 episodes; hash + episodes + PoA-hat",
                   "episodes": E, "routes": runner_rows(scorings, w.W), "scorings_per_step": scorings},
        "episodes_per_s": E / (ms_step * 1e-3),
        "routes_per_s": scorings / w.W / (ms_step * 1e-3),
        "stage_ms": {k: round(v, 4) for k, v in stage_ms.items()},
        "pipeline": "two runners take turns: step k's episodes on the main stream while the second stream "
                    "runs step k-1's PoA-hat and hashes and clears step k+1's tables (stage times are "
                    "measured under that overlap); every step's PoA-hat and routes are checked against a "
                    "sequential step",
        "table_clear": {"kernel": "episode_clear_kernel", "avg_ms": round(clear_ms, 4),
                        "stream": "second stream, beside the next step's episodes",
                        "roofline": {"bound": "hbm", "achieved": round(clear_bytes / (clear_ms * 1e-3) / 1e9, 3),
                                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                     "frac": round(clear_bytes / (clear_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 6),
                                     "algorithmic_bytes": clear_bytes}},
        "poa_hat_by_C": per_C,
        "roofline": roofline,
        "score_batch": score,
        "policies": pol,
        "cache_policies": cache_pol,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def runner_rows(scorings, W):
    return scorings // W


if __name__ == "__main__":
    main()
