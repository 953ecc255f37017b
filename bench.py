"""Benchmark of the KV-aware routing hot path on one MI355X.

Headline (one step = one pass of the whole path over the largest workload):
the saturation / overload-controller sweep -- 256 traces of 2,048 requests, 16
workers, 10,240 routing episodes (C in 8..1024 x 5 overlap weights x 256
seeds, the load controller on) -- block-hash chains of every trace, every
episode, and the PoA-hat windows and per-episode ratios.  The episodes run in
one launch on a fixed set of episode workspaces that the workgroups reuse.
Inputs (tokens, offsets, parameters) are resident in HBM before timing.

Also measured in the same run, each with the oracle's results compared
element by element on the episodes the oracle ran:
  * the 1P/5D-shaped sweep (320 episodes, W = 6), consecutive steps
    overlapped on two streams, every episode checked against the oracle;
  * the batched scoring kernel on 65,536 requests x 64 workers with 2^20-slot
    per-worker tables (1,024 sampled requests against the oracle), and the
    global-index scorer on the same key sets;
  * the single tiny episode (W = 4, 64 requests), against the oracle;
  * the long-context multi-turn traces (128 episodes, W = 32) under LRU, and
    under frequency eviction and memory tiers on 16 of them;
  * the selection policies on the 1P/5D-shaped traces.
The CPU oracle's rate on a bounded sample of the headline workload is
reported as cpu_baseline.

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
LINE_RATE_PEAK = 8.0e12 / 128.0        # random 128-byte lines per second at 8 TB/s
PROFILE_DIR = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = {
    "episode_kernel": ["paper_2606_17081_amd/csrc/episode.hip", "paper_2606_17081_amd/csrc/rk_internal.h"],
    "score_kernel": ["paper_2606_17081_amd/csrc/score.hip", "paper_2606_17081_amd/csrc/rk_internal.h"],
    "score_index_kernel": ["paper_2606_17081_amd/csrc/index.hip", "paper_2606_17081_amd/csrc/rk_internal.h"],
    "poa_window_kernel": ["paper_2606_17081_amd/csrc/poa.hip", "paper_2606_17081_amd/csrc/rk_internal.h"],
    "block_fnv_kernel": ["paper_2606_17081_amd/csrc/abi.hip", "paper_2606_17081_amd/csrc/rk_internal.h"],
}
COUNTER_LEVEL = ("TCC_EA0 read/write bytes (L2 egress to the memory fabric): Infinity Cache hits are "
                 "counted, so the figure is an upper bound on HBM bytes")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_digest(kernel: str) -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """Memory traffic per launch from the committed rocprofv3 counter summary,
    if it was taken on the current kernel source; else None."""
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


def cpu_info(threads: int) -> dict:
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        aff = len(os.sched_getaffinity(0))
    except AttributeError:
        aff = os.cpu_count() or 1
    return {"cores": threads, "nproc": os.cpu_count(), "affinity": aff, "cpu_model": model}


def oracle_threads() -> int:
    """Threads for the oracle: the CPUs this process may run on, at most 16 (the
    host share of one GPU)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


# ---------------------------------------------------------------- byte models

def logical_probes(runner) -> float:
    """Sum over routes and workers of o_ij + [o_ij < P_i]: the table lookups a
    first-miss scan makes (the blocks found cached plus the one miss)."""
    torch = runner.torch
    n = runner.n_rows
    ov = runner.overlap[:n]
    P = runner.route_blocks[:n].unsqueeze(1)
    return float((ov.to(torch.int64).sum() + (ov < P).to(torch.int64).sum()).item())


def episode_survey_bytes(runner) -> dict:
    """The workload's algorithmic bytes per episode launch, each access at its
    natural width: 8 B per logical probe, 24 B per prompt block of a route (the
    chain hash and key of a touch or insert, the stamp and the log record), 20 B
    per eviction (log record, stamp read and write, key), plus the outputs."""
    n = runner.n_rows
    W = runner.W
    probes = logical_probes(runner)
    sumP = float(runner.route_blocks[:n].to(runner.torch.int64).sum().item())
    ev = float(runner.evict_count[:n].to(runner.torch.int64).sum().item())
    outs = n * (8 * W + 28)
    return {"bytes": 8.0 * probes + 24.0 * sumP + 20.0 * ev + outs, "logical_probes": probes,
            "prompt_blocks": sumP, "evictions": ev}


def episode_kernel_bytes(runner) -> float:
    """Bytes the kernel's own algorithm must move per launch (no cache-line
    rounding): per route and worker a binary search for the first miss,
    ceil(log2(P + 1)) keys of 8 B; outputs; the route's first chain hash
    compared with those of its batch; on a worker that evicts during the
    episode the touch of P blocks (28 B) and insert of P - o keys (8 B), on one
    that never evicts only the P - o missing blocks (16 B each); 20 B per
    eviction."""
    W = runner.W
    n = runner.n_rows
    P = runner.route_blocks[:n].cpu().numpy().astype(np.float64)
    sig = runner.route_worker[:n].cpu().numpy()
    ov = runner.overlap[:n].cpu().numpy()
    o_sig = ov[np.arange(n), sig].astype(np.float64)
    ev = runner.evict_count[:n].cpu().numpy().astype(np.float64)
    probes = np.ceil(np.log2(P + 1.0))
    evicting = np.zeros(n, bool)
    for (r0, nr, _, _) in runner.rows:
        sl = slice(r0, r0 + nr)
        ws = np.unique(sig[sl][ev[sl] > 0])
        if ws.size:
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
    union must see: M_i + [M_i < P_i] positions, M_i = max_j o_ij."""
    B, W = inst.B, inst.W
    P = np.diff(inst.chain_off).astype(np.float64)
    M = overlap.max(axis=1).astype(np.float64) if W > 0 else np.zeros(B)
    index = 16.0 * np.sum(M + (M < P))
    chains = inst.chains.size * 8
    offs = (B + 1) * 8 + W * 4
    outs = B * W * (4 + 4) + B * 4
    return float(index + chains + offs + outs)


def roofline(kernel, workload, alg_bytes, ms, **extra):
    achieved = alg_bytes / (ms * 1e-3) / 1e9
    out = {"kernel": kernel, "bound": "hbm", "achieved": round(achieved, 3), "peak": HBM_PEAK_GBS, "unit": "GB/s",
           "frac": round(achieved / HBM_PEAK_GBS, 6), "traffic": measured_traffic(kernel, workload),
           "algorithmic_bytes": alg_bytes, "avg_ms": round(ms, 4)}
    out.update(extra)
    return out


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
    events on the launching stream around all of them."""
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(n):
        fn()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / n


# ---------------------------------------------------------------- parity with the oracle

REL = 1e-9


def compare_episode(g: dict, o: dict, poa_ref: dict):
    """First difference between a GPU episode and the oracle's, or None: routes,
    turns, steps, prompt lengths, evictions and their digests, last hashes,
    overlaps and costs bit for bit; totals exactly; window sums and PoA-hat
    within 1e-9 relative."""
    n = len(o["route_worker"])
    if len(g["route_worker"]) != n:
        return f"{len(g['route_worker'])} routes, oracle {n}"
    for k in ("route_turn", "route_worker", "route_step", "route_blocks", "evict_count", "evict_digest",
              "last_hash"):
        bad = np.nonzero(np.asarray(g[k]) != np.asarray(o[k]))[0]
        if bad.size:
            return f"{k} differs first at route {int(bad[0])}"
    if not np.array_equal(g["overlap"], o["overlap"]):
        return "overlap"
    if "cost" in g and not np.array_equal(g["cost"].view(np.uint32), o["cost"].view(np.uint32)):
        return "cost bits"
    if not np.array_equal(g["totals"], o["totals"]):
        return f"totals {g['totals'].tolist()} vs {o['totals'].tolist()}"
    for k in ("selfish", "coordinated"):
        if not np.allclose(g[k], poa_ref[k], rtol=REL, atol=0.0):
            return k
    if not abs(g["poa_hat"] - poa_ref["poa_hat"]) <= REL * abs(poa_ref["poa_hat"]):
        return "poa_hat"
    return None


def run_oracle(workload, specs, threads, keep=True):
    """The CPU oracle over the given episodes: each trace hashed once, then
    every episode simulated and its PoA-hat windows solved, threads across
    traces and episodes.  Returns (seconds, routes, {episode index: outputs})."""
    from concurrent.futures import ThreadPoolExecutor
    from oracle import oracle as O
    from paper_2606_17081_amd.workload import POA_PARAMS
    seeds = sorted({sp.seed for _, sp in specs})
    # longest first: the PoA-hat of the widest windows dominates
    order = sorted(specs, key=lambda es: -es[1].concurrency)
    t0 = time.perf_counter()
    with ThreadPoolExecutor(max_workers=threads) as ex:
        chains = dict(zip(seeds, ex.map(lambda s: O.trace_chains(workload.traces[s]), seeds)))

        def one(es):
            e, sp = es
            out = O.simulate_trace(workload.W, workload.cache_blocks, sp, workload.traces[sp.seed], chains[sp.seed])
            ref = O.episode_poa(out, workload.W, sp.concurrency, POA_PARAMS)
            return e, out, ref
        res = list(ex.map(one, order))
    dt = time.perf_counter() - t0
    routes = sum(len(out["route_worker"]) for _, out, _ in res)
    return dt, routes, ({e: (out, ref) for e, out, ref in res} if keep else {})


def check_parity(runner, oracle_out: dict, label: str) -> dict:
    """Compare every episode the oracle ran with the GPU runner's results."""
    bad = []
    for e, (out, ref) in sorted(oracle_out.items()):
        why = compare_episode(runner.episode_results(e), out, ref)
        if why is not None:
            sp = runner.episodes[e]
            bad.append(f"episode {e} (seed {sp.seed}, C {sp.concurrency}, w_ov {sp.w_ov}): {why}")
    if bad:
        log(f"PARITY MISMATCH in {label}: {len(bad)} episodes; first: {bad[:3]}")
    return {"episodes_checked": len(oracle_out), "mismatches": len(bad), "first": bad[:3]}


# ---------------------------------------------------------------- legs

def saturation_bench(torch, rk, wl, stream, steps, warmup, slots, pipeline=True):
    """The headline: 10,240 saturation / controller episodes per step.  With
    pipeline, two runners take turns so that consecutive steps overlap: step
    k's episodes run on the main stream while a second stream computes step
    k-1's PoA-hat and hashes step k+1's traces; each step still does all of
    its work inside the timed region."""
    from paper_2606_17081_amd.episodes import EpisodeRunner
    log("generating the saturation sweep (256 traces of 2,048 requests)")
    w = wl.saturation_workload()
    runners = [EpisodeRunner(w, keep_cost=True, ws_slots=slots) for _ in range(2 if pipeline else 1)]
    r = runners[0]
    torch.cuda.synchronize()
    log(f"{len(r.episodes)} episodes, {r.n_rows} routes, {r.n_windows} PoA windows, {slots} episode workspaces "
        f"({r.workspace.numel() / 1e9:.1f} GB per runner, {len(runners)} runners); warmup {warmup}")
    for _ in range(max(1, warmup)):
        for x in runners:
            x.step(stream=stream)
    torch.cuda.synchronize()
    assert rk.device_status(reset=True) == 0
    E, n = len(r.episodes), r.n_rows
    ref_poa = r.poa_hat[:E].clone()
    ref_route = r.route_worker[:n].clone()
    side = torch.cuda.Stream() if pipeline else stream
    t_sim = KernelTimer(torch, stream)
    t_hash, t_poa = KernelTimer(torch, side), KernelTimer(torch, side)
    e_sim = [None] * steps

    def prepare(k):
        x = runners[k % len(runners)]
        if pipeline and k >= 2:
            side.wait_event(e_sim[k - 2])
        with t_hash:
            x.hash(stream=side)
        ready = torch.cuda.Event()
        ready.record(side)
        return ready

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ready = prepare(0)
    for k in range(steps):
        x = runners[k % len(runners)]
        stream.wait_event(ready)
        with t_sim:
            x.simulate(stream=stream)
        done = torch.cuda.Event()
        done.record(stream)
        e_sim[k] = done
        if pipeline and k + 1 < steps:
            ready = prepare(k + 1)
        side.wait_event(done)
        with t_poa:
            x.poa(stream=side)
        if not pipeline and k + 1 < steps:
            ready = prepare(k + 1)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    assert rk.device_status(reset=True) == 0
    for x in runners[: min(len(runners), steps)]:
        assert torch.equal(x.poa_hat[:E], ref_poa), "timed steps differ from the warmup step (PoA-hat)"
        assert torch.equal(x.route_worker[:n], ref_route), "timed steps differ from the warmup step (routes)"
    del runners[1:]
    ms_step = wall * 1e3 / steps
    stage = dict(hash=t_hash.mean_ms(), simulate=t_sim.mean_ms(), poa=t_poa.mean_ms())
    log(f"saturation step {ms_step:.2f} ms; stages {stage}")
    sv = episode_survey_bytes(r)
    kb = episode_kernel_bytes(r)
    sim_s = stage["simulate"] * 1e-3
    poa_hat = r.poa_hat[:E].cpu().numpy()
    tot = r.totals[:E].cpu().numpy()
    per = {}
    for C in wl.SATURATION_C:
        for wv in wl.SATURATION_WOV:
            es = [e for e, sp in enumerate(r.episodes) if sp.concurrency == C and sp.w_ov == wv]
            v = poa_hat[es]
            per[f"C={C} w_ov={wv:g}"] = {"poa_hat": [round(float(v.mean()), 6), round(float(v.std()), 6)],
                                         "ctrl_routes_share": round(float(tot[es, 3].sum() / (len(es) * 2048)), 4)}
    res = {
        "workload": "saturation/controller sweep: W=16 workers, 2048 requests per episode, lognormal(ln 2048, 1.2) "
                    "tokens in [128, 16384], C in {8..1024} x w_ov in {0, .25, .5, 1, 2} x 256 seeds = 10240 "
                    "episodes, load controller (w_ov -> 0.25 above 0.9 of cap over 128 routes); "
                    "hash + episodes + PoA-hat",
        "episodes": E, "routes": n, "scorings_per_step": n * r.W,
        "ms_per_step": round(ms_step, 4),
        "stage_ms": {k: round(v, 4) for k, v in stage.items()},
        "episode_workspaces": slots,
        "pipeline": ("two runners take turns: step k's episodes on the main stream while the second stream runs "
                     "step k-1's PoA-hat and hashes step k+1's traces (stage times measured under that overlap); "
                     "the timed steps' PoA-hat and routes are checked against the warmup step")
        if pipeline else "one stream: hash, episodes, PoA-hat",
        "roofline": roofline("episode_kernel", "saturation", sv["bytes"], stage["simulate"],
                             byte_model="survey: 8 B per logical probe sum(o + [o < P]), 24 B per prompt block, "
                                        "20 B per eviction, outputs",
                             kernel_model_bytes=kb,
                             kernel_model_frac=round(kb / sim_s / 1e9 / HBM_PEAK_GBS, 6),
                             counter_level=COUNTER_LEVEL),
        "probe_rate": {"logical_probes": sv["logical_probes"], "per_s": sv["logical_probes"] / sim_s,
                       "peak_lines_per_s": LINE_RATE_PEAK, "frac": round(sv["logical_probes"] / sim_s / LINE_RATE_PEAK, 6)},
        "evictions_per_step": sv["evictions"],
        "by_C_and_w_ov": per,
    }
    return r, w, res


def tiny_bench(torch, rk, wl, stream, steps, oracle=True):
    """The single tiny episode (W = 4, 64 requests, C = 8): one step = hash +
    episode + PoA-hat, timed over back-to-back steps; the oracle runs the same
    episode and every output is compared."""
    from paper_2606_17081_amd.episodes import EpisodeRunner
    w = wl.tiny_workload()
    r = EpisodeRunner(w, keep_cost=True)
    for _ in range(3):
        r.step(stream=stream)
    n = max(steps, 20)
    ms = burst_ms(torch, stream, lambda: r.step(stream=stream), n)
    assert rk.device_status(reset=True) == 0
    res = {"workload": "tiny: one episode, W=4 workers, 64 requests of 4..32 blocks, 8 prefix groups, cache 256, "
                       "cap 512, C=8; hash + episode + PoA-hat",
           "episodes": 1, "routes": r.n_rows, "ms_per_step": round(ms, 4),
           "scorings_per_s": r.n_rows * w.W / (ms * 1e-3), "episodes_per_s": 1.0 / (ms * 1e-3),
           "poa_hat": float(r.poa_hat[0].item())}
    if oracle:
        dt, routes, outs = run_oracle(w, list(enumerate(r.episodes)), 1)
        res["oracle"] = {"seconds": round(dt, 6), "scorings_per_s": routes * w.W / dt, "threads": 1}
        res["parity"] = check_parity(r, outs, "tiny")
    log(f"tiny step {ms:.4f} ms")
    return res


def sweep_bench(torch, rk, wl, stream, steps, warmup):
    """The 1P/5D-shaped sweep (320 episodes): consecutive steps overlap on two
    streams (two runners take turns)."""
    from paper_2606_17081_amd.episodes import EpisodeRunner
    log("generating the 1P/5D-shaped sweep (64 traces of 4,096 requests)")
    w = wl.sweep70b_workload()
    runners = [EpisodeRunner(w, keep_cost=True) for _ in range(2)]
    runner = runners[0]
    torch.cuda.synchronize()
    for _ in range(max(1, warmup)):
        for r in runners:
            r.step()
    torch.cuda.synchronize()
    assert rk.device_status(reset=True) == 0
    E0, n0 = len(runner.episodes), runner.n_rows
    ref_poa = runner.poa_hat[:E0].clone()
    ref_route = runner.route_worker[:n0].clone()

    side = torch.cuda.Stream()
    t_sim = KernelTimer(torch, stream)
    t_hash, t_poa = KernelTimer(torch, side), KernelTimer(torch, side)
    e_sim = [None] * steps

    def prepare(k):
        r = runners[k % 2]
        if k >= 2:
            side.wait_event(e_sim[k - 2])
        with t_hash:
            r.hash(stream=side)
        ready = torch.cuda.Event()
        ready.record(side)
        return ready

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ready = prepare(0)
    for k in range(steps):
        r = runners[k % 2]
        stream.wait_event(ready)
        with t_sim:
            r.simulate(stream=stream)
        done = torch.cuda.Event()
        done.record(stream)
        e_sim[k] = done
        if k + 1 < steps:
            ready = prepare(k + 1)
        side.wait_event(done)
        with t_poa:
            r.poa(stream=side)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    assert rk.device_status(reset=True) == 0
    for r in runners[: min(2, steps)]:
        assert torch.equal(r.poa_hat[:E0], ref_poa), "pipelined steps differ from the sequential step (PoA-hat)"
        assert torch.equal(r.route_worker[:n0], ref_route), "pipelined steps differ from the sequential step (routes)"
    ms_step = wall * 1e3 / steps
    stage = dict(hash=t_hash.mean_ms(), simulate=t_sim.mean_ms(), poa=t_poa.mean_ms())
    log(f"sweep step {ms_step:.3f} ms; stages {stage}")
    poa_hat = runner.poa_hat[:E0].cpu().numpy()
    per_C = {}
    for C in wl.SWEEP70B_C:
        v = np.array([poa_hat[e] for e, sp in enumerate(runner.episodes) if sp.concurrency == C])
        per_C[str(C)] = [round(float(v.mean()), 6), round(float(v.std()), 6)]
    sv = episode_survey_bytes(runner)
    kb = episode_kernel_bytes(runner)
    sim_s = stage["simulate"] * 1e-3
    del runners[1]
    res = {
        "workload": "sweep70b: 70B-1P/5D-shaped sweep, W=6 workers, 4096 requests per episode, "
                    "C in {32,64,128,256,512} x 64 seeds = 320 episodes; hash + episodes + PoA-hat",
        "episodes": E0, "routes": n0, "scorings_per_step": n0 * runner.W, "ms_per_step": round(ms_step, 4),
        "scorings_per_s": n0 * runner.W / (ms_step * 1e-3), "episodes_per_s": E0 / (ms_step * 1e-3),
        "stage_ms": {k: round(v, 4) for k, v in stage.items()},
        "pipeline": "two runners take turns: step k's episodes on the main stream while the second stream "
                    "runs step k-1's PoA-hat and hashes step k+1's traces",
        "roofline": roofline("episode_kernel", "sweep70b", sv["bytes"], stage["simulate"],
                             kernel_model_bytes=kb,
                             kernel_model_frac=round(kb / sim_s / 1e9 / HBM_PEAK_GBS, 6)),
        "probe_rate": {"logical_probes": sv["logical_probes"], "per_s": sv["logical_probes"] / sim_s,
                       "frac": round(sv["logical_probes"] / sim_s / LINE_RATE_PEAK, 6)},
        "poa_hat_by_C": per_C,
    }
    return runner, w, res


def index_log2_slots(n_keys: int) -> int:
    """Index slots for n_keys insertions at load <= 0.25 (2^27 slots, 2 GiB, for
    the 65,536 x 64 instance)."""
    b = 4
    while (1 << b) < 4 * n_keys:
        b += 1
    return b


def scoring_bench(torch, rk, wl, stream, steps, oracle=False):
    """The 65,536 x 64 snapshot scoring on the per-worker tables
    (rk_route_score_batch), and on the global block index
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
    ov_ref = ov.cpu().numpy()
    P = np.diff(inst.chain_off)
    probes = float(ov_ref.sum() + (ov_ref < P[:, None]).sum())
    salg = score_algorithmic_bytes(inst)
    ach = salg / (ms * 1e-3) / 1e9
    log(f"scoring (tables): {ms:.4f} ms, {inst.B * inst.W / (ms * 1e-3):.4g} scorings/s, {ach:.1f} GB/s compulsory")
    orc = None
    if oracle:
        # the oracle on every request, in contiguous ranges on the host threads (each call sorts the
        # 64 key sets itself), compared element by element
        from concurrent.futures import ThreadPoolExecutor
        from oracle import oracle as O
        threads = oracle_threads()
        cuts = np.linspace(0, inst.B, threads + 1).astype(np.int64)
        parts = [np.arange(cuts[k], cuts[k + 1]) for k in range(threads) if cuts[k + 1] > cuts[k]]
        t0 = time.perf_counter()
        with ThreadPoolExecutor(max_workers=threads) as ex:
            res = list(ex.map(lambda rows: O.score_batch(inst.chains, inst.chain_off, inst.keys, inst.key_off,
                                                         inst.active, inst.w_ov, inst.w_act, inst.w_sat, inst.cap,
                                                         rows=rows), parts))
        dt = time.perf_counter() - t0
        r_ov = np.concatenate([x[0] for x in res])
        r_co = np.concatenate([x[1] for x in res])
        r_am = np.concatenate([x[2] for x in res])
        co_ref, am_ref = co.cpu().numpy(), am.cpu().numpy()
        bad = int(((ov_ref != r_ov).any(axis=1) | (co_ref.view(np.uint32) != r_co.view(np.uint32)).any(axis=1)
                   | (am_ref != r_am)).sum())
        orc = {"sample": f"all {inst.B} requests x {inst.W} workers, in {len(parts)} ranges on {threads} threads, "
                         f"each range sorting the {inst.W} key sets", "seconds": round(dt, 3),
               "scorings_per_s": inst.B * inst.W / dt, "threads": threads}
        parity = {"requests_checked": int(inst.B), "mismatches": bad}
        log(f"scoring oracle {dt:.2f} s on all {inst.B} requests ({threads} threads); mismatches {bad}")
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
    build_ms = tb.mean_ms()
    log(f"scoring (index): {ms_i:.4f} ms; index build {build_ms:.3f} ms")
    wl_name = "scoring 65536 requests x 64 workers, 2^20-slot tables at load 0.5, chains of 16..512"
    out = {"workload": wl_name,
            "scorings_per_s": inst.B * inst.W / (ms * 1e-3), "avg_ms": round(ms, 4),
            "roofline": roofline("score_kernel", "scoring", salg, ms,
                                 byte_model="survey compulsory: every table slot, chain hash and offset once, "
                                            "the outputs", counter_level=COUNTER_LEVEL),
            "probe_rate": {"logical_probes": probes, "per_s": probes / (ms * 1e-3),
                           "frac": round(probes / (ms * 1e-3) / LINE_RATE_PEAK, 6)},
            "index": {"workload": wl_name + "; the same key sets in one global block index of "
                                            f"2^{lg} 16-byte slots (a different input layout: the per-worker "
                                            "tables are not read)",
                      "scorings_per_s": inst.B * inst.W / (ms_i * 1e-3), "avg_ms": round(ms_i, 4),
                      "index_build_ms": round(build_ms, 4),
                      "scorings_per_s_with_build": inst.B * inst.W / ((ms_i + build_ms) * 1e-3),
                      "survey_compulsory_frac": round(salg / (ms_i * 1e-3) / 1e9 / HBM_PEAK_GBS, 6),
                      "roofline": roofline("score_index_kernel", "scoring", ialg, ms_i,
                                           byte_model="own: chains, offsets, outputs and one 16-byte index "
                                                      "slot per position of the union's first-miss scan")}}
    if orc is not None:
        out["oracle"] = orc
        out["parity"] = parity
    return out


def policy_bench(torch, rk, wl, stream, steps):
    """The 1P/5D-shaped traces under every selection policy: 16 seeds x 5
    concurrency levels x (5 policies + the regime controller) in one launch."""
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


def _cache_stats(r, E):
    tot = r.totals[:E].cpu().numpy()
    poa = r.poa_hat[:E].cpu().numpy()
    res = {"poa_hat": [round(float(poa.mean()), 6), round(float(poa.std()), 6)],
           "recomputed_blocks_total": int(tot[:, 0].sum()),
           "recomputed_blocks_per_episode": round(float(tot[:, 0].mean()), 1),
           "reused_blocks_per_episode": round(float(tot[:, 6].mean()), 1),
           "evicted_blocks_per_episode": round(float(tot[:, 1].mean()), 1)}
    if r.tier_overlap is not None:
        n = r.n_rows
        sig = r.route_worker[:n].long()
        rows = r.torch.arange(n, device=sig.device)
        t = r.tier_overlap[:n][rows, sig].long().cpu().numpy()
        o = r.overlap[:n][rows, sig].long().cpu().numpy()
        g1, g2, g3 = t[:, 0].sum(), (t[:, 1] - t[:, 0]).sum(), (o - t[:, 1]).sum()
        res["reused_blocks_share_G1_G2_G3"] = [round(float(x / max(o.sum(), 1)), 4) for x in (g1, g2, g3)]
    return res


def multiturn_bench(torch, rk, wl, stream, steps, seeds=128, variant_seeds=16):
    """The long-context multi-turn workload: 128 episodes (W = 32, 512
    conversations, 16,384-block caches, C = 256) under LRU in one launch,
    then frequency eviction (decay every 4 and 64 steps) and LRU with memory
    tiers (G1 = G2 = 4,096 blocks, G3 the other 8,192; weights 0, 0.25, 0.5)
    on the first 16 traces."""
    from paper_2606_17081_amd.episodes import EpisodeRunner
    log(f"generating {seeds} multi-turn traces")
    base = wl.multiturn_workload(seeds=range(seeds))
    r = EpisodeRunner(base, keep_cost=True)
    r.step()
    torch.cuda.synchronize()
    ts, th, tp = KernelTimer(torch, stream), KernelTimer(torch, stream), KernelTimer(torch, stream)
    for _ in range(max(1, steps // 4)):
        with th:
            r.hash()
        with ts:
            r.simulate()
        with tp:
            r.poa()
    torch.cuda.synchronize()
    assert rk.device_status(reset=True) == 0
    E = len(base.episodes)
    ms = ts.mean_ms() + th.mean_ms() + tp.mean_ms()
    lru = {"episodes": E, "routes": r.n_rows, "step_ms": round(ms, 3),
           "stage_ms": {"hash": round(th.mean_ms(), 4), "simulate": round(ts.mean_ms(), 4),
                        "poa": round(tp.mean_ms(), 4)},
           "episodes_per_s": round(E / (ms * 1e-3), 1), "routes_per_s": float(r.n_rows / (ms * 1e-3)),
           "scorings_per_s": float(r.n_rows * r.W / (ms * 1e-3)),
           "occupancy": f"{E} episodes, one 256-thread workgroup each, on 256 CUs"}
    lru.update(_cache_stats(r, E))
    log(f"multi-turn LRU: {lru}")
    variants = [("frequency, decay every 4 steps", dict(evict_policy=wl.EVICT_FREQ, decay_steps=4)),
                ("frequency, decay every 64 steps", dict(evict_policy=wl.EVICT_FREQ, decay_steps=64)),
                ("lru, tiers G1/G2/G3 = 4096/4096/8192", dict(tier_g1=4096, tier_g2=4096))]
    out = {}
    sub = [sp for sp in base.episodes if sp.seed < variant_seeds]
    for name, kw in variants:
        eps = [wl.EpisodeSpec(**{**sp.__dict__, **kw}) for sp in sub]
        w = wl.Workload(base.name, W=base.W, cache_blocks=base.cache_blocks,
                        traces={s: base.traces[s] for s in range(variant_seeds)}, episodes=eps)
        rv = EpisodeRunner(w, keep_cost=False)
        rv.hash()
        rv.simulate()
        rv.poa()
        torch.cuda.synchronize()
        tv = KernelTimer(torch, stream)
        for _ in range(max(1, steps // 4)):
            with tv:
                rv.simulate()
        rv.poa()
        torch.cuda.synchronize()
        assert rk.device_status(reset=True) == 0
        res = {"episodes": len(eps), "simulate_ms": round(tv.mean_ms(), 3),
               "episodes_per_s": round(len(eps) / (tv.mean_ms() * 1e-3), 1)}
        res.update(_cache_stats(rv, len(eps)))
        log(f"multi-turn {name}: {res}")
        out[name] = res
        del rv
    return r, base, {"workload": f"long-context multi-turn traces, W=32, 512 conversations of 2..16 turns, "
                                 f"16384-block caches, cap 4096, C=256; LRU on {seeds} seeds, the other "
                                 f"eviction variants on seeds 0..{variant_seeds - 1}",
                     "lru": lru, "variants": out}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--slots", type=int, default=512, help="episode workspaces of the headline launch")
    ap.add_argument("--pipeline", action="store_true",
                    help="headline steps overlapped on two streams (PoA-hat and hashing beside the next episodes)")
    ap.add_argument("--no-pipeline", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--cpu-seeds", type=int, default=32, help="saturation seeds the oracle runs (all 40 episodes each)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only", choices=("all", "saturation", "sweep", "scoring", "policies", "multiturn", "tiny"),
                    default="all", help="profiling passes: run one leg only, without the oracle")
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
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()

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
    only = args.only
    if only == "scoring":
        print(json.dumps({"score_batch": scoring_bench(torch, rk, wl, stream, args.steps)}), flush=True)
        return
    if only == "tiny":
        print(json.dumps({"tiny": tiny_bench(torch, rk, wl, stream, args.steps, oracle=False)}), flush=True)
        return
    if only == "policies":
        print(json.dumps({"policies": policy_bench(torch, rk, wl, stream, args.steps)}), flush=True)
        return
    if only == "multiturn":
        print(json.dumps({"multiturn": multiturn_bench(torch, rk, wl, stream, args.steps)[2]}), flush=True)
        return
    if only == "sweep":
        print(json.dumps({"sweep70b": sweep_bench(torch, rk, wl, stream, args.steps, args.warmup)[2]}), flush=True)
        return

    threads = oracle_threads()
    parity = {}
    # ---- headline: the saturation / controller sweep
    r4, w4, sat = saturation_bench(torch, rk, wl, stream, args.steps, args.warmup, args.slots,
                                   pipeline=args.pipeline and not args.no_pipeline)
    if only == "saturation":
        print(json.dumps({"saturation": sat}), flush=True)
        return
    cpu = None
    if not args.no_cpu_baseline:
        seeds = list(range(args.cpu_seeds))
        specs = [(e, sp) for e, sp in enumerate(r4.episodes) if sp.seed in seeds]
        log(f"oracle on {len(specs)} saturation episodes (seeds 0..{args.cpu_seeds - 1}) with {threads} threads")
        dt, routes, outs = run_oracle(w4, specs, threads)
        parity["saturation"] = check_parity(r4, outs, "saturation")
        del outs
        full_s = dt * len(r4.episodes) / len(specs)
        cpu = {"value": routes * w4.W / dt, "unit": "scorings/s", "kind": "oracle",
               "sample": f"{len(specs)} of the 10240 saturation episodes (seeds 0..{args.cpu_seeds - 1}, every C "
                         f"and w_ov) incl. hashing their traces and the PoA-hat windows; {routes} routes in "
                         f"{dt:.2f} s",
               "extrapolated": len(specs) < len(r4.episodes),
               "full_config_seconds_extrapolated": round(full_s, 1),
               "episodes_per_s": len(specs) / dt, "seconds": round(dt, 3)}
        cpu.update(cpu_info(threads))
        log(f"oracle: {cpu['value']:.4g} scorings/s ({len(specs)} episodes in {dt:.2f} s); parity "
            f"{parity['saturation']}")
    del r4
    torch.cuda.empty_cache()

    # ---- the 1P/5D-shaped sweep, every episode against the oracle
    r2, w2, sweep = sweep_bench(torch, rk, wl, stream, args.steps, args.warmup)
    if not args.no_cpu_baseline:
        specs = list(enumerate(r2.episodes))
        log(f"oracle on all {len(specs)} sweep episodes with {threads} threads")
        dt, routes, outs = run_oracle(w2, specs, threads)
        parity["sweep70b"] = check_parity(r2, outs, "sweep70b")
        del outs
        sweep["oracle"] = {"scorings_per_s": routes * w2.W / dt, "episodes_per_s": len(specs) / dt,
                           "seconds": round(dt, 3), "threads": threads}
        log(f"sweep oracle {dt:.2f} s; parity {parity['sweep70b']}")
    del r2
    torch.cuda.empty_cache()

    score = scoring_bench(torch, rk, wl, stream, args.steps, oracle=not args.no_cpu_baseline)
    if "parity" in score:
        parity["scoring"] = score["parity"]
    torch.cuda.empty_cache()

    tiny = tiny_bench(torch, rk, wl, stream, args.steps, oracle=not args.no_cpu_baseline)
    if "parity" in tiny:
        parity["tiny"] = tiny["parity"]

    r5, w5, multi = multiturn_bench(torch, rk, wl, stream, args.steps)
    if not args.no_cpu_baseline:
        specs = list(enumerate(r5.episodes))
        log(f"oracle on all {len(specs)} multi-turn episodes with {threads} threads")
        dt, routes, outs = run_oracle(w5, specs, threads)
        parity["multiturn"] = check_parity(r5, outs, "multiturn")
        del outs
        multi["oracle"] = {"scorings_per_s": routes * w5.W / dt, "episodes_per_s": len(specs) / dt,
                           "seconds": round(dt, 3), "threads": threads}
        log(f"multi-turn oracle {dt:.2f} s; parity {parity['multiturn']}")
    del r5
    torch.cuda.empty_cache()

    pol = policy_bench(torch, rk, wl, stream, args.steps)

    ms_step = sat["ms_per_step"]
    line = {
        "metric": METRIC,
        "value": sat["scorings_per_step"] / (ms_step * 1e-3),
        "unit": "scorings/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64/i32 hashing and probes, f32 cost, f64 PoA sums",
        "data": "synthetic",
        "config": {"workload": sat["workload"], "episodes": sat["episodes"], "routes": sat["routes"],
                   "scorings_per_step": sat["scorings_per_step"]},
        "episodes_per_s": sat["episodes"] / (ms_step * 1e-3),
        "routes_per_s": sat["routes"] / (ms_step * 1e-3),
        "stage_ms": sat["stage_ms"],
        "roofline": sat["roofline"],
        "probe_rate": sat["probe_rate"],
        "cpu_baseline": cpu,
        "parity": parity,
        "saturation": {k: v for k, v in sat.items() if k not in ("roofline", "probe_rate", "stage_ms")},
        "tiny": tiny,
        "sweep70b": sweep,
        "score_batch": score,
        "multiturn": multi,
        "policies": pol,
    }
    print(json.dumps(line), flush=True)
    if any(p["mismatches"] for p in parity.values()):
        log("parity mismatches: the throughput rows are invalid")
        sys.exit(3)


if __name__ == "__main__":
    main()
