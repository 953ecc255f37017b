"""ctypes driver of the plain C oracle (``oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the routing library.  It shares no code
with the HIP path; both consume the same seeded inputs from the workload
generator.

All arrays are host numpy arrays.  The functions mirror the definitions stated
in the header of ``oracle.c`` (Section 2.2 Eq. router-cost, Section 4.3,
Section 5.1 Eq. latency-superlinear, Section 6.4 Eq. poa-estimate).
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import threading
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

CFLAGS = ["-std=c11", "-O2", "-fno-fast-math", "-ffp-contract=off", "-Wall", "-shared", "-fPIC"]


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so (plain gcc, IEEE fp32, no contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB):
                build(force=True)
            L = C.CDLL(_LIB)
            p = C.c_void_p
            i32, i64, f32, u64 = C.c_int32, C.c_int64, C.c_float, C.c_uint64
            L.orc_fnv1a64.restype = u64
            L.orc_fnv1a64.argtypes = [p, i64]
            L.orc_splitmix64.restype = u64
            L.orc_splitmix64.argtypes = [u64]
            L.orc_block_fnv.restype = u64
            L.orc_block_fnv.argtypes = [p]
            L.orc_chain_step.restype = u64
            L.orc_chain_step.argtypes = [u64, u64]
            L.orc_hash_chains.restype = C.c_int
            L.orc_hash_chains.argtypes = [i64, p, p, p, p, p]
            L.orc_route_cost.restype = f32
            L.orc_route_cost.argtypes = [f32, f32, f32, i32, i32, i32, i64]
            L.orc_score_batch.restype = C.c_int
            L.orc_score_batch.argtypes = [i32, i32, p, p, p, p, p, f32, f32, f32, i32, p, p, p]
            L.orc_simulate_episode.restype = C.c_int
            L.orc_simulate_episode.argtypes = [
                i32, i32, i32, i32, f32, f32, f32, i32, i32, f32, i32, i32, i32,
                i32, f32, p,
                p, p, p, p,
                i32, i32,
                i32, i32, p, p,
                i32, p, p, p, p,
                p, p, p, p, p, p, p, p, p, p,
                p, p, p, i64, p]
            L.orc_exp_neg.restype = f32
            L.orc_exp_neg.argtypes = [f32]
            L.orc_select.restype = i32
            L.orc_select.argtypes = [i32, f32, i32, p, i64, C.c_uint32, C.c_uint32]
            L.orc_latency.restype = C.c_double
            L.orc_latency.argtypes = [p, p, i64]
            L.orc_regime_step.restype = C.c_int
            L.orc_regime_step.argtypes = [p, p, C.c_double, i64, p, p, p, p]
            L.orc_poa_matrix.restype = C.c_int
            L.orc_poa_matrix.argtypes = [i32, i32, p, p, p, f32, f32, f32, i32, i32, f32, p, p]
            L.orc_poa_window.restype = C.c_int
            L.orc_poa_window.argtypes = [i32, i32, p, p, p, f32, f32, f32, i32, i32, f32, i32,
                                         p, p, p]
            L.orc_poa_windows.restype = C.c_int
            L.orc_poa_windows.argtypes = [i64, i32, i32, p, p, p, f32, f32, f32, i32, i32, f32,
                                          i32, p, p]
            _lib = L
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else C.c_void_p(a.ctypes.data)


def _c(a, dt) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dt)


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what} failed with code {rc}")


# ------------------------------------------------------------------ hashing

def fnv1a64(data: bytes) -> int:
    buf = np.frombuffer(bytes(data), dtype=np.uint8) if len(data) else np.zeros(1, np.uint8)
    return int(lib().orc_fnv1a64(_ptr(buf), len(data)))


def splitmix64(x: int) -> int:
    return int(lib().orc_splitmix64(C.c_uint64(x & 0xFFFFFFFFFFFFFFFF)))


def block_fnv(tokens16) -> int:
    t = _c(tokens16, np.int32)
    assert t.shape == (16,)
    return int(lib().orc_block_fnv(_ptr(t)))


def chain_step(prev: int, f: int) -> int:
    return int(lib().orc_chain_step(C.c_uint64(prev), C.c_uint64(f)))


def hash_chains(tokens, tok_off, nblocks, chain_off=None) -> np.ndarray:
    tokens = _c(tokens, np.int32)
    tok_off = _c(tok_off, np.int64)
    nblocks = _c(nblocks, np.int32)
    if chain_off is None:
        chain_off = np.zeros(nblocks.shape[0] + 1, np.int64)
        np.cumsum(nblocks, out=chain_off[1:])
    chain_off = _c(chain_off, np.int64)
    out = np.zeros(int(chain_off[-1]), np.uint64)
    rc = lib().orc_hash_chains(nblocks.shape[0], _ptr(tokens if tokens.size else np.zeros(1, np.int32)),
                               _ptr(tok_off), _ptr(nblocks), _ptr(chain_off),
                               _ptr(out if out.size else np.zeros(1, np.uint64)))
    _check(rc, "hash_chains")
    return out


def trace_chains(trace) -> np.ndarray:
    return hash_chains(trace.tokens, trace.tok_off, trace.chain_blocks, trace.chain_off)


# ------------------------------------------------------------------ scoring

def route_cost(w_ov, w_act, w_sat, cap, P, o, A) -> np.float32:
    return np.float32(lib().orc_route_cost(w_ov, w_act, w_sat, cap, P, o, A))


def score_batch(chains, chain_off, keys, key_off, active, w_ov=1.0, w_act=0.5, w_sat=4.0,
                cap=32768, rows: Optional[Sequence[int]] = None):
    """Overlap/cost per (request, worker) and argmin per request.

    ``rows`` restricts the evaluation to a subset of requests (sampled checks
    at full size); results are returned for those rows only.
    """
    chains = _c(chains, np.uint64)
    chain_off = _c(chain_off, np.int64)
    keys = _c(keys, np.uint64)
    key_off = _c(key_off, np.int64)
    active = _c(active, np.int32)
    W = active.shape[0]
    if rows is not None:
        rows = np.asarray(rows, np.int64)
        lens = chain_off[rows + 1] - chain_off[rows]
        sub_off = np.zeros(rows.shape[0] + 1, np.int64)
        np.cumsum(lens, out=sub_off[1:])
        sub = np.concatenate([chains[chain_off[r]:chain_off[r + 1]] for r in rows]) \
            if rows.size else np.zeros(0, np.uint64)
        chains, chain_off = _c(sub, np.uint64), sub_off
    B = chain_off.shape[0] - 1
    ov = np.zeros((B, W), np.int32)
    co = np.zeros((B, W), np.float32)
    am = np.zeros(B, np.int32)
    dummy = np.zeros(1, np.uint64)
    rc = lib().orc_score_batch(B, W, _ptr(chains if chains.size else dummy), _ptr(chain_off),
                               _ptr(keys if keys.size else dummy), _ptr(key_off), _ptr(active),
                               w_ov, w_act, w_sat, cap, _ptr(ov), _ptr(co), _ptr(am))
    _check(rc, "score_batch")
    return ov, co, am


# ------------------------------------------------------------------ episodes

def exp_neg(x: float) -> float:
    """The oracle's float exp for x <= 0 (Cody-Waite reduction, Taylor degree 7)."""
    return float(lib().orc_exp_neg(float(x)))


def select(policy: int, tau: float, costs, t: int = 0, r0: int = 0, r1: int = 0) -> int:
    """Worker a route with these float costs is sent to under a selection policy."""
    c = _c(costs, np.float32)
    return int(lib().orc_select(int(policy), float(tau), int(c.shape[0]), _ptr(c), int(t), int(r0), int(r1)))


def regime_arrays(regime=None):
    """(fp64, int32, fp32) parameter arrays of the regime controller."""
    from paper_2606_17081_amd.workload import REGIME_PARAMS
    r = dict(REGIME_PARAMS if regime is None else regime)
    rd = np.array([r["alpha"], r["theta1"], r["theta2"], r["eps"], r["a"], r["b"], r["d"]], np.float64)
    ri = np.array([r["k"], r["beta"], r["n_sat"]], np.int32)
    rf = np.array(list(r["tau"]) + list(r["w_ov"]), np.float32)
    return rd, ri, rf


def latency(n: int, regime=None) -> float:
    rd, ri, _ = regime_arrays(regime)
    return float(lib().orc_latency(_ptr(rd), _ptr(ri), int(n)))


def regime_step(lat: float, sample: int, state, regime=None):
    """One sample of the regime controller; state = [ewma, regime, up, down] is updated."""
    rd, ri, _ = regime_arrays(regime)
    e = np.array([state[0]], np.float64)
    g = np.array(state[1:4], np.int32)
    moved = lib().orc_regime_step(_ptr(rd), _ptr(ri), float(lat), int(sample), _ptr(e), _ptr(g[0:]),
                                  C.c_void_p(g.ctypes.data + 4), C.c_void_p(g.ctypes.data + 8))
    state[:] = [float(e[0]), int(g[0]), int(g[1]), int(g[2])]
    return int(moved)


def simulate_episode(W, cache_blocks, spec, turn_off, turn_blocks, chain_off, chains,
                     dump: bool = False, evicted_cap: int = 0, rand=None, regime=None) -> Dict[str, np.ndarray]:
    """One routing episode; arrays must be rebased (turn_off[0] == chain_off[0] == 0).
    rand: two uint32 words per route (the stochastic policies' draws); drawn by
    workload.route_rand when not given."""
    turn_off = _c(turn_off, np.int64)
    turn_blocks = _c(turn_blocks, np.int32)
    chain_off = _c(chain_off, np.int64)
    chains = _c(chains, np.uint64)
    assert turn_off[0] == 0 and chain_off[0] == 0
    n_conv = turn_off.shape[0] - 1
    n = int(turn_off[-1])
    out = dict(
        route_turn=np.zeros(n, np.int32), route_worker=np.zeros(n, np.int32),
        route_step=np.zeros(n, np.int32), route_blocks=np.zeros(n, np.int32),
        overlap=np.zeros((n, W), np.int32), cost=np.zeros((n, W), np.float32),
        evict_count=np.zeros(n, np.int32), evict_digest=np.zeros(n, np.uint64),
        last_hash=np.zeros(n, np.uint64), totals=np.zeros(8, np.int64), route_regime=np.zeros(n, np.int32),
        tier_overlap=np.zeros((n, W, 2), np.int32))
    tw = np.ascontiguousarray(getattr(spec, "tier_w", (0.0, 0.25, 0.5)), dtype=np.float32)
    policy = int(getattr(spec, "policy", 0))
    tau = float(getattr(spec, "tau", 0.0))
    rd, ri, rf = regime_arrays(regime)
    if rand is None:
        if policy in (1, 3, 4) or (spec.controller == 2 and np.any(rf[:3] > 0)):   # draws per route
            from paper_2606_17081_amd.workload import route_rand
            rand = route_rand(spec, n)
        else:
            rand = np.zeros(2 * n, np.uint32)
    rand = _c(rand, np.uint32)
    assert rand.shape[0] >= 2 * n
    fk = np.zeros((W, cache_blocks), np.uint64) if dump else None
    fc = np.zeros(W, np.int32) if dump else None
    ek = np.zeros(max(evicted_cap, 1), np.uint64) if evicted_cap > 0 else None
    ne = np.zeros(1, np.int64)
    g = lambda a: _ptr(a if a.size else np.zeros(1, a.dtype))
    rc = lib().orc_simulate_episode(
        W, cache_blocks, spec.hold_steps, spec.routes_per_step,
        spec.w_ov, spec.w_act, spec.w_sat, spec.cap,
        spec.controller, spec.ctrl_w_ov, spec.ctrl_window, spec.ctrl_num, spec.ctrl_den,
        policy, tau, g(rand),
        _ptr(rd), _ptr(ri), _ptr(rf), g(out["route_regime"]),
        int(getattr(spec, "evict_policy", 0)), int(getattr(spec, "decay_steps", 0)),
        int(getattr(spec, "tier_g1", 0)), int(getattr(spec, "tier_g2", 0)), _ptr(tw), g(out["tier_overlap"]),
        n_conv, _ptr(turn_off), g(turn_blocks), _ptr(chain_off), g(chains),
        g(out["route_turn"]), g(out["route_worker"]), g(out["route_step"]),
        g(out["route_blocks"]), g(out["overlap"]), g(out["cost"]),
        g(out["evict_count"]), g(out["evict_digest"]), g(out["last_hash"]), _ptr(out["totals"]),
        _ptr(fk), _ptr(fc), _ptr(ek), int(evicted_cap), _ptr(ne))
    _check(rc, "simulate_episode")
    if dump:
        out["final_keys"] = [fk[j, :fc[j]].copy() for j in range(W)]
    if ek is not None:
        out["evicted_keys"] = ek[:min(int(ne[0]), evicted_cap)].copy()
    return out


def simulate_trace(W, cache_blocks, spec, trace, chains=None, **kw):
    """Episode over a whole trace (hashing it first unless chains are given)."""
    if chains is None:
        chains = trace_chains(trace)
    return simulate_episode(W, cache_blocks, spec, trace.turn_off, trace.turn_blocks,
                            trace.chain_off, chains, **kw)


# ------------------------------------------------------------------ PoA-hat

def poa_matrix(worker, overlap, blocks, W, a, b, d, beta, C_cap, w_c):
    worker = _c(worker, np.int32)
    overlap = _c(overlap, np.int32)
    blocks = _c(blocks, np.int32)
    m = worker.shape[0]
    c = np.zeros((m, W), np.float32)
    n = np.zeros(W, np.int32)
    g = lambda a_: _ptr(a_ if a_.size else np.zeros(1, a_.dtype))
    rc = lib().orc_poa_matrix(m, W, g(worker), g(overlap), g(blocks), a, b, d, beta, C_cap, w_c,
                              g(c), _ptr(n))
    _check(rc, "poa_matrix")
    return c, n


def poa_window(worker, overlap, blocks, W, a, b, d, beta, C_cap, w_c, K=0):
    """(selfish, coordinated, opt_worker) of one window."""
    worker = _c(worker, np.int32)
    overlap = _c(overlap, np.int32)
    blocks = _c(blocks, np.int32)
    m = worker.shape[0]
    s = np.zeros(1, np.float64)
    o = np.zeros(1, np.float64)
    ow = np.zeros(max(m, 1), np.int32)
    g = lambda a_: _ptr(a_ if a_.size else np.zeros(1, a_.dtype))
    rc = lib().orc_poa_window(m, W, g(worker), g(overlap), g(blocks), a, b, d, beta, C_cap, w_c,
                              K, _ptr(s), _ptr(o), _ptr(ow))
    _check(rc, "poa_window")
    return float(s[0]), float(o[0]), ow[:m].copy()


def poa_windows(worker, overlap, blocks, W, window, a, b, d, beta, C_cap, w_c, K=0):
    worker = _c(worker, np.int32)
    overlap = _c(overlap, np.int32)
    blocks = _c(blocks, np.int32)
    n = worker.shape[0]
    nw = (n + window - 1) // window
    s = np.zeros(max(nw, 1), np.float64)
    o = np.zeros(max(nw, 1), np.float64)
    g = lambda a_: _ptr(a_ if a_.size else np.zeros(1, a_.dtype))
    rc = lib().orc_poa_windows(n, W, window, g(worker), g(overlap), g(blocks), a, b, d, beta,
                               C_cap, w_c, K, _ptr(s), _ptr(o))
    _check(rc, "poa_windows")
    return s[:nw].copy(), o[:nw].copy()


def episode_poa(out, W, window, params) -> Dict[str, object]:
    """Per-window sums and the episode's PoA-hat = sum selfish / sum coordinated."""
    s, o = poa_windows(out["route_worker"], out["overlap"], out["route_blocks"], W, window,
                       params["a"], params["b"], params["d"], params["beta"], params["C_cap"],
                       params["w_c"])
    tot_s, tot_o = float(s.sum()), float(o.sum())
    return dict(selfish=s, coordinated=o, poa_hat=(tot_s / tot_o) if tot_o != 0 else float("nan"))


# ------------------------------------------------------- threaded driver

def run_episodes(W, cache_blocks, jobs, threads: int):
    """Run (spec, trace, chains) jobs on a thread pool; ctypes releases the GIL."""
    def one(job):
        spec, trace, chains = job
        return simulate_trace(W, cache_blocks, spec, trace, chains)
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return list(ex.map(one, jobs))
