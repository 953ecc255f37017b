"""Seeded synthetic workloads for KV-aware routing (inputs only).

This module draws every input that the routing path and its CPU oracle both
consume: token streams for the episode workloads, and key sets plus block-hash
chains for the snapshot-scoring workload.  It contains none of the method's own
arithmetic (no block hashing, no cost, no cache policy): it only produces
random integers with numpy's PCG64 generator, so that the GPU path and the
oracle can be compared on identical inputs.

Workload shapes follow the paper's setting (requests sharing a few prompt
prefixes, a concurrency grid, a small pool of decode workers; Section 7.4 and
Section 7.7) at the sizes of the five named workloads:

* ``tiny``      4 workers, 64 requests, 8 prefix groups (single episode)
* ``sweep70b``  6 workers (the 1P/5D topology), 4,096 requests, C in 32..512
* ``scoring``   65,536 requests x 64 workers, tables of 2^20 slots
* ``saturation`` 16 workers, 2,048 requests, C in 8..1024, five overlap weights
* ``multiturn`` 32 workers, 512 conversations of 2..16 turns

Every draw is made in a fixed order from one ``Generator(PCG64(seed))`` so a
seed fully determines a trace, independently of the concurrency level or the
routing weights it is later simulated with (common random numbers).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

VOCAB = 32000          # token ids are uniform in [0, VOCAB)
BLOCK_TOKENS = 16      # tokens per KV block


# ---------------------------------------------------------------------------
# random helpers (inputs only)
# ---------------------------------------------------------------------------

def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(int(seed)))


def zipf_finite(rng: np.random.Generator, n_items: int, s: float, size) -> np.ndarray:
    """Finite-support Zipf: Pr(rank k) proportional to k^-s for k = 1..n_items.

    Returns 0-based item indices (rank - 1).  numpy's own ``zipf`` has infinite
    support and rejects s <= 1, so the inverse CDF is used instead.
    """
    k = np.arange(1, n_items + 1, dtype=np.float64)
    w = k ** (-float(s))
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    u = rng.random(size)
    idx = np.searchsorted(cdf, u, side="right")
    return np.minimum(idx, n_items - 1).astype(np.int32)


def _shared_bounds(P: np.ndarray):
    """Inclusive integer bounds of a shared prefix covering 25-75% of P blocks."""
    lo = (P + 3) // 4            # ceil(P/4)
    hi = (3 * P) // 4            # floor(3P/4)
    hi = np.maximum(hi, lo)
    return lo, hi


# ---------------------------------------------------------------------------
# episode traces
# ---------------------------------------------------------------------------

@dataclass
class Trace:
    """Requests of one episode trace, grouped by conversation.

    A conversation owns one token sequence; its turns are requests whose
    prompts are prefixes of that sequence (single-turn workloads have one turn
    per conversation).  All offsets are CSR-style.

    tokens       int32 [T]          token ids of every conversation, concatenated
    tok_off      int64 [n_conv+1]   conversation c owns tokens[tok_off[c]:tok_off[c+1]]
    chain_blocks int32 [n_conv]     full blocks of the conversation that are hashed
    chain_off    int64 [n_conv+1]   exclusive prefix sum of chain_blocks
    turn_off     int64 [n_conv+1]   turns of conversation c are turn_off[c]..turn_off[c+1]-1
    turn_blocks  int32 [n_turns]    prompt length of each turn, in blocks
    group        int32 [n_conv]     prefix group (-1 when none); metadata only
    shared       int32 [n_conv]     shared-prefix blocks; metadata only
    """
    seed: int
    tokens: np.ndarray
    tok_off: np.ndarray
    chain_blocks: np.ndarray
    chain_off: np.ndarray
    turn_off: np.ndarray
    turn_blocks: np.ndarray
    group: np.ndarray
    shared: np.ndarray

    @property
    def n_conv(self) -> int:
        return int(self.chain_blocks.shape[0])

    @property
    def n_turns(self) -> int:
        return int(self.turn_blocks.shape[0])

    @property
    def n_blocks(self) -> int:
        return int(self.chain_off[-1])


def _assemble_single_turn(seed, rng, P, n_groups, zipf_s) -> Trace:
    n = P.shape[0]
    g = zipf_finite(rng, n_groups, zipf_s, n)
    lo, hi = _shared_bounds(P)
    s = rng.integers(lo, hi + 1).astype(np.int64)
    s_max = int(s.max()) if n else 0
    group_tok = rng.integers(0, VOCAB, size=(n_groups, s_max * BLOCK_TOKENS), dtype=np.int32)
    n_priv = int(((P - s) * BLOCK_TOKENS).sum())
    priv = rng.integers(0, VOCAB, size=n_priv, dtype=np.int32)

    tok_len = P.astype(np.int64) * BLOCK_TOKENS
    tok_off = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(tok_len, out=tok_off[1:])
    tokens = np.empty(int(tok_off[-1]), dtype=np.int32)
    p_off = 0
    for i in range(n):
        a = int(tok_off[i])
        sh = int(s[i]) * BLOCK_TOKENS
        tokens[a:a + sh] = group_tok[g[i], :sh]
        npv = int(tok_len[i]) - sh
        tokens[a + sh:a + sh + npv] = priv[p_off:p_off + npv]
        p_off += npv
    chain_blocks = P.astype(np.int32)
    chain_off = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(chain_blocks, out=chain_off[1:])
    turn_off = np.arange(n + 1, dtype=np.int64)
    return Trace(seed=int(seed), tokens=tokens, tok_off=tok_off, chain_blocks=chain_blocks,
                 chain_off=chain_off, turn_off=turn_off, turn_blocks=P.astype(np.int32).copy(),
                 group=g.astype(np.int32), shared=s.astype(np.int32))


def lognormal_blocks(rng, n, mu, sigma, lo_tok, hi_tok) -> np.ndarray:
    """Prompt lengths: lognormal tokens clipped to [lo_tok, hi_tok], full blocks only."""
    L = rng.lognormal(mean=mu, sigma=sigma, size=n)
    L = np.clip(np.floor(L), lo_tok, hi_tok).astype(np.int64)
    return (L // BLOCK_TOKENS).astype(np.int64)


def tiny_trace(seed: int = 0, n_req: int = 64) -> Trace:
    """Tiny single episode: prompts of 4..32 blocks, 8 prefix groups, Zipf(1.1)."""
    rng = _rng(seed)
    P = rng.integers(4, 33, size=n_req).astype(np.int64)
    return _assemble_single_turn(seed, rng, P, 8, 1.1)


def sweep70b_trace(seed: int, n_req: int = 4096) -> Trace:
    """1P/5D-shaped trace: lognormal(ln 1024, 1.0) tokens in [128, 8192], 64 groups, Zipf(1.0)."""
    rng = _rng(seed)
    P = lognormal_blocks(rng, n_req, np.log(1024.0), 1.0, 128, 8192)
    return _assemble_single_turn(seed, rng, P, 64, 1.0)


def saturation_trace(seed: int, n_req: int = 2048) -> Trace:
    """Saturation sweep trace: lognormal(ln 2048, 1.2) tokens in [128, 16384], 64 groups, Zipf(1.0)."""
    rng = _rng(seed)
    P = lognormal_blocks(rng, n_req, np.log(2048.0), 1.2, 128, 16384)
    return _assemble_single_turn(seed, rng, P, 64, 1.0)


def multiturn_trace(seed: int, n_conv: int = 512, max_turns: int = 16,
                    add_lo: int = 256, add_hi: int = 2048, ctx_max: int = 32768) -> Trace:
    """Long-context multi-turn trace.

    Conversation c asks for T_c ~ U{2..16} turns; each turn appends U[256, 2048]
    tokens to the context, which is clipped at 32,768 tokens, and a conversation
    ends at the turn whose context reaches that limit.  A turn's prompt is the
    whole context so far, in full blocks.  Each conversation draws its own
    tokens (no shared groups).
    """
    rng = _rng(seed)
    T = rng.integers(2, max_turns + 1, size=n_conv)
    adds = rng.integers(add_lo, add_hi + 1, size=(n_conv, max_turns))
    turn_lens: List[List[int]] = []
    for c in range(n_conv):
        ctx = 0
        lens = []
        for k in range(int(T[c])):
            ctx = min(ctx + int(adds[c, k]), ctx_max)
            lens.append(ctx)
            if ctx >= ctx_max:
                break
        turn_lens.append(lens)
    final = np.array([l[-1] for l in turn_lens], dtype=np.int64)
    tok_off = np.zeros(n_conv + 1, dtype=np.int64)
    np.cumsum(final, out=tok_off[1:])
    tokens = rng.integers(0, VOCAB, size=int(tok_off[-1]), dtype=np.int32)
    turn_blocks = np.array([x // BLOCK_TOKENS for l in turn_lens for x in l], dtype=np.int32)
    nt = np.array([len(l) for l in turn_lens], dtype=np.int64)
    turn_off = np.zeros(n_conv + 1, dtype=np.int64)
    np.cumsum(nt, out=turn_off[1:])
    chain_blocks = (final // BLOCK_TOKENS).astype(np.int32)
    chain_off = np.zeros(n_conv + 1, dtype=np.int64)
    np.cumsum(chain_blocks, out=chain_off[1:])
    return Trace(seed=int(seed), tokens=tokens, tok_off=tok_off, chain_blocks=chain_blocks,
                 chain_off=chain_off, turn_off=turn_off, turn_blocks=turn_blocks,
                 group=np.full(n_conv, -1, np.int32), shared=np.zeros(n_conv, np.int32))


# ---------------------------------------------------------------------------
# episode workload descriptions
# ---------------------------------------------------------------------------

@dataclass
class EpisodeSpec:
    """Parameters of one routing episode over one trace."""
    seed: int
    concurrency: int          # C: requests in flight once the ramp is over
    hold_steps: int = 4       # H: routing steps a request stays active
    w_ov: float = 1.0
    w_act: float = 0.5
    w_sat: float = 4.0
    cap: int = 512            # active blocks at which the overload term starts
    controller: int = 0       # 1: switch to ctrl_w_ov when the windowed load is high; 2: regime controller
    ctrl_w_ov: float = 0.25
    ctrl_window: int = 128
    ctrl_num: int = 9         # threshold num/den of mean load per unit capacity
    ctrl_den: int = 10
    policy: int = 0           # POLICY_ARGMIN, POLICY_SOFTMAX, POLICY_ROUND_ROBIN, POLICY_RANDOM, POLICY_P2C
    tau: float = 0.0          # softmax temperature (> 0 with POLICY_SOFTMAX), in cost units
    evict_policy: int = 0     # EVICT_LRU, or EVICT_FREQ (the KV block manager's frequency policy)
    decay_steps: int = 0      # EVICT_FREQ: routing steps per time-decay step (>= 1)
    tier_g1: int = 0          # memory tiers (LRU only): blocks in G1 (0 = no tiers) ...
    tier_g2: int = 0          # ... and in G2; G3 holds the rest of the cache
    tier_w: tuple = (0.0, 0.25, 0.5)   # prefill weight of a block served from G1, G2, G3

    @property
    def routes_per_step(self) -> int:
        return self.concurrency // self.hold_steps


# Eviction policies of the workers' block caches (the routing library's RK_EVICT_* codes).
EVICT_LRU = 0    # least recently used block first
EVICT_FREQ = 1   # least frequent block first (1 on insert, x2 per hit, -1 per decay step, floor 1)


# Regime controller (controller = 2): the paper's EWMA weight, its 70B thresholds
# (seconds) and its (temperature, overlap weight) per regime Below / Transition /
# Saturated; the latency model is the PoA-hat matrix's; k and eps are not given
# by the paper (fill-ins).
REGIME_PARAMS = dict(alpha=0.3, theta1=0.3, theta2=2.0, eps=0.05, k=3, a=0.005, b=0.020, d=0.010, beta=2,
                     n_sat=64, tau=(0.0, 0.7, 0.8), w_ov=(1.0, 1.0, 0.1))


# Worker-selection policies of an episode (the routing library's RK_POLICY_* codes).
POLICY_ARGMIN = 0        # least cost, lowest index on ties (temperature 0)
POLICY_SOFTMAX = 1       # sample by exp(-cost / tau)
POLICY_ROUND_ROBIN = 2   # route t goes to worker t mod W
POLICY_RANDOM = 3        # uniform worker
POLICY_P2C = 4           # two distinct uniform candidates, the cheaper one
POLICY_NAMES = {POLICY_ARGMIN: "argmin", POLICY_SOFTMAX: "softmax", POLICY_ROUND_ROBIN: "round-robin",
                POLICY_RANDOM: "random", POLICY_P2C: "power-of-two"}


def route_rand(spec: "EpisodeSpec", n_routes: int) -> np.ndarray:
    """Two uniform 32-bit words per route of an episode, in routing order (the
    random draws of the stochastic policies, passed to the router as inputs)."""
    ss = np.random.SeedSequence([0x5EED, int(spec.seed), int(spec.concurrency), int(spec.policy) & 0xFFFFFFFF,
                                 int(np.float32(spec.tau).view(np.uint32))])
    return np.random.Generator(np.random.PCG64(ss)).integers(0, 1 << 32, size=2 * n_routes,
                                                             dtype=np.uint64).astype(np.uint32)


@dataclass
class Workload:
    name: str
    W: int
    cache_blocks: int
    traces: Dict[int, Trace]
    episodes: List[EpisodeSpec]
    poa: dict = field(default_factory=dict)
    regime: dict = field(default_factory=lambda: dict(REGIME_PARAMS))   # controller = 2 episodes


POA_PARAMS = dict(a=0.005, b=0.020, d=0.010, beta=2, C_cap=64, w_c=0.015)
"""Frozen parametric latency model of the PoA estimator (Section 6.4)."""


def tiny_workload() -> Workload:
    tr = tiny_trace(0)
    eps = [EpisodeSpec(seed=0, concurrency=8, cap=512)]
    return Workload("tiny", W=4, cache_blocks=256, traces={0: tr}, episodes=eps)


SWEEP70B_C = (32, 64, 128, 256, 512)
SATURATION_C = tuple(2 ** k for k in range(3, 11))          # 8..1024
SATURATION_WOV = (0.0, 0.25, 0.5, 1.0, 2.0)


def sweep70b_workload(seeds: Sequence[int] = range(64), concurrency: Sequence[int] = SWEEP70B_C,
                      n_req: int = 4096) -> Workload:
    traces = {int(s): sweep70b_trace(int(s), n_req) for s in seeds}
    eps = [EpisodeSpec(seed=int(s), concurrency=int(C), cap=32768)
           for C in concurrency for s in seeds]
    return Workload("sweep70b", W=6, cache_blocks=65536, traces=traces, episodes=eps)


# The static counterfactual policies next to the router's own (argmin and a
# softmax whose temperature is in cost units, i.e. blocks).
POLICY_SWEEP = ((POLICY_ARGMIN, 0.0), (POLICY_SOFTMAX, 16.0), (POLICY_ROUND_ROBIN, 0.0),
                (POLICY_RANDOM, 0.0), (POLICY_P2C, 0.0))


def policy_workload(seeds: Sequence[int] = range(16), concurrency: Sequence[int] = SWEEP70B_C,
                    policies: Sequence = POLICY_SWEEP, n_req: int = 4096, regime: bool = True) -> Workload:
    """The 1P/5D-shaped sweep traces routed by each selection policy, and (regime)
    by the regime controller with the paper's parameters."""
    traces = {int(s): sweep70b_trace(int(s), n_req) for s in seeds}
    eps = [EpisodeSpec(seed=int(s), concurrency=int(C), cap=32768, policy=int(p), tau=float(tau))
           for p, tau in policies for C in concurrency for s in seeds]
    if regime:
        eps += [EpisodeSpec(seed=int(s), concurrency=int(C), cap=32768, controller=2)
                for C in concurrency for s in seeds]
    return Workload("policies", W=6, cache_blocks=65536, traces=traces, episodes=eps)


def saturation_workload(seeds: Sequence[int] = range(256), concurrency: Sequence[int] = SATURATION_C,
                        w_ov: Sequence[float] = SATURATION_WOV, n_req: int = 2048) -> Workload:
    traces = {int(s): saturation_trace(int(s), n_req) for s in seeds}
    eps = [EpisodeSpec(seed=int(s), concurrency=int(C), w_ov=float(w), cap=2048, controller=1)
           for C in concurrency for w in w_ov for s in seeds]
    return Workload("saturation", W=16, cache_blocks=32768, traces=traces, episodes=eps)


def multiturn_workload(seeds: Sequence[int] = range(128), n_conv: int = 512) -> Workload:
    traces = {int(s): multiturn_trace(int(s), n_conv) for s in seeds}
    eps = [EpisodeSpec(seed=int(s), concurrency=256, cap=4096) for s in seeds]
    return Workload("multiturn", W=32, cache_blocks=16384, traces=traces, episodes=eps)


# ---------------------------------------------------------------------------
# snapshot scoring workload
# ---------------------------------------------------------------------------

@dataclass
class ScoringInstance:
    """Fixed worker key sets and a batch of block-hash chains.

    Keys are distinct by construction: bits 63..32 hold a unique nonzero index
    and bits 31..0 are uniform random, so no key is zero and any hash-table home
    slot taken from the low bits is uniform.

    keys       uint64 [sum]    worker j holds keys[key_off[j]:key_off[j+1]]
    key_off    int64 [W+1]
    chains     uint64 [sum]    request i's chain is chains[chain_off[i]:chain_off[i+1]]
    chain_off  int64 [B+1]
    active     int32 [W]       active blocks per worker
    """
    W: int
    B: int
    keys: np.ndarray
    key_off: np.ndarray
    chains: np.ndarray
    chain_off: np.ndarray
    active: np.ndarray
    cap: int = 32768
    w_ov: float = 1.0
    w_act: float = 0.5
    w_sat: float = 4.0
    log2_slots: int = 20
    group: Optional[np.ndarray] = None


class _KeyMaker:
    def __init__(self, rng):
        self.rng = rng
        self.next = 1

    def make(self, n: int) -> np.ndarray:
        idx = np.arange(self.next, self.next + n, dtype=np.uint64)
        self.next += n
        low = self.rng.integers(0, 2 ** 32, size=n, dtype=np.uint64)
        return (idx << np.uint64(32)) | low


def scoring_instance(seed: int = 0, B: int = 65536, W: int = 64, log2_slots: int = 20,
                     n_groups: int = 256, zipf_s: float = 0.9, len_lo: int = 16,
                     len_hi: int = 512, keys_per_worker: Optional[int] = None) -> ScoringInstance:
    """Batched-scoring stress instance.

    Each worker's table is filled to half its slots: repeatedly a group g is
    drawn by Zipf(0.9), its chain prefix R_g[0..d-1] (d ~ U{16..512}) is
    inserted, followed by a private continuation of U{16..512} fresh keys,
    until the worker holds exactly ``keys_per_worker`` distinct keys.  Every
    request draws a group, a length L ~ U{16..512}, a shared prefix of
    U{ceil(L/4)..floor(3L/4)} blocks from R_g, then fresh private keys.
    """
    rng = _rng(seed)
    km = _KeyMaker(rng)
    if keys_per_worker is None:
        keys_per_worker = (1 << log2_slots) // 2
    R = km.make(n_groups * len_hi).reshape(n_groups, len_hi)
    active = rng.integers(0, 65537, size=W).astype(np.int32)

    keys_list = []
    for j in range(W):
        depth = np.zeros(n_groups, dtype=np.int64)
        parts = []
        have = 0
        while have < keys_per_worker:
            g = int(zipf_finite(rng, n_groups, zipf_s, 1)[0])
            d = int(rng.integers(len_lo, len_hi + 1))
            c = int(rng.integers(len_lo, len_hi + 1))
            if d > depth[g]:
                new = R[g, depth[g]:d]
                take = min(new.shape[0], keys_per_worker - have)
                parts.append(new[:take])
                have += take
                depth[g] = depth[g] + take
            if have < keys_per_worker:
                take = min(c, keys_per_worker - have)
                parts.append(km.make(take))
                have += take
        keys_list.append(np.concatenate(parts))
    key_off = np.zeros(W + 1, dtype=np.int64)
    np.cumsum([k.shape[0] for k in keys_list], out=key_off[1:])
    keys = np.concatenate(keys_list)

    g = zipf_finite(rng, n_groups, zipf_s, B)
    L = rng.integers(len_lo, len_hi + 1, size=B).astype(np.int64)
    lo, hi = _shared_bounds(L)
    s = rng.integers(lo, hi + 1).astype(np.int64)
    chain_off = np.zeros(B + 1, dtype=np.int64)
    np.cumsum(L, out=chain_off[1:])
    chains = np.empty(int(chain_off[-1]), dtype=np.uint64)
    priv = km.make(int((L - s).sum()))
    p = 0
    for i in range(B):
        a = int(chain_off[i])
        si = int(s[i])
        chains[a:a + si] = R[g[i], :si]
        n_p = int(L[i]) - si
        chains[a + si:a + si + n_p] = priv[p:p + n_p]
        p += n_p
    return ScoringInstance(W=W, B=B, keys=keys, key_off=key_off, chains=chains,
                           chain_off=chain_off, active=active, log2_slots=log2_slots, group=g)


# ---------------------------------------------------------------------------
# flattening helpers shared by the GPU binding and the oracle driver
# ---------------------------------------------------------------------------

@dataclass
class FlatTraces:
    """Several traces concatenated into one set of CSR arrays."""
    seeds: List[int]
    tokens: np.ndarray
    tok_off: np.ndarray
    chain_blocks: np.ndarray
    chain_off: np.ndarray
    turn_off: np.ndarray
    turn_blocks: np.ndarray
    conv_begin: Dict[int, int]     # seed -> first conversation index
    conv_count: Dict[int, int]


def flatten_traces(traces: Dict[int, Trace]) -> FlatTraces:
    seeds = sorted(traces)
    toks, tlen, cb, tb, nturns = [], [], [], [], []
    conv_begin, conv_count = {}, {}
    c0 = 0
    for s in seeds:
        t = traces[s]
        conv_begin[s] = c0
        conv_count[s] = t.n_conv
        c0 += t.n_conv
        toks.append(t.tokens)
        tlen.append(np.diff(t.tok_off))
        cb.append(t.chain_blocks)
        tb.append(t.turn_blocks)
        nturns.append(np.diff(t.turn_off))
    tokens = np.concatenate(toks) if toks else np.zeros(0, np.int32)
    tlen = np.concatenate(tlen) if tlen else np.zeros(0, np.int64)
    tok_off = np.zeros(tlen.shape[0] + 1, np.int64)
    np.cumsum(tlen, out=tok_off[1:])
    chain_blocks = np.concatenate(cb) if cb else np.zeros(0, np.int32)
    chain_off = np.zeros(chain_blocks.shape[0] + 1, np.int64)
    np.cumsum(chain_blocks, out=chain_off[1:])
    nt = np.concatenate(nturns) if nturns else np.zeros(0, np.int64)
    turn_off = np.zeros(nt.shape[0] + 1, np.int64)
    np.cumsum(nt, out=turn_off[1:])
    turn_blocks = np.concatenate(tb) if tb else np.zeros(0, np.int32)
    return FlatTraces(seeds=seeds, tokens=tokens, tok_off=tok_off, chain_blocks=chain_blocks,
                      chain_off=chain_off, turn_off=turn_off, turn_blocks=turn_blocks,
                      conv_begin=conv_begin, conv_count=conv_count)
