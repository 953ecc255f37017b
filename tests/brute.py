"""Pure-Python brute-force twins used to pin the C oracle on tiny inputs.

These use different data structures from the oracle (Python sets and an
OrderedDict LRU instead of a chained hash map with a linked recency list;
exhaustive enumeration instead of the Hungarian method) so that a mistake in
either implementation shows up as a disagreement.
"""
from __future__ import annotations

import itertools
from collections import OrderedDict

import numpy as np

f32 = np.float32


def cost_f32(w_ov, w_act, w_sat, cap, P, o, A):
    """Router cost in fp32, one IEEE operation at a time (numpy scalars do not fuse)."""
    t1 = f32(w_ov) * f32(P - o)
    t2 = f32(w_act) * f32(A)
    r = f32(A + P) / f32(cap)
    x = max(r - f32(1.0), f32(0.0))
    t3 = f32(w_sat) * (x * x)
    return f32(f32(t1 + t2) + t3)


def cost_tiers_f32(w_ov, w_act, w_sat, cap, P, o, o1, o12, tw, A):
    """Router cost with the cached prefix split over memory tiers: o1 blocks in
    G1, o12 - o1 in G2, o - o12 in G3, each weighted by tw in the prefill term."""
    pf = f32(P - o)
    pf = f32(pf + f32(tw[0]) * f32(o1))
    pf = f32(pf + f32(tw[1]) * f32(o12 - o1))
    pf = f32(pf + f32(tw[2]) * f32(o - o12))
    t1 = f32(w_ov) * pf
    t2 = f32(w_act) * f32(A)
    r = f32(A + P) / f32(cap)
    x = max(r - f32(1.0), f32(0.0))
    t3 = f32(w_sat) * (x * x)
    return f32(f32(t1 + t2) + t3)


def overlap_set(chain, cached: set) -> int:
    o = 0
    while o < len(chain) and int(chain[o]) in cached:
        o += 1
    return o


def episode(W, cache_blocks, H, rps, w_ov, w_act, w_sat, cap, turn_off, turn_blocks, chains_per_conv,
            controller=0, ctrl_w_ov=0.25, ctrl_window=128, ctrl_num=9, ctrl_den=10, select=None, regime=None,
            freq=None, tiers=None):
    """Sequential routing episode with OrderedDict LRU caches; select(costs, t)
    picks the worker of route t (default: least cost, lowest index).  With
    controller 2, regime = (params(r) -> (tau, w_ov), step(n, t) -> new
    regime, select_tau(costs, t, tau)) drives the regime controller.  With
    freq = (decay_steps, cap) the caches evict by frequency: a block enters at 1,
    doubles per hit (at most cap), loses 1 per decay step (never below 1), and
    the least frequent block, oldest among equals, is evicted first.  With
    tiers = (k1, k2, tw) a worker's k1 most recent blocks are G1 and the next k2
    G2; routes record (o1, o12) per worker and pay the tiered cost."""
    n_conv = len(turn_off) - 1
    caches = [OrderedDict() for _ in range(W)]   # key -> None, oldest first
    A = [0] * W
    queue = [c for c in range(n_conv) if turn_off[c + 1] > turn_off[c]]
    next_turn = [turn_off[c] for c in range(n_conv)]
    steps = {}                                    # step -> list of (worker, P, conv)
    routes = []
    us = []
    prev_active = False
    nflight = [0] * W
    rg = 0
    s = 0
    while True:
        if s - H in steps:
            for (j, P, c) in steps.pop(s - H):
                A[j] -= P
                nflight[j] -= 1
                if next_turn[c] < turn_off[c + 1]:
                    queue.append(c)
        inflight = sum(len(v) for k, v in steps.items() if s - H < k < s)
        if not queue and inflight == 0:
            break
        if freq is not None and s > 0 and s % freq[0] == 0:
            for cch in caches:
                for key in cch:
                    cch[key] = max(cch[key] - 1, 1)
        take, queue = queue[:rps], queue[rps:]
        steps[s] = []
        for c in take:
            turn = next_turn[c]
            next_turn[c] += 1
            P = int(turn_blocks[turn])
            h = [int(x) for x in chains_per_conv[c][:P]]
            w_eff = f32(w_ov)
            active = (controller == 1 and len(us) >= ctrl_window and
                      ctrl_den * sum(us[-ctrl_window:]) > ctrl_num * ctrl_window * W * cap)
            if active:
                w_eff = min(f32(w_ov), f32(ctrl_w_ov))
            route_regime = rg if controller == 2 else 0
            if controller == 2:
                rtau, rw = regime[0](rg)
                w_eff = f32(rw)
            ovl = [overlap_set(h, caches[j].keys()) for j in range(W)]
            if tiers is None:
                costs = [cost_f32(w_eff, w_act, w_sat, cap, P, ovl[j], A[j]) for j in range(W)]
                tov = None
            else:
                k1, k2, tw = tiers
                tov = []
                for j in range(W):
                    order = list(caches[j].keys())[::-1]          # newest first
                    g1, g12 = set(order[:k1]), set(order[:k1 + k2])
                    tov.append((overlap_set(h, g1), overlap_set(h, g12)))
                costs = [cost_tiers_f32(w_eff, w_act, w_sat, cap, P, ovl[j], tov[j][0], tov[j][1], tw, A[j])
                         for j in range(W)]
            if controller == 2 and rtau > 0:
                sigma = int(regime[2](costs, len(routes), rtau))
            elif select is None:
                sigma = 0
                for j in range(1, W):
                    if costs[j] < costs[sigma]:
                        sigma = j
            else:
                sigma = int(select(costs, len(routes)))
            cache = caches[sigma]
            for k in range(P - 1, -1, -1):
                if h[k] in cache:
                    cache.move_to_end(h[k])
                    if freq is not None:
                        cache[h[k]] = min(2 * cache[h[k]], freq[1])
                else:
                    cache[h[k]] = 1
            evicted = []
            while len(cache) > cache_blocks:
                if freq is None:
                    key, _ = cache.popitem(last=False)
                else:
                    fmin = min(cache.values())
                    key = next(k for k, v in cache.items() if v == fmin)
                    del cache[key]
                evicted.append(key)
            A[sigma] += P
            nflight[sigma] += 1
            if controller == 2:
                rg = int(regime[1](nflight[sigma], len(routes)))
            us.append(sum(A))
            routes.append(dict(turn=turn, worker=sigma, step=s, P=P, overlap=ovl, cost=costs, regime=route_regime,
                               tier_overlap=tov,
                               evicted=evicted, active=bool(active),
                               first_active=bool(active and not prev_active)))
            prev_active = bool(active)
            steps[s].append((sigma, P, c))
        s += 1
    final = [list(c.keys()) for c in caches]
    return routes, final


def opt_bruteforce(c: np.ndarray, K: int) -> float:
    """Min over assignments of m rows to W columns with at most K rows per column."""
    m, W = c.shape
    best = None
    for assign in itertools.product(range(W), repeat=m):
        counts = np.bincount(np.asarray(assign, dtype=np.int64), minlength=W)
        if counts.max(initial=0) > K:
            continue
        v = sum(float(c[i, assign[i]]) for i in range(m))
        if best is None or v < best:
            best = v
    return best
