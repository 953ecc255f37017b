"""Device-resident episode batches: one pass of the routing hot path.

``EpisodeRunner`` uploads a workload's traces once (tokens, offsets), lays out
the per-episode parameters and output buffers, and runs one step of the path
through the C ABI: block-hash chains (rk_hash_chains), every routing episode
(rk_simulate_episodes), and the PoA-hat windows and per-episode ratios
(rk_poa_estimate).  Windows are the C consecutive routes of an episode, the
last one possibly shorter.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np

from . import rkroute as rk
from .workload import POA_PARAMS, EpisodeSpec, Workload, flatten_traces, route_rand


class EpisodeRunner:
    def __init__(self, workload: Workload, episodes: Optional[Sequence[EpisodeSpec]] = None,
                 probe_mode: int = rk.RK_PROBE_PREFIX, poa_params: Optional[dict] = None,
                 keep_cost: bool = True, device=None, chains: Optional[np.ndarray] = None,
                 ws_slots: int = 0):
        torch = rk._torch()
        self.torch = torch
        self.device = torch.device("cuda") if device is None else torch.device(device)
        self.W = workload.W
        self.cache_blocks = workload.cache_blocks
        self.episodes: List[EpisodeSpec] = list(workload.episodes if episodes is None else episodes)
        self.probe_mode = probe_mode
        self.flat = flat = flatten_traces({s: workload.traces[s] for s in
                                           sorted({e.seed for e in self.episodes})})
        dev = self.device
        up = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        self.tokens = up(flat.tokens if flat.tokens.size else np.zeros(16, np.int32), torch.int32)
        self.tok_off = up(flat.tok_off, torch.int64)
        self.chain_off = up(flat.chain_off, torch.int64)
        self.turn_off = up(flat.turn_off, torch.int64)
        self.turn_blocks = up(flat.turn_blocks if flat.turn_blocks.size else np.zeros(1, np.int32), torch.int32)
        self.chains = torch.empty(max(int(flat.chain_off[-1]), 1), dtype=torch.int64, device=dev)
        self.hash_enabled = chains is None
        if chains is not None:                     # block hashes given directly (no token hashing)
            ch = np.ascontiguousarray(chains, dtype=np.uint64)
            assert ch.shape[0] == int(flat.chain_off[-1])
            if ch.size:
                self.chains[: ch.size].copy_(torch.from_numpy(ch.view(np.int64)))

        E = len(self.episodes)
        prm = np.zeros(E, dtype=rk.EPISODE_PARAMS_DTYPE)
        win_off, ep_win_off = [0], [0]
        out_base = 0
        self.rows = []            # (first row, n_routes, conv_begin, turn_begin) per episode
        for e, sp in enumerate(self.episodes):
            cb, nc = flat.conv_begin[sp.seed], flat.conv_count[sp.seed]
            tb = int(flat.turn_off[cb])
            n_routes = int(flat.turn_off[cb + nc]) - tb
            prm[e] = (cb, nc, sp.hold_steps, sp.routes_per_step, sp.controller, sp.ctrl_window,
                      sp.ctrl_num, sp.ctrl_den, sp.cap, sp.w_ov, sp.w_act, sp.w_sat, sp.ctrl_w_ov, out_base,
                      sp.policy, sp.tau, sp.evict_policy, sp.decay_steps, sp.tier_g1, sp.tier_g2,
                      tuple(float(x) for x in sp.tier_w), 0)
            self.rows.append((out_base, n_routes, cb, tb))
            for k in range(0, n_routes, sp.concurrency):
                win_off.append(out_base + min(k + sp.concurrency, n_routes))
            ep_win_off.append(len(win_off) - 1)
            out_base += n_routes
        self.n_rows = out_base
        self.params_host = prm
        # the stochastic policies' draws: two words per output row (inputs, seeded per episode)
        self.regime = dict(workload.regime)
        self.route_rand = None
        if any(sp.policy in (rk.RK_POLICY_SOFTMAX, rk.RK_POLICY_RANDOM, rk.RK_POLICY_P2C) or
               (sp.controller == 2 and max(self.regime["tau"]) > 0) for sp in self.episodes):
            rr = np.zeros(2 * max(out_base, 1), np.uint32)
            for sp, (b0, n_routes, _, _) in zip(self.episodes, self.rows):
                rr[2 * b0: 2 * (b0 + n_routes)] = route_rand(sp, n_routes)
            self.route_rand = up(rr.view(np.int32), torch.int32)
        self.params = up(prm.view(np.uint8), torch.uint8)
        self.max_blocks = max(int(flat.turn_blocks.max()) if flat.turn_blocks.size else 1, 1)
        self.max_conv = max((flat.conv_count[sp.seed] for sp in self.episodes), default=0)
        self.max_rps = max((sp.routes_per_step for sp in self.episodes), default=1)
        self.max_inflight = max((sp.routes_per_step * sp.hold_steps for sp in self.episodes), default=1)
        self.max_ctrl_window = max([sp.ctrl_window for sp in self.episodes if sp.controller == 1] + [1])
        self.max_window = max((sp.concurrency for sp in self.episodes), default=1)

        R, W = max(self.n_rows, 1), self.W
        z = lambda shape, dt: torch.zeros(shape, dtype=dt, device=dev)
        self.route_turn = z(R, torch.int32)
        self.route_worker = z(R, torch.int32)
        self.route_step = z(R, torch.int32)
        self.route_blocks = z(R, torch.int32)
        self.overlap = z((R, W), torch.int32)
        self.cost = z((R, W), torch.float32) if keep_cost else None
        self.evict_count = z(R, torch.int32)
        self.evict_digest = z(R, torch.int64)     # uint64 bits
        self.last_hash = z(R, torch.int64)        # uint64 bits
        self.totals = z((max(E, 1), 8), torch.int64)
        self.route_regime = z(R, torch.int32)
        self.tiers = any(sp.tier_g1 > 0 for sp in self.episodes)
        self.tier_overlap = z((R, W, 2), torch.int32) if self.tiers else None
        self.max_routes = max([n for (_, n, _, _) in self.rows] + [0])
        # ws_slots < E: that many episode workspaces, reused by the workgroups that take the
        # episodes in turn (a batch larger than device memory runs in one launch)
        self.ws_slots = int(ws_slots) if 0 < int(ws_slots) < E else 0
        n_ws = self.ws_slots if self.ws_slots else E
        ws = rk.simulate_workspace_size(n_ws, W, self.cache_blocks, self.max_blocks, self.max_conv, self.max_routes)
        self.workspace = torch.empty(max(ws, 256), dtype=torch.uint8, device=dev)

        self.win_off = up(np.array(win_off, np.int64), torch.int64)
        self.ep_win_off = up(np.array(ep_win_off, np.int64), torch.int64)
        self.n_windows = len(win_off) - 1
        self.selfish = z(max(self.n_windows, 1), torch.float64)
        self.coord = z(max(self.n_windows, 1), torch.float64)
        self.poa_hat = z(max(E, 1), torch.float64)
        pp = dict(POA_PARAMS if poa_params is None else poa_params)
        self.poa_params = rk.PoaParams(pp["a"], pp["b"], pp["d"], pp["beta"], pp["C_cap"], pp["w_c"],
                                       int(pp.get("K_fixed", 0)))
        self.poa_ws = torch.empty(max(rk.poa_workspace_size(self.n_rows, W), 256), dtype=torch.uint8,
                                  device=dev)

        P = rk._ptr
        self.batch = rk.EpisodeBatch(E, W, self.cache_blocks, self.max_blocks, self.max_conv,
                                     self.max_inflight, self.max_rps, self.max_ctrl_window, probe_mode,
                                     int(self.tiers), self.max_routes, 0, self.ws_slots, 0,
                                     P(self.params), P(self.turn_off), P(self.turn_blocks), P(self.chain_off),
                                     P(self.chains), P(self.route_rand), rk.regime_params(self.regime))
        self.outputs = rk.EpisodeOutputs(P(self.route_turn), P(self.route_worker), P(self.route_step),
                                         P(self.route_blocks), P(self.overlap), P(self.cost),
                                         P(self.evict_count), P(self.evict_digest), P(self.last_hash),
                                         P(self.totals), P(self.route_regime), P(self.tier_overlap))

    # ---- the three stages of one step
    def hash(self, stream=None):
        rk.hash_chains(self.tokens, self.tok_off, self.chain_off, self.chains, stream=stream)

    def simulate(self, stream=None):
        rk.simulate_episodes(self.batch, self.outputs, self.workspace, stream=stream)

    def poa(self, stream=None):
        rk.poa_estimate(self.win_off, self.ep_win_off, self.n_rows, self.max_window, self.W,
                        self.route_worker, self.overlap, self.route_blocks, self.poa_params,
                        self.selfish, self.coord, self.poa_hat, self.poa_ws, stream=stream)

    def step(self, stream=None):
        if self.hash_enabled:
            self.hash(stream)
        self.simulate(stream)
        self.poa(stream)

    # ---- results on the host
    def episode_results(self, e: int) -> Dict[str, np.ndarray]:
        r0, n, cb, tb = self.rows[e]
        W = self.W
        cpu = lambda t: t.cpu().numpy()
        out = dict(
            route_turn=cpu(self.route_turn[r0:r0 + n]) - tb,
            route_worker=cpu(self.route_worker[r0:r0 + n]),
            route_step=cpu(self.route_step[r0:r0 + n]),
            route_blocks=cpu(self.route_blocks[r0:r0 + n]),
            overlap=cpu(self.overlap[r0:r0 + n]).reshape(n, W),
            evict_count=cpu(self.evict_count[r0:r0 + n]),
            evict_digest=cpu(self.evict_digest[r0:r0 + n]).view(np.uint64),
            last_hash=cpu(self.last_hash[r0:r0 + n]).view(np.uint64),
            totals=cpu(self.totals[e]),
            route_regime=cpu(self.route_regime[r0:r0 + n]),
        )
        if self.cost is not None:
            out["cost"] = cpu(self.cost[r0:r0 + n]).reshape(n, W)
        if self.tier_overlap is not None:
            out["tier_overlap"] = cpu(self.tier_overlap[r0:r0 + n]).reshape(n, W, 2)
        w0, w1 = int(self.ep_win_off[e]), int(self.ep_win_off[e + 1])
        out["selfish"] = cpu(self.selfish[w0:w1])
        out["coordinated"] = cpu(self.coord[w0:w1])
        out["poa_hat"] = float(self.poa_hat[e])
        return out

    def chains_host(self) -> np.ndarray:
        return self.chains[: int(self.flat.chain_off[-1])].cpu().numpy().view(np.uint64)
