"""ctypes binding of ``librkroute.so`` (the C ABI in include/rkroute.h).

Argument marshalling only: every computation runs in the HIP library.  PyTorch
supplies device memory and the current stream.  Importing this module does
not need a GPU; calling a compute entry point without the built library or a
GPU raises immediately.
"""
from __future__ import annotations

import ctypes as C
import os
import threading
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librkroute.so")

RK_OK, RK_EINVAL, RK_ENOMEM, RK_EHIP, RK_ETABLEFULL, RK_EUNSUPPORTED = 0, -1, -2, -3, -4, -5
RK_PROBE_PREFIX, RK_PROBE_SCAN = 0, 1
RK_POLICY_ARGMIN, RK_POLICY_SOFTMAX, RK_POLICY_ROUND_ROBIN, RK_POLICY_RANDOM, RK_POLICY_P2C = range(5)
RK_EVICT_LRU, RK_EVICT_FREQ = 0, 1
RK_FREQ_CAP = 1 << 20
DEV_BITS = {0x1: "bad offsets", 0x2: "short input", 0x4: "zero key", 0x8: "table full",
            0x10: "too large", 0x20: "no convergence", 0x40: "bad policy parameters"}

EXPORTED = ("rk_status_string", "rk_last_error", "rk_device_status", "rk_hash_chains",
            "rk_table_build", "rk_route_score_batch", "rk_index_build", "rk_route_score_index",
            "rk_simulate_workspace_size",
            "rk_simulate_episodes", "rk_poa_workspace_size", "rk_poa_estimate",
            "rk_poa_estimate_noalloc")
RK_POA_NOALLOC_BYTES = 64 << 20


class RkError(RuntimeError):
    pass


class CostParams(C.Structure):
    _fields_ = [("w_ov", C.c_float), ("w_act", C.c_float), ("w_sat", C.c_float),
                ("cap_blocks", C.c_int32)]


class PoaParams(C.Structure):
    _fields_ = [("a", C.c_float), ("b", C.c_float), ("d", C.c_float), ("beta", C.c_int32),
                ("C_cap", C.c_int32), ("w_c", C.c_float), ("K_fixed", C.c_int32)]


class RegimeParams(C.Structure):
    _fields_ = [("alpha", C.c_double), ("theta1", C.c_double), ("theta2", C.c_double), ("eps", C.c_double),
                ("k", C.c_int32), ("beta", C.c_int32), ("a", C.c_double), ("b", C.c_double), ("d", C.c_double),
                ("n_sat", C.c_int32), ("tau", C.c_float * 3), ("w_ov", C.c_float * 3)]


def regime_params(r: dict) -> RegimeParams:
    return RegimeParams(r["alpha"], r["theta1"], r["theta2"], r["eps"], r["k"], r["beta"], r["a"], r["b"], r["d"],
                        r["n_sat"], (C.c_float * 3)(*r["tau"]), (C.c_float * 3)(*r["w_ov"]))


class EpisodeBatch(C.Structure):
    _fields_ = [("E", C.c_int32), ("W", C.c_int32), ("cache_blocks", C.c_int32),
                ("max_blocks", C.c_int32), ("max_conv", C.c_int32), ("max_inflight", C.c_int32),
                ("max_routes_per_step", C.c_int32), ("max_ctrl_window", C.c_int32),
                ("probe_mode", C.c_int32), ("tiers", C.c_int32), ("max_routes", C.c_int32),
                ("flags", C.c_int32), ("ws_slots", C.c_int32), ("ws_pad", C.c_int32),
                ("params", C.c_void_p), ("turn_off", C.c_void_p), ("turn_blocks", C.c_void_p),
                ("chain_off", C.c_void_p), ("chains", C.c_void_p), ("route_rand", C.c_void_p),
                ("regime", RegimeParams)]


class EpisodeOutputs(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("route_turn", "route_worker", "route_step", "route_blocks",
                                          "overlap", "cost", "evict_count", "evict_digest",
                                          "last_hash", "totals", "route_regime", "tier_overlap")]


# rk_episode_params, 104 bytes, as a numpy record
EPISODE_PARAMS_DTYPE = np.dtype([
    ("conv_begin", "<i8"), ("n_conv", "<i4"), ("hold_steps", "<i4"), ("routes_per_step", "<i4"),
    ("controller", "<i4"), ("ctrl_window", "<i4"), ("ctrl_num", "<i4"), ("ctrl_den", "<i4"),
    ("cap_blocks", "<i4"), ("w_ov", "<f4"), ("w_act", "<f4"), ("w_sat", "<f4"),
    ("ctrl_w_ov", "<f4"), ("out_base", "<i8"), ("policy", "<i4"), ("tau", "<f4"),
    ("evict_policy", "<i4"), ("decay_steps", "<i4"), ("tier_g1", "<i4"), ("tier_g2", "<i4"),
    ("tier_w", "<f4", (3,)), ("tier_pad", "<i4")])
assert EPISODE_PARAMS_DTYPE.itemsize == 104

_lock = threading.Lock()
_lib = None


def library_available() -> bool:
    return os.path.exists(LIB_PATH)


def lib():
    """Load librkroute.so; raises if it has not been built."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RkError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_17081_amd.build`")
            L = C.CDLL(LIB_PATH)
            vp, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
            L.rk_status_string.restype = C.c_char_p
            L.rk_status_string.argtypes = [C.c_int]
            L.rk_last_error.restype = C.c_char_p
            L.rk_last_error.argtypes = []
            L.rk_device_status.restype = C.c_int
            L.rk_device_status.argtypes = [C.c_int, vp, vp]
            L.rk_hash_chains.restype = C.c_int
            L.rk_hash_chains.argtypes = [i64, vp, vp, vp, vp, vp]
            L.rk_table_build.restype = C.c_int
            L.rk_table_build.argtypes = [i32, vp, vp, vp, i32, vp]
            L.rk_route_score_batch.restype = C.c_int
            L.rk_route_score_batch.argtypes = [i32, i32, vp, vp, vp, i32, vp, CostParams, i32, vp, vp, vp, vp]
            L.rk_index_build.restype = C.c_int
            L.rk_index_build.argtypes = [i32, vp, vp, vp, i32, vp]
            L.rk_route_score_index.restype = C.c_int
            L.rk_route_score_index.argtypes = [i32, i32, vp, vp, vp, i32, vp, CostParams, i32, vp, vp, vp, vp]
            L.rk_simulate_workspace_size.restype = sz
            L.rk_simulate_workspace_size.argtypes = [i32, i32, i32, i32, i32, i32]
            L.rk_simulate_episodes.restype = C.c_int
            L.rk_simulate_episodes.argtypes = [C.POINTER(EpisodeBatch), C.POINTER(EpisodeOutputs), vp, sz, vp]
            L.rk_poa_workspace_size.restype = sz
            L.rk_poa_workspace_size.argtypes = [i64, i32]
            L.rk_poa_estimate.restype = C.c_int
            L.rk_poa_estimate.argtypes = [i32, vp, i32, vp, i64, i32, i32, vp, vp, vp, PoaParams,
                                          vp, vp, vp, vp, sz, vp]
            L.rk_poa_estimate_noalloc.restype = C.c_int
            L.rk_poa_estimate_noalloc.argtypes = [i32, vp, i32, vp, i64, i32, i32, vp, vp, vp, PoaParams,
                                                  vp, vp, vp, vp]
            _lib = L
    return _lib


def _check(rc: int, what: str):
    if rc != RK_OK:
        L = lib()
        raise RkError(f"{what}: {L.rk_status_string(rc).decode()} ({rc}): {L.rk_last_error().decode()}")


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RkError("no GPU visible: the routing library runs on an MI355X (gfx950) device only")
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _need(t, dtype, name):
    torch = _torch()
    if t is None:
        return
    ok = (torch.int64, torch.uint64) if dtype in (torch.int64, torch.uint64) and name in _HASH_ARGS else (dtype,)
    if not t.is_cuda or t.dtype not in ok or not t.is_contiguous():
        raise RkError(f"{name} must be a contiguous CUDA tensor of {dtype}")


def _outputs_fit(B, W, overlap, cost, argmin):
    for t, n, name in ((overlap, B * W, "overlap"), (cost, B * W, "cost"), (argmin, B, "argmin")):
        if t is not None and t.numel() < n:
            raise RkError(f"{name} holds {t.numel()} elements, {n} needed")


# 64-bit block hashes may live in int64 tensors (same bits; PyTorch supports
# more int64 operations than uint64 ones).
_HASH_ARGS = ("chains", "keys", "tables", "index", "evict_digest", "last_hash")


def to_device(a: np.ndarray, device="cuda"):
    """Upload a numpy array; uint64 arrays become int64 tensors with the same bits."""
    torch = _torch()
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint64:
        a = a.view(np.int64)
    return torch.from_numpy(a).to(device)


def to_host_u64(t) -> np.ndarray:
    """Copy a 64-bit hash tensor back as uint64."""
    return t.cpu().numpy().view(np.uint64)


# ------------------------------------------------------------------ entry points

def device_status(reset: bool = True, stream=None) -> int:
    bits = np.zeros(1, np.int32)
    _check(lib().rk_device_status(int(reset), C.c_void_p(bits.ctypes.data), _stream(stream)),
           "rk_device_status")
    return int(bits[0])


def hash_chains(tokens, tok_off, chain_off, chains=None, stream=None):
    """Block-hash chains of token sequences (see rk_hash_chains)."""
    torch = _torch()
    _need(tokens, torch.int32, "tokens")
    _need(tok_off, torch.int64, "tok_off")
    _need(chain_off, torch.int64, "chain_off")
    n_seq = tok_off.numel() - 1
    if chains is None:
        n = int(chain_off[-1].item()) if n_seq > 0 else 0
        chains = torch.empty(max(n, 1), dtype=torch.int64, device=tokens.device)
    _need(chains, torch.uint64, "chains")
    _check(lib().rk_hash_chains(n_seq, _ptr(tokens), _ptr(tok_off), _ptr(chain_off), _ptr(chains),
                                _stream(stream)), "rk_hash_chains")
    return chains


def table_build(keys, key_off: np.ndarray, log2_slots: int, tables=None, stream=None):
    """W open-addressing tables from per-worker key lists (key_off is a host array)."""
    torch = _torch()
    _need(keys, torch.uint64, "keys")
    key_off = np.ascontiguousarray(key_off, dtype=np.int64)
    W = key_off.shape[0] - 1
    if tables is None:
        tables = torch.empty(W << log2_slots, dtype=torch.int64, device=keys.device)
    _need(tables, torch.uint64, "tables")
    _check(lib().rk_table_build(W, _ptr(keys), C.c_void_p(key_off.ctypes.data), _ptr(tables), log2_slots,
                                _stream(stream)), "rk_table_build")
    return tables


def route_score_batch(chains, chain_off, tables, log2_slots: int, active_blocks, w_ov=1.0, w_act=0.5,
                      w_sat=4.0, cap_blocks=32768, probe_mode=RK_PROBE_PREFIX, overlap=None, cost=None,
                      argmin=None, want_overlap=True, want_cost=True, stream=None):
    """Overlap and cost per (request, worker) and argmin per request."""
    torch = _torch()
    _need(chains, torch.uint64, "chains")
    _need(chain_off, torch.int64, "chain_off")
    _need(tables, torch.uint64, "tables")
    _need(active_blocks, torch.int32, "active_blocks")
    B = chain_off.numel() - 1
    W = active_blocks.numel()
    dev = chains.device
    if overlap is None and want_overlap:
        overlap = torch.empty((B, W), dtype=torch.int32, device=dev)
    if cost is None and want_cost:
        cost = torch.empty((B, W), dtype=torch.float32, device=dev)
    if argmin is None:
        argmin = torch.empty(B, dtype=torch.int32, device=dev)
    _need(overlap, torch.int32, "overlap")
    _need(cost, torch.float32, "cost")
    _need(argmin, torch.int32, "argmin")
    _outputs_fit(B, W, overlap, cost, argmin)
    p = CostParams(w_ov, w_act, w_sat, cap_blocks)
    _check(lib().rk_route_score_batch(B, W, _ptr(chains), _ptr(chain_off), _ptr(tables), log2_slots,
                                      _ptr(active_blocks), p, probe_mode, _ptr(overlap), _ptr(cost),
                                      _ptr(argmin), _stream(stream)), "rk_route_score_batch")
    return overlap, cost, argmin


def index_build(keys, key_off: np.ndarray, log2_slots: int, index=None, stream=None):
    """The global block index (key, worker mask) over W workers' key lists
    (key_off is a host array); 16-byte slots held as int64 pairs."""
    torch = _torch()
    _need(keys, torch.uint64, "keys")
    key_off = np.ascontiguousarray(key_off, dtype=np.int64)
    W = key_off.shape[0] - 1
    if index is None:
        index = torch.empty(2 << log2_slots, dtype=torch.int64, device=keys.device)
    _need(index, torch.uint64, "index")
    if index.numel() < (2 << log2_slots):
        raise RkError("index holds fewer than 2^log2_slots 16-byte slots")
    _check(lib().rk_index_build(W, _ptr(keys), C.c_void_p(key_off.ctypes.data), _ptr(index), log2_slots,
                                _stream(stream)), "rk_index_build")
    return index


def route_score_index(chains, chain_off, index, log2_slots: int, active_blocks, w_ov=1.0, w_act=0.5,
                      w_sat=4.0, cap_blocks=32768, probe_mode=RK_PROBE_PREFIX, overlap=None, cost=None,
                      argmin=None, want_overlap=True, want_cost=True, stream=None):
    """route_score_batch against the global block index (rk_route_score_index)."""
    torch = _torch()
    _need(chains, torch.uint64, "chains")
    _need(chain_off, torch.int64, "chain_off")
    _need(index, torch.uint64, "index")
    _need(active_blocks, torch.int32, "active_blocks")
    B = chain_off.numel() - 1
    W = active_blocks.numel()
    if index.numel() < (2 << log2_slots):
        raise RkError("index holds fewer than 2^log2_slots 16-byte slots")
    dev = chains.device
    if overlap is None and want_overlap:
        overlap = torch.empty((B, W), dtype=torch.int32, device=dev)
    if cost is None and want_cost:
        cost = torch.empty((B, W), dtype=torch.float32, device=dev)
    if argmin is None:
        argmin = torch.empty(B, dtype=torch.int32, device=dev)
    _need(overlap, torch.int32, "overlap")
    _need(cost, torch.float32, "cost")
    _need(argmin, torch.int32, "argmin")
    _outputs_fit(B, W, overlap, cost, argmin)
    p = CostParams(w_ov, w_act, w_sat, cap_blocks)
    _check(lib().rk_route_score_index(B, W, _ptr(chains), _ptr(chain_off), _ptr(index), log2_slots,
                                      _ptr(active_blocks), p, probe_mode, _ptr(overlap), _ptr(cost),
                                      _ptr(argmin), _stream(stream)), "rk_route_score_index")
    return overlap, cost, argmin


def simulate_workspace_size(E, W, cache_blocks, max_blocks, max_conv, max_routes) -> int:
    return int(lib().rk_simulate_workspace_size(E, W, cache_blocks, max_blocks, max_conv, max_routes))


def simulate_episodes(batch: EpisodeBatch, outputs: EpisodeOutputs, workspace, stream=None):
    """Launch rk_simulate_episodes on prepared structs (see EpisodeRunner for the usual path)."""
    _check(lib().rk_simulate_episodes(C.byref(batch), C.byref(outputs), _ptr(workspace),
                                      workspace.numel() * workspace.element_size(), _stream(stream)),
           "rk_simulate_episodes")


def poa_workspace_size(n_rows: int, W: int) -> int:
    return int(lib().rk_poa_workspace_size(n_rows, W))


def poa_estimate(win_off, ep_win_off, n_rows: int, max_window: int, W: int, route_worker, overlap,
                 route_blocks, params: PoaParams, selfish, coord, poa_hat, workspace, stream=None):
    n_windows = win_off.numel() - 1
    n_eps = 0 if ep_win_off is None else ep_win_off.numel() - 1
    _check(lib().rk_poa_estimate(n_windows, _ptr(win_off), n_eps, _ptr(ep_win_off), n_rows, max_window, W,
                                 _ptr(route_worker), _ptr(overlap), _ptr(route_blocks), params,
                                 _ptr(selfish), _ptr(coord), _ptr(poa_hat), _ptr(workspace),
                                 workspace.numel() * workspace.element_size(), _stream(stream)),
           "rk_poa_estimate")


def poa_estimate_noalloc(win_off, ep_win_off, n_rows: int, max_window: int, W: int, route_worker, overlap,
                         route_blocks, params: PoaParams, selfish, coord, poa_hat, stream=None):
    """poa_estimate on the library's static device buffer (rk_poa_estimate_noalloc):
    no workspace argument, nothing allocated by the call."""
    n_windows = win_off.numel() - 1
    n_eps = 0 if ep_win_off is None else ep_win_off.numel() - 1
    _check(lib().rk_poa_estimate_noalloc(n_windows, _ptr(win_off), n_eps, _ptr(ep_win_off), n_rows, max_window, W,
                                         _ptr(route_worker), _ptr(overlap), _ptr(route_blocks), params,
                                         _ptr(selfish), _ptr(coord), _ptr(poa_hat), _stream(stream)),
           "rk_poa_estimate_noalloc")
