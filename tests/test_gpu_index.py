"""GPU parity of the global-block-index scorer (rk_index_build +
rk_route_score_index) against the CPU oracle's per-worker definition of the
overlap, cost and argmin: integers and fp32 costs bit for bit."""
import sys

import numpy as np
import pytest

from paper_2606_17081_amd import workload as wl

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


def _status_clean(rk):
    bits = rk.device_status(reset=True)
    assert bits == 0, [v for k, v in rk.DEV_BITS.items() if bits & k]


def index_log2(n_keys: int) -> int:
    """Smallest power-of-two slot count keeping the index at load <= 0.5."""
    b = 4
    while (1 << b) < 2 * n_keys:
        b += 1
    return b


def _score_index(rk, torch, inst, mode, index=None, lg=None):
    up = rk.to_device
    lg = lg if lg is not None else index_log2(int(inst.key_off[-1]))
    if index is None:
        index = rk.index_build(up(inst.keys), inst.key_off, lg)
    ov, co, am = rk.route_score_index(up(inst.chains), up(inst.chain_off), index, lg, up(inst.active),
                                      inst.w_ov, inst.w_act, inst.w_sat, inst.cap, probe_mode=mode)
    torch.cuda.synchronize()
    return ov.cpu().numpy(), co.cpu().numpy(), am.cpu().numpy(), index


def _check(got, ref, rows=None):
    ov, co, am = got[:3]
    if rows is not None:
        ov, co, am = ov[rows], co[rows], am[rows]
    bad = np.nonzero((ov != ref[0]).any(axis=1))[0]
    assert bad.size == 0, f"overlap differs on requests {bad[:8]}"
    assert np.array_equal(co.view(np.uint32), ref[1].view(np.uint32))
    assert np.array_equal(am, ref[2])


@pytest.mark.parametrize("W,len_hi", [(64, 70), (5, 300), (33, 600), (64, 900)])
def test_index_small_both_modes(gpu, orc, W, len_hi):
    """Chains of 1..len_hi blocks: all three search rounds and the ragged tails."""
    torch, rk = gpu
    inst = wl.scoring_instance(seed=W + len_hi, B=1200, W=W, log2_slots=11, len_lo=1, len_hi=len_hi)
    ref = orc.score_batch(inst.chains, inst.chain_off, inst.keys, inst.key_off, inst.active,
                          inst.w_ov, inst.w_act, inst.w_sat, inst.cap)
    for mode in (rk.RK_PROBE_PREFIX, rk.RK_PROBE_SCAN):
        say("index score W", W, "len_hi", len_hi, "mode", mode)
        _check(_score_index(rk, torch, inst, mode), ref)
    _status_clean(rk)


def test_index_staircase_many_intervals(gpu, orc):
    """One long chain per request, every worker caching a prefix of a different
    depth: the third round spans many chunks of 64 positions."""
    torch, rk = gpu
    rng = np.random.default_rng(11)
    W, B, n = 64, 96, 6000
    base = rng.integers(1, 2 ** 63, size=n, dtype=np.int64).astype(np.uint64) | np.uint64(1)
    depth = rng.permutation(np.arange(1, n, (n - 1) // W)[:W]).astype(np.int64)
    depth[:3] = [0, n, n - 1]
    keys = np.concatenate([base[:d] for d in depth])
    key_off = np.zeros(W + 1, np.int64)
    np.cumsum(depth, out=key_off[1:])
    L = rng.integers(1, n + 1, size=B)
    L[:4] = [n, n, 1, 65]
    chain_off = np.zeros(B + 1, np.int64)
    np.cumsum(L, out=chain_off[1:])
    chains = np.concatenate([base[:l] for l in L])
    inst = wl.ScoringInstance(W=W, B=B, keys=keys, key_off=key_off, chains=chains, chain_off=chain_off,
                              active=rng.integers(0, 9000, W).astype(np.int32), log2_slots=20)
    ref = orc.score_batch(inst.chains, inst.chain_off, inst.keys, inst.key_off, inst.active,
                          inst.w_ov, inst.w_act, inst.w_sat, inst.cap)
    for mode in (rk.RK_PROBE_PREFIX, rk.RK_PROBE_SCAN):
        say("staircase mode", mode)
        _check(_score_index(rk, torch, inst, mode), ref)
    _status_clean(rk)


def prefix_depth_instance(depths, lengths, n=4096, seed=0):
    """Worker j caches the first depths[j] blocks of one base chain; request i
    is its first lengths[i] blocks.  The depths place the workers' first misses
    where a test wants them."""
    rng = np.random.default_rng(seed)
    base = rng.integers(1, 2 ** 63, size=n, dtype=np.int64).astype(np.uint64) | np.uint64(1)
    depths = np.asarray(depths, np.int64)
    keys = np.concatenate([base[:d] for d in depths]) if depths.sum() else np.zeros(0, np.uint64)
    key_off = np.zeros(depths.size + 1, np.int64)
    np.cumsum(depths, out=key_off[1:])
    L = np.asarray(lengths, np.int64)
    chain_off = np.zeros(L.size + 1, np.int64)
    np.cumsum(L, out=chain_off[1:])
    chains = np.concatenate([base[:l] for l in L])
    return wl.ScoringInstance(W=depths.size, B=L.size, keys=keys, key_off=key_off, chains=chains,
                              chain_off=chain_off, active=rng.integers(0, 9000, depths.size).astype(np.int32),
                              log2_slots=20)


PATH_LENGTHS = [1, 2, 17, 63, 64, 65, 100, 255, 256, 257, 511, 512, 700, 833, 1000, 1024, 1500, 2048, 3000,
                4000, 4096]


def path_depths(case, rng, W=64):
    """Depth sets for the prefix search's paths: few boundaries everywhere;
    few sample boundaries but many first misses inside the intervals between
    them; many sample boundaries; few boundaries but more than 64 positions
    between samples; many boundaries among the first 64 blocks."""
    if case == "few":
        return rng.choice([0, 37, 300, 301, 833, 4096], size=W)
    if case == "clustered":
        return np.array([16 * a + int(rng.integers(0, 15)) for a in rng.choice([5, 20, 33, 50], size=W)])
    if case == "spread":
        return rng.permutation(np.arange(0, 4096, 64))[:W]
    if case == "wide":
        return rng.choice([1500, 2900, 4096], size=W)
    if case == "dense":
        return rng.integers(0, 64, size=W)
    raise ValueError(case)


@pytest.mark.parametrize("case", ["few", "clustered", "spread", "wide", "dense"])
def test_index_prefix_search_paths(gpu, orc, case):
    """Each path of the prefix search (scalar loops over few boundaries, the
    per-worker LDS searches when a round has many, the chunked third round when
    the sample intervals hold more than 64 positions) against the oracle, on
    requests that end before, at and past every worker's depth."""
    torch, rk = gpu
    rng = np.random.default_rng({"few": 1, "clustered": 2, "spread": 3, "wide": 4, "dense": 5}[case])
    inst = prefix_depth_instance(path_depths(case, rng), PATH_LENGTHS, seed=5)
    ref = orc.score_batch(inst.chains, inst.chain_off, inst.keys, inst.key_off, inst.active,
                          inst.w_ov, inst.w_act, inst.w_sat, inst.cap)
    say("prefix search paths", case)
    _check(_score_index(rk, torch, inst, rk.RK_PROBE_PREFIX), ref)
    _status_clean(rk)


@pytest.mark.parametrize("case", ["few", "clustered", "spread", "wide", "dense", "w0-empty", "w0-full", "one"])
def test_tables_shared_search_paths(gpu, orc, case):
    """The per-worker-table scorer's shared search (worker 0's overlap found by
    the whole wavefront, then checked on every table) when the check holds for
    every worker, for some, for none, when worker 0 caches nothing or the whole
    chain, and with a single worker."""
    torch, rk = gpu
    rng = np.random.default_rng(17)
    if case == "w0-empty":
        depths = np.concatenate([[0], rng.choice([300, 833, 4096], size=63)])
    elif case == "w0-full":
        depths = np.concatenate([[4096], np.zeros(63, np.int64)])
    elif case == "one":
        depths = np.array([833])
    else:
        depths = path_depths(case, np.random.default_rng({"few": 1, "clustered": 2, "spread": 3, "wide": 4,
                                                           "dense": 5}[case]))
    inst = prefix_depth_instance(depths, PATH_LENGTHS, seed=7)
    ref = orc.score_batch(inst.chains, inst.chain_off, inst.keys, inst.key_off, inst.active,
                          inst.w_ov, inst.w_act, inst.w_sat, inst.cap)
    up = rk.to_device
    say("table scorer shared search", case)
    tables = rk.table_build(up(inst.keys), inst.key_off, 14)
    for mode in (rk.RK_PROBE_PREFIX, rk.RK_PROBE_SCAN):
        ov, co, am = rk.route_score_batch(up(inst.chains), up(inst.chain_off), tables, 14, up(inst.active),
                                          inst.w_ov, inst.w_act, inst.w_sat, inst.cap, probe_mode=mode)
        torch.cuda.synchronize()
        _check((ov.cpu().numpy(), co.cpu().numpy(), am.cpu().numpy()), ref)
    _status_clean(rk)


def test_index_scan_mode_arbitrary_sets(gpu, orc):
    """Keys from a tiny alphabet: worker sets are not prefix-closed along chains."""
    torch, rk = gpu
    rng = np.random.default_rng(4)
    W, B = 17, 900
    L = rng.integers(0, 150, size=B)
    chain_off = np.zeros(B + 1, np.int64)
    np.cumsum(L, out=chain_off[1:])
    chains = rng.integers(1, 12, size=int(chain_off[-1])).astype(np.uint64)
    keys = [np.unique(rng.integers(1, 12, size=int(rng.integers(0, 14)))).astype(np.uint64) for _ in range(W)]
    key_off = np.zeros(W + 1, np.int64)
    np.cumsum([k.size for k in keys], out=key_off[1:])
    inst = wl.ScoringInstance(W=W, B=B, keys=np.concatenate(keys), key_off=key_off, chains=chains,
                              chain_off=chain_off, active=rng.integers(0, 50, W).astype(np.int32), cap=16,
                              log2_slots=6)
    ref = orc.score_batch(inst.chains, inst.chain_off, inst.keys, inst.key_off, inst.active,
                          inst.w_ov, inst.w_act, inst.w_sat, inst.cap)
    _check(_score_index(rk, torch, inst, rk.RK_PROBE_SCAN), ref)
    _status_clean(rk)


@pytest.mark.parametrize("spare", [0, 1])
def test_index_full_size_sampled(gpu, orc, spare):
    """65,536 requests x 64 workers on the benchmark's key sets, index at load
    <= 0.5 and (as benchmarked) <= 0.25: 300 sampled requests against the
    oracle; every request against the per-worker-table scorer."""
    torch, rk = gpu
    say("generating the 65,536 x 64 scoring instance")
    inst = wl.scoring_instance(seed=0)
    lg = index_log2(int(inst.key_off[-1])) + spare
    say("index scoring, log2 slots", lg)
    got = _score_index(rk, torch, inst, rk.RK_PROBE_PREFIX, lg=lg)
    _status_clean(rk)
    rng = np.random.default_rng(1)
    rows = np.unique(np.concatenate([[0, inst.B - 1], rng.integers(0, inst.B, 298)]))
    ref = orc.score_batch(inst.chains, inst.chain_off, inst.keys, inst.key_off, inst.active,
                          inst.w_ov, inst.w_act, inst.w_sat, inst.cap, rows=rows)
    _check(got, ref, rows=rows)
    up = rk.to_device
    tables = rk.table_build(up(inst.keys), inst.key_off, inst.log2_slots)
    ov_t, co_t, am_t = rk.route_score_batch(up(inst.chains), up(inst.chain_off), tables, inst.log2_slots,
                                            up(inst.active))
    torch.cuda.synchronize()
    assert np.array_equal(got[0], ov_t.cpu().numpy())
    assert np.array_equal(got[1].view(np.uint32), co_t.cpu().numpy().view(np.uint32))
    assert np.array_equal(got[2], am_t.cpu().numpy())
    say("scan mode on the same index")
    got2 = _score_index(rk, torch, inst, rk.RK_PROBE_SCAN, index=got[3], lg=lg)
    assert np.array_equal(got2[0], got[0]) and np.array_equal(got2[2], got[2])
    _status_clean(rk)


def test_index_empty_and_degenerate(gpu, orc):
    torch, rk = gpu
    inst = wl.scoring_instance(seed=9, B=40, W=3, log2_slots=6, len_lo=1, len_hi=90)
    n4 = int(inst.chain_off[5] - inst.chain_off[4])                       # make request 4 empty
    inst.chains = np.delete(inst.chains, np.s_[inst.chain_off[4]:inst.chain_off[5]])
    inst.chain_off[5:] -= n4
    ref = orc.score_batch(inst.chains, inst.chain_off, inst.keys, inst.key_off, inst.active,
                          inst.w_ov, inst.w_act, inst.w_sat, inst.cap)
    for mode in (rk.RK_PROBE_PREFIX, rk.RK_PROBE_SCAN):
        _check(_score_index(rk, torch, inst, mode), ref)
    # a worker with no keys, and B = 0
    W = 4
    koff = np.array([0, 0, 0, 0, 0], np.int64)
    idx = rk.index_build(torch.zeros(1, dtype=torch.int64, device="cuda"), koff, 4)
    z = torch.zeros(1, dtype=torch.int64, device="cuda")
    o, c, a = rk.route_score_index(z, z, idx, 4, torch.zeros(W, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    assert a.numel() == 0
    with pytest.raises(rk.RkError):
        rk.route_score_index(z, z, idx, 4, torch.zeros(65, dtype=torch.int32, device="cuda"))
    _status_clean(rk)
