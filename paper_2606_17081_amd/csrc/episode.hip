// episode.hip -- independent sequential routing episodes, one workgroup each.
//
// Per episode the workgroup (256 threads, 4 wavefronts) keeps in LDS the
// worker loads A_j, the LRU bookkeeping of every worker, the in-flight routes
// of the last H steps and the controller's load window.  Each worker's cached
// blocks live in HBM as an open-addressing table of 16-byte slots (key, stamp)
// plus a ring log of touches:
//   - a touch of a block at stamp p sets slot.stamp to p (the largest stamp
//     wins) and writes log[p] = slot, so stamps are log positions and recency
//     order is log order;
//   - a log record p is live iff the stamp of slot log[p] still equals p;
//     eviction pops the log head, skipping stale records, and tombstones the
//     slot (stamp kTomb);
//   - when tombstones or the log would fill up, the live records are
//     compacted, re-stamped in order and re-inserted into a cleared table.
//
// Routes are processed in batches of up to NB queued requests (the queue
// order is the routing order, so the next requests are known in advance):
//   A. every (request, worker) overlap of the batch is searched at once
//      against the caches as they stand, and so is the longest common prefix
//      of every pair of the batch's chains;
//   B. one wavefront makes the routing decisions in order (releases, queue,
//      controller, cost, argmin, loads).  Route b changes only the cache of
//      its worker sigma, and only by adding its chain: with caches
//      prefix-closed along the chains and chained hashes naming whole
//      prefixes, a later request b'' then has overlap
//      max(o[b''][sigma], lcp(b'', b)) on sigma and unchanged overlaps
//      elsewhere.  The cache writes themselves are deferred;
//   C. meanwhile the other three wavefronts apply the touches and inserts of
//      the decided routes, a few routes per claim.
// A route that must evict (and every route in scan mode, where caches need
// not be prefix-closed) stops phase B: once every decided route's writes are
// in, blocks are evicted and the pending requests searched again on that
// worker.
//
// Recency is kept lazily under LRU: until a worker first has to evict, its
// stamps decide nothing, so the writers only insert the blocks it lacks (no
// stamp or log writes, no touches of blocks it holds).  The routes' order and
// worker are kept in a per-episode history; at the first eviction the
// worker's recency is rebuilt from it -- every block gets the stamp of its
// last touch, and the live records are laid down in the log in that order
// (two passes over the worker's routes) -- and from then on the worker is
// maintained eagerly.  Results are those of eager upkeep; episodes whose
// caches never fill skip the recency work altogether.
//
// Frequency eviction keeps, per slot, the key K = f + e of a block whose
// frequency was f after its last update in decay epoch e (epoch = routing
// step / decay_steps); in epoch E its frequency is max(K - E, 1), the eager
// decay applied lazily.  Within one epoch a hit doubles the frequency (capped)
// and an insert leaves it at 1, operations that commute, so the writers apply
// them with atomics in any order; phase B stops at every epoch change until
// the earlier epoch's writes are in.  A parent block is at least as frequent
// as its child and touched later, so caches stay prefix-closed, and the
// victims -- the least frequent blocks, oldest first -- are the oldest blocks
// at frequency 1: the route's own new blocks are such blocks, so there are
// always enough.  Eviction walks the log from its head and skips the more
// frequent records, which keep the head from moving past them.
//
// Memory tiers (LRU): G1 is the tier_g1 newest live records of a worker's log
// and G1 u G2 the tier_g1 + tier_g2 newest, so each is the run of the log
// from a boundary position to the tail, and a block is in G1 iff its stamp is
// at least G1's boundary.  A route moves the boundaries of its worker: its P
// touches add P records to each run and remove the hits whose old records lay
// in it (the writers count those from the stamps atomicMax returns); the
// boundary then walks forward over surplus live records.  Along a cached
// prefix the stamps fall, so the tier overlaps o1 and o12 are found by binary
// search on stamps.  Every route stops the batch so that later requests are
// searched against the new boundaries.
#include <hip/hip_runtime.h>

#include "rk_internal.h"

namespace rk {

constexpr int NT = kEpisodeThreads;
constexpr int NW = NT / 64;
constexpr int kMaxBatch = 64;       // routes per batch (at most one wavefront of lanes)
constexpr int32_t kMoreTurns = 0x40000000;   // flag on an in-flight conversation index: it has a next turn

enum : int32_t { EV_BATCH = 0, EV_DONE = 1, EV_FLUSH = 2, EV_EPOCH = 3, EV_ROOM = 4 };

struct EpArgs {
    int32_t E, W, cache, max_blocks, max_conv, max_inflight, max_rps, max_ctrl_window, probe_mode, NB, tiers,
        max_routes, n_slots, flags;
    const rk_episode_params* params;
    const int64_t* turn_off;
    const int32_t* turn_blocks;
    const int64_t* chain_off;
    const uint64_t* chains;
    const uint32_t* route_rand;
    rk_regime_params regime;
    rk_episode_outputs out;
    unsigned char* ws;
    EpisodeLayout L;
    int32_t* status;
    uint32_t lds_w, lds_inflight, lds_u, lds_roff, lds_batch;
};


// Which copy of the decision loop runs: 0 the full one, 1 the lean one (prefix
// mode, argmin, LRU, no tiers, no controller), 2 the lean one with the load
// controller.
template <int V>
struct LeanTag {
    static constexpr int value = V;
};

struct EpShared {
    int32_t next_e, nlist, jn, jsync, jnext, jp, jpnext, jq, jqnext;
    int32_t qhead, qsize, nb, event, ev_b, ins, remaining, ev, decided, claimed, stop, tdone, h1, h2;
    uint32_t new_head, first_kept, adv;
    int64_t ev_row, ev_total;
    unsigned long long digest, rb_mask;
    int32_t wtot[NW];
};

// Exclusive rank of `flag` among the workgroup's threads (thread order) and the
// total count.  Every thread of the workgroup must call it.
__device__ __forceinline__ int32_t block_scan(bool flag, int32_t* wtot, int32_t& total)
{
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const unsigned long long b = __ballot(flag);
    const int32_t rank = __popcll(b & ((1ull << lane) - 1ull));
    if (lane == 0) wtot[w] = __popcll(b);
    __syncthreads();
    int32_t off = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < NW; ++k) {
        const int32_t v = wtot[k];
        off += k < w ? v : 0;
        tot += v;
    }
    __syncthreads();
    total = tot;
    return off + rank;
}

// Exclusive prefix sum of v over the workgroup's threads (thread order) and the
// total.  Every thread of the workgroup must call it.
__device__ __forceinline__ int32_t block_excl_sum(int32_t v, int32_t* wtot, int32_t& total)
{
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int32_t x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int32_t o = __shfl_up(x, off, 64);
        if (lane >= off) x += o;
    }
    if (lane == 63) wtot[w] = x;
    __syncthreads();
    int32_t off = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < NW; ++k) {
        const int32_t t = wtot[k];
        off += k < w ? t : 0;
        tot += t;
    }
    __syncthreads();
    total = tot;
    return off + x - v;
}

__device__ __forceinline__ void load_slot(const Slot* p, uint64_t& key, uint32_t& stamp)
{
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    key = (uint64_t)v.x | ((uint64_t)v.y << 32);
    stamp = v.z;
}

__device__ __forceinline__ void load_slot(const Slot* p, uint64_t& key, uint32_t& stamp, uint32_t& fkey)
{
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    key = (uint64_t)v.x | ((uint64_t)v.y << 32);
    stamp = v.z;
    fkey = v.w;
}

// Frequency update of a touched block in decay epoch ep: an insert leaves the
// frequency at 1 (K at least ep + 1), a hit doubles max(K - ep, 1) up to
// RK_FREQ_CAP.  Within one epoch these commute, so concurrent touches of a
// block by several routes give the sequential result in any order.
__device__ __forceinline__ void freq_touch(uint32_t* fk, bool inserted, uint32_t ep)
{
    if (inserted) {
        __hip_atomic_fetch_max(fk, ep + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        return;
    }
    uint32_t old = __hip_atomic_load(fk, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    for (;;) {
        const uint32_t f = old > ep + 1u ? old - ep : 1u;
        const uint32_t nf = f >= (uint32_t)RK_FREQ_CAP / 2u ? (uint32_t)RK_FREQ_CAP : 2u * f;
        if (__hip_atomic_compare_exchange_strong(fk, &old, nf + ep, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_WORKGROUP))
            return;
    }
}

constexpr int kWin = 4;    // slots of a group: one lookup reads one aligned group (64 bytes)

// A key's walk starts at the first slot of its aligned group of kWin slots and
// goes group by group; within every group it visits the slots in its own
// rotated order, from slot slot_pref(h) (hash bits independent of the group
// index) on, so concurrent claims in one group rarely aim at the same slot.
// An insert takes the first empty slot of that walk, and slots only fill
// between compactions, so a lookup walking the same order meets the key
// before any empty slot.  Callers load a group in the key's order: element r
// of a loaded group is slot group_slot(h, r).
__device__ __forceinline__ uint64_t home_slot(uint64_t h, uint64_t smask)
{
    return h & smask & ~(uint64_t)(kWin - 1);
}

__device__ __forceinline__ uint32_t slot_pref(uint64_t h) { return (uint32_t)(h >> 62) & (uint32_t)(kWin - 1); }

// Offset within its group of the r-th slot of h's order.
__device__ __forceinline__ uint32_t group_slot(uint64_t h, int r)
{
    return (slot_pref(h) + (uint32_t)r) & (uint32_t)(kWin - 1);
}

// Membership test finishing a walk whose first group (from s, in h's order) is
// loaded; stamp receives the live slot's stamp.
__device__ __forceinline__ bool finish_lookup_stamp(const Slot* t, uint64_t smask, uint64_t h, uint64_t s,
                                                    const uint64_t* k, const uint32_t* st, uint32_t& stamp)
{
#pragma unroll
    for (int r = 0; r < kWin; ++r) {
        if (k[r] == kEmpty) return false;
        if (k[r] == h && st[r] != kTomb) {
            stamp = st[r];
            return true;
        }
    }
    // further groups one slot at a time (rare: a full first group)
    for (uint64_t n = kWin; n <= smask; n += kWin) {
        s = (s + kWin) & smask;
#pragma unroll 1
        for (int r = 0; r < kWin; ++r) {
            uint64_t kk;
            uint32_t ss;
            load_slot(t + s + group_slot(h, r), kk, ss);
            if (kk == kEmpty) return false;
            if (kk == h && ss != kTomb) {
                stamp = ss;
                return true;
            }
        }
    }
    return false;
}

__device__ __forceinline__ bool finish_lookup(const Slot* t, uint64_t smask, uint64_t h, uint64_t s,
                                              const uint64_t* k, const uint32_t* st)
{
    uint32_t stamp;
    return finish_lookup_stamp(t, smask, h, s, k, st, stamp);
}

constexpr int32_t kFullProbe = 64;   // intervals this wide are probed position by position

// Positions sampled in a round over an interval of `span` > kFullProbe blocks:
// about sqrt(span), so two rounds cover span with few probes, and at most 64
// so that the next interval fits one round when span <= 64 * 64.
__device__ __forceinline__ int32_t fanout(int32_t span)
{
    int32_t f = (int32_t)ceilf(sqrtf((float)span));
    f = f < 4 ? 4 : f;
    f = f > 64 ? 64 : f;
    return span > 64 * f ? 64 : f;     // the next interval, at most ceil(span / f) wide, fits 64
}

// Longest cached prefix of the staged chain on the workers j = jfirst,
// jfirst + jstride, ... (< W) handled by this wavefront; worker jspecial's
// search starts at block lo_special (its blocks below are known cached).
// Every round issues, per lane, one probe (two adjacent slots) for each
// unresolved worker before any result is used, so all of the wavefront's
// probes are in flight together.
//   PREFIX mode (caches prefix-closed along the chain): while an interval is
//   wider than kFullProbe a round probes spread positions and keeps the
//   sub-interval holding the first miss; the last round probes every position.
//   SCAN mode: rounds probe blocks [lo, lo + 64) from block 0 on.
template <int JPW>
__device__ void wave_overlaps(const uint64_t* s_chain, int32_t P, int32_t jfirst, int32_t jstride, int32_t W,
                              const Slot* slots, uint64_t S, int mode, int32_t* s_ov, int32_t jspecial,
                              int32_t lo_special)
{
    const int lane = threadIdx.x & 63;
    const uint64_t smask = S - 1;
    int32_t lo[JPW], hi[JPW];
    uint32_t open = 0;
#pragma unroll
    for (int jj = 0; jj < JPW; ++jj) {
        const int32_t j = jfirst + jj * jstride;
        lo[jj] = j == jspecial ? lo_special : 0;
        hi[jj] = P;
        if (j < W) open |= 1u << jj;
    }
    while (open) {
        uint64_t hk[JPW], kw[JPW][kWin], sh0[JPW];
        uint32_t sw[JPW][kWin];
        int32_t q[JPW];
        bool valid[JPW];
#pragma unroll
        for (int jj = 0; jj < JPW; ++jj) {
            valid[jj] = false;
            if (!((open >> jj) & 1u)) continue;
            const int32_t span = hi[jj] - lo[jj];
            if (mode == RK_PROBE_PREFIX && span > kFullProbe) {
                const uint32_t f = (uint32_t)fanout(span);
                q[jj] = lo[jj] + (int32_t)(((uint32_t)(lane + 1) * (uint32_t)span) / f) - 1;
                valid[jj] = (uint32_t)lane < f;
            } else {
                q[jj] = lo[jj] + lane;
                valid[jj] = q[jj] < hi[jj];
            }
            if (valid[jj]) {
                const Slot* t = slots + (uint64_t)(jfirst + jj * jstride) * S;
                hk[jj] = s_chain[q[jj]];
                sh0[jj] = home_slot(hk[jj], smask);
#pragma unroll
                for (int i = 0; i < kWin; ++i) load_slot(t + sh0[jj] + group_slot(hk[jj], i), kw[jj][i], sw[jj][i]);
            }
        }
#pragma unroll
        for (int jj = 0; jj < JPW; ++jj) {
            if (!((open >> jj) & 1u)) continue;
            bool hit = true;
            if (valid[jj]) {
                const Slot* t = slots + (uint64_t)(jfirst + jj * jstride) * S;
                hit = finish_lookup(t, smask, hk[jj], sh0[jj], kw[jj], sw[jj]);
            }
            const unsigned long long miss = __ballot(valid[jj] && !hit);
            const int32_t span = hi[jj] - lo[jj];
            int32_t o = -1;
            if (mode == RK_PROBE_PREFIX && span > kFullProbe) {
                if (miss == 0ull) {
                    o = hi[jj];
                } else {
                    // lane t holds the first missing sample; lanes t and t-1 computed its bounds
                    const int t = __ffsll(miss) - 1;
                    const int32_t qt = __shfl(q[jj], t, 64);
                    const int32_t qprev = __shfl(q[jj], t > 0 ? t - 1 : 0, 64);
                    const int32_t qp = t == 0 ? lo[jj] - 1 : qprev;
                    lo[jj] = qp + 1;
                    hi[jj] = qt;
                    if (hi[jj] == lo[jj]) o = lo[jj];
                }
            } else if (mode == RK_PROBE_PREFIX) {
                o = miss ? lo[jj] + __ffsll(miss) - 1 : hi[jj];
            } else {
                if (miss) o = lo[jj] + __ffsll(miss) - 1;
                else if (lo[jj] + 64 >= hi[jj]) o = hi[jj];
                else lo[jj] += 64;
            }
            if (o >= 0) {
                open &= ~(1u << jj);
                if (lane == 0) s_ov[jfirst + jj * jstride] = o;
            }
        }
    }
}

// Find the live slot of h, or claim the first empty slot of its walk.
// Concurrent callers may insert the same key: they walk the same order, so
// the loser of a claim finds the key in that slot; a slot taken by another key
// sends the walk to the next slot of the order.
__device__ __forceinline__ uint64_t insert_or_touch(Slot* __restrict__ t, uint64_t smask, uint64_t h, int& inserted,
                                                   int32_t* status)
{
    inserted = 0;
    uint64_t g = home_slot(h, smask);
    for (uint64_t n = 0; n <= smask; n += kWin) {
#pragma unroll 1
        for (int r = 0; r < kWin; ++r) {
            const uint64_t sl = g + group_slot(h, r);
            const uint64_t k = __hip_atomic_load(&t[sl].key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            const uint32_t st = t[sl].stamp;
            if (k == h) {
                if (st != kTomb) return sl;
            } else if (k == kEmpty) {
                uint64_t prev = kEmpty;
                if (__hip_atomic_compare_exchange_strong(&t[sl].key, &prev, h, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_WORKGROUP)) {
                    inserted = 1;
                    return sl;
                }
                if (prev == h) return sl;    // a concurrent insert of h claimed it first
            }
        }
        g = (g + kWin) & smask;
    }
    atomicOr(status, RK_DEV_TABLE_FULL);
    return ~0ull;
}

// Same result as insert_or_touch, in one memory round trip in the usual
// case.  A block the overlap search found cached is looked up in its group.
// For a block past the overlap, the claim of the first slot of its order is
// issued together with the loads of the group's other slots: an empty first
// slot proves the key absent (slots never return to empty between
// compactions, and an insert of the key would have taken it), and an occupied
// one usually leaves a free slot further along the group.  Anything else falls
// back to the full walk.
__device__ __forceinline__ uint64_t touch_hinted(Slot* __restrict__ t, uint64_t smask, uint64_t h, bool cached_hint,
                                                 int& inserted, int32_t* status)
{
    const uint64_t s = home_slot(h, smask);
    inserted = 0;
    uint64_t k[kWin];
    uint32_t st[kWin];
    if (cached_hint) {
#pragma unroll
        for (int r = 0; r < kWin; ++r) load_slot(t + s + group_slot(h, r), k[r], st[r]);
#pragma unroll
        for (int r = 0; r < kWin; ++r)
            if (k[r] == h && st[r] != kTomb) return s + group_slot(h, r);
    } else {
        uint64_t prev = kEmpty;
        const uint64_t s0 = s + group_slot(h, 0);
        const bool won = __hip_atomic_compare_exchange_strong(&t[s0].key, &prev, h, __ATOMIC_RELAXED,
                                                              __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
#pragma unroll
        for (int r = 1; r < kWin; ++r) load_slot(t + s + group_slot(h, r), k[r], st[r]);
        if (won) {
            inserted = 1;
            return s0;
        }
        if (prev != h) {           // the first slot holds another key: look further along the group
#pragma unroll
            for (int r = 1; r < kWin; ++r) {
                const uint64_t si = s + group_slot(h, r);
                if (k[r] == h) {
                    if (st[r] != kTomb) return si;
                    continue;
                }
                if (k[r] != kEmpty) continue;
                uint64_t pi = kEmpty;
                if (__hip_atomic_compare_exchange_strong(&t[si].key, &pi, h, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_WORKGROUP)) {
                    inserted = 1;
                    return si;
                }
                break;             // lost a race for the slot: walk from the start
            }
        }
    }
    return insert_or_touch(t, smask, h, inserted, status);
}


// touch_hinted for two keys of a lane at once (act: the key is to be touched;
// hint as there), the claims (compare-and-swap returning the slot's previous
// key) and group loads of both issued before either result is used.
__device__ __forceinline__ void touch_hinted2(Slot* const* t, uint64_t smask, const uint64_t* h, const bool* hint,
                                              const bool* act, uint64_t* sl, int* ins, int32_t* status)
{
    uint64_t s[2], prev[2], k[2][kWin];
    uint32_t st[2][kWin];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        s[u] = home_slot(h[u], smask);
        prev[u] = kEmpty;
        if (act[u] && !hint[u])
            prev[u] = atomicCAS(reinterpret_cast<unsigned long long*>(&t[u][s[u] + group_slot(h[u], 0)].key), kEmpty,
                                h[u]);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const Slot* g = t[u] + s[u];
#pragma unroll
        for (int r = 0; r < kWin; ++r) load_slot(g + group_slot(h[u], r), k[u][r], st[u][r]);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        sl[u] = ~0ull;
        ins[u] = 0;
        if (!act[u]) continue;
        bool done = false;
        if (hint[u]) {
#pragma unroll
            for (int r = 0; r < kWin; ++r)
                if (!done && k[u][r] == h[u] && st[u][r] != kTomb) {
                    sl[u] = s[u] + group_slot(h[u], r);
                    done = true;
                }
        } else if (prev[u] == kEmpty) {
            sl[u] = s[u] + group_slot(h[u], 0);
            ins[u] = 1;
            done = true;
        } else if (prev[u] != h[u]) {   // the first slot holds another key: look further along the group
            bool stop = false;
#pragma unroll
            for (int r = 1; r < kWin; ++r) {
                if (done || stop) continue;
                const uint64_t si = s[u] + group_slot(h[u], r);
                if (k[u][r] == h[u]) {
                    if (st[u][r] != kTomb) {
                        sl[u] = si;
                        done = true;
                    }
                    continue;
                }
                if (k[u][r] != kEmpty) continue;
                uint64_t pi = kEmpty;
                if (__hip_atomic_compare_exchange_strong(&t[u][si].key, &pi, h[u], __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_WORKGROUP)) {
                    sl[u] = si;
                    ins[u] = 1;
                    done = true;
                } else {
                    stop = true;   // lost a race for the slot: walk from the start
                }
            }
        }
        if (!done) sl[u] = insert_or_touch(t[u], smask, h[u], ins[u], status);
    }
}

constexpr int kRU = 4;   // touches a thread keeps in flight while a worker's recency is rebuilt

// touch_hinted(t, smask, h[u], false, ...) for kRU keys (kEmpty: none) with the
// claims and group loads of all of them issued before any result is used; the
// slot of each key (~0 if none) goes to sl.
__device__ __forceinline__ void touch_batch(Slot* __restrict__ t, uint64_t smask, const uint64_t* h, uint64_t* sl,
                                            int32_t* status)
{
    uint64_t s0[kRU], prev[kRU], k[kRU][kWin];
    uint32_t stv[kRU][kWin];
    // the claims return the slots' previous keys and the group loads use masked addresses (an
    // empty key reads the first group), so nothing waits before all are issued
#pragma unroll
    for (int u = 0; u < kRU; ++u) {
        const uint64_t s = home_slot(h[u], smask);
        s0[u] = s + group_slot(h[u], 0);
        prev[u] = kEmpty;
        if (h[u] != kEmpty) prev[u] = atomicCAS(reinterpret_cast<unsigned long long*>(&t[s0[u]].key), kEmpty, h[u]);
    }
#pragma unroll
    for (int u = 0; u < kRU; ++u) {
        const Slot* g = t + ((uint64_t)(-(int64_t)(h[u] != kEmpty)) & home_slot(h[u], smask));
#pragma unroll
        for (int r = 1; r < kWin; ++r) load_slot(g + group_slot(h[u], r), k[u][r], stv[u][r]);
    }
#pragma unroll
    for (int u = 0; u < kRU; ++u) {
        sl[u] = ~0ull;
        if (h[u] == kEmpty) continue;
        if (prev[u] == kEmpty || prev[u] == h[u]) {
            sl[u] = s0[u];
            continue;
        }
        const uint64_t s = home_slot(h[u], smask);
        bool done = false, retry = false;
#pragma unroll
        for (int r = 1; r < kWin && !done && !retry; ++r) {
            const uint64_t si = s + group_slot(h[u], r);
            if (k[u][r] == h[u]) {
                if (stv[u][r] != kTomb) {
                    sl[u] = si;
                    done = true;
                }
                continue;
            }
            if (k[u][r] != kEmpty) continue;
            uint64_t pi = kEmpty;
            if (__hip_atomic_compare_exchange_strong(&t[si].key, &pi, h[u], __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_WORKGROUP)) {
                sl[u] = si;
                done = true;
            } else {
                retry = true;      // lost a race for the slot: walk from the start
            }
        }
        if (!done) {
            int ins;
            sl[u] = insert_or_touch(t, smask, h[u], ins, status);
        }
    }
}

// The live slot of each of kRU keys (kEmpty: none) and whether its stamp equals
// st[u]; the groups of all of them are loaded before any result is used.
__device__ __forceinline__ void find_batch(const Slot* __restrict__ t, uint64_t smask, const uint64_t* h, uint64_t* sl,
                                           const uint32_t* st, bool* last)
{
    uint64_t k[kRU][kWin];
    uint32_t stv[kRU][kWin];
#pragma unroll
    for (int u = 0; u < kRU; ++u) {
        const uint64_t s = home_slot(h[u], smask);
#pragma unroll
        for (int r = 0; r < kWin; ++r) {
            k[u][r] = kEmpty;
            stv[u][r] = 0;
            if (h[u] != kEmpty) load_slot(t + s + group_slot(h[u], r), k[u][r], stv[u][r]);
        }
    }
#pragma unroll
    for (int u = 0; u < kRU; ++u) {
        sl[u] = ~0ull;
        last[u] = false;
        if (h[u] == kEmpty) continue;
        const uint64_t s = home_slot(h[u], smask);
        uint32_t stamp = 0;
        bool found = false;
#pragma unroll
        for (int r = 0; r < kWin && !found; ++r) {
            if (k[u][r] == kEmpty) break;
            if (k[u][r] == h[u] && stv[u][r] != kTomb) {
                sl[u] = s + group_slot(h[u], r);
                stamp = stv[u][r];
                found = true;
            }
        }
        if (!found) {
            // further groups (a full first group)
            uint64_t g = s;
            for (uint64_t n = kWin; n <= smask && !found; n += kWin) {
                g = (g + kWin) & smask;
                bool stop = false;
#pragma unroll 1
                for (int r = 0; r < kWin && !found && !stop; ++r) {
                    uint64_t kk;
                    uint32_t ss;
                    load_slot(t + g + group_slot(h[u], r), kk, ss);
                    if (kk == kEmpty) stop = true;
                    else if (kk == h[u] && ss != kTomb) {
                        sl[u] = g + group_slot(h[u], r);
                        stamp = ss;
                        found = true;
                    }
                }
                if (stop) break;
            }
        }
        last[u] = found && stamp == st[u];
    }
}

static __device__ __forceinline__ void ep_wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Minimum over the wavefront: DPP moves within each row of 16 lanes (pair
// swap, quad swap, half-row mirror, row mirror), then the four row minima.
static __device__ __forceinline__ uint32_t ep_wave_min_u32(uint32_t v)
{
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0xB1, 0xF, 0xF, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x4E, 0xF, 0xF, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x141, 0xF, 0xF, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x140, 0xF, 0xF, false));
    const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)v, 0);
    const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)v, 16);
    const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)v, 32);
    const uint32_t r3 = (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
    return min(min(r0, r1), min(r2, r3));
}

constexpr int KI = 4;   // searches a thread keeps in flight together
constexpr int KP = 4;   // batch pairs a thread searches together for their common prefix

// Longest cached prefix for items i = threadIdx.x, + NT, ... < n: item i
// names a chain, its length, its hash at block 0 and a worker table (info,
// false for an item this search does not handle), and receives the first
// chain position missing from the table (put).  A first probe of every item's
// block 0 decides the items that miss it (o = 0) and lists the others in
// `list`; those then run a binary search over [1, P), exact for tables
// prefix-closed along the chain, several per thread at most.  A step loads
// the probed block's group and the chain hashes of both positions the next
// step may probe, so a step costs one memory round trip; the KI searches of a
// thread issue the same loads from addresses chosen by masks (a finished
// search reads the first group of the slots and the first chain hash again),
// so that no branch separates them and all are in flight together.
template <class Info, class Put>
__device__ __forceinline__ void prefix_searches(int32_t n, const Info& info, const Put& put, const Slot* slots,
                                                uint64_t S, const uint64_t* chains, uint16_t* list,
                                                int32_t* nlist)
{
    const uint64_t smask = S - 1;
    {
        const int lane = threadIdx.x & 63;
        __syncthreads();           // the list's previous users are done
        if (threadIdx.x == 0) *nlist = 0;
        __syncthreads();
        for (int32_t base = 0; base < n; base += NT * KI) {
            uint64_t tbo[KI], h0[KI], kw[KI][kWin];
            uint32_t sw[KI][kWin];
            bool own[KI];
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                const int32_t i = base + u * NT + (int32_t)threadIdx.x;
                const uint64_t* ch = chains;
                int32_t P = 0, j = 0;
                h0[u] = 0ull;
                own[u] = i < n && info(i, ch, P, j, h0[u]);
                if (own[u] && P == 0) {
                    put(i, 0);
                    own[u] = false;
                }
                tbo[u] = (uint64_t)j * S;
                const Slot* g = slots + ((uint64_t)(-(int64_t)own[u]) & (tbo[u] + home_slot(h0[u], smask)));
#pragma unroll
                for (int x = 0; x < kWin; ++x) load_slot(g + group_slot(h0[u], x), kw[u][x], sw[u][x]);
            }
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                const int32_t i = base + u * NT + (int32_t)threadIdx.x;
                bool hit = false;
                if (own[u]) {
                    hit = finish_lookup(slots + tbo[u], smask, h0[u], home_slot(h0[u], smask), kw[u], sw[u]);
                    if (!hit) put(i, 0);
                }
                const unsigned long long m = __ballot(hit);
                int32_t wb = 0;
                if (lane == 0 && m) wb = atomicAdd(nlist, (int32_t)__popcll(m));
                wb = __builtin_amdgcn_readfirstlane(wb);
                if (hit) list[wb + __popcll(m & ((1ull << lane) - 1ull))] = (uint16_t)i;
            }
        }
        __syncthreads();
        n = *nlist;
    }
    for (int32_t base = 0; base < n; base += NT * KI) {
        int32_t lo[KI], hi[KI];
        int64_t cb[KI];
        uint64_t tbo[KI], hk[KI];
        bool own[KI];
#pragma unroll
        for (int u = 0; u < KI; ++u) {
            const int32_t i2 = base + u * NT + (int32_t)threadIdx.x;
            lo[u] = 0;
            hi[u] = 0;
            cb[u] = 0;
            tbo[u] = 0;
            own[u] = false;
            if (i2 < n) {
                const uint64_t* ch = chains;
                int32_t P, j;
                uint64_t h0;
                own[u] = info((int32_t)list[i2], ch, P, j, h0);
                lo[u] = 1;                 // block 0 is cached
                hi[u] = P;
                cb[u] = ch - chains;
                tbo[u] = (uint64_t)j * S;
            }
        }
        bool act = false;
#pragma unroll
        for (int u = 0; u < KI; ++u) act |= lo[u] < hi[u];
        // (the chains are not empty when some search of the thread is open)
#pragma unroll
        for (int u = 0; u < KI; ++u) {
            const int64_t m = -(int64_t)(lo[u] < hi[u]);
            hk[u] = act ? chains[m & (cb[u] + ((lo[u] + hi[u]) >> 1))] : 0ull;
        }
        for (;;) {
            bool any = false;
#pragma unroll
            for (int u = 0; u < KI; ++u) any |= lo[u] < hi[u];
            if (!any) break;
            int32_t mid[KI];
            uint64_t kw[KI][kWin], hc[KI], hd[KI];
            uint32_t sw[KI][kWin];
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                mid[u] = (lo[u] + hi[u]) >> 1;
                const int64_t m = -(int64_t)(lo[u] < hi[u]);
                // the next probe after a hit (hc) and after a miss (hd); an empty range reads block 0
                const int32_t mh = mid[u] + 1 < hi[u] ? (mid[u] + 1 + hi[u]) >> 1 : 0;
                const int32_t mm = lo[u] < mid[u] ? (lo[u] + mid[u]) >> 1 : 0;
                const Slot* g = slots + ((uint64_t)m & (tbo[u] + home_slot(hk[u], smask)));
#pragma unroll
                for (int x = 0; x < kWin; ++x) load_slot(g + group_slot(hk[u], x), kw[u][x], sw[u][x]);
                hc[u] = chains[m & (cb[u] + mh)];
                hd[u] = chains[m & (cb[u] + mm)];
            }
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                if (lo[u] < hi[u]) {
                    if (finish_lookup(slots + tbo[u], smask, hk[u], home_slot(hk[u], smask), kw[u], sw[u])) {
                        lo[u] = mid[u] + 1;
                        hk[u] = hc[u];
                    } else {
                        hi[u] = mid[u];
                        hk[u] = hd[u];
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < KI; ++u) {
            const int32_t i2 = base + u * NT + (int32_t)threadIdx.x;
            if (i2 < n && own[u]) put((int32_t)list[i2], lo[u]);
        }
    }
}

// ---- the run index of workers that keep no recency yet
//
// Until a worker first evicts (under LRU, in prefix mode), its cached set is
// the union of the prefixes of the chains routed to it, i.e. a trie of blocks;
// a route adds one path to that trie, the blocks [o, P) past the overlap o it
// was decided with.  Such a path is a run.  A run is entered in the index under
// the hash of its first block and under the hash of every block of it at a
// chain position that is a multiple of kCkpt (a checkpoint); each entry names
// the run's chain and end.  The chained hash names the whole prefix, so an
// entry keyed by the hash of block p of another chain is found exactly when
// that chain reaches the entry's block, and since every cached block belongs
// to exactly one run, block p at a checkpoint position is cached iff the
// index holds it.  Caches are prefix-closed, so that membership is monotone
// along a chain: a binary search over a chain's checkpoints finds the last
// cached checkpoint c, and the first miss lies in (c, c + kCkpt].  There the
// search follows c's run while the two chains agree (the first differing hash
// by binary search) and looks up a run that starts where they part or where
// the run ends; a branch off a run is always the first block of a later run.
// A few entries per route replace an insert per new block.  All workers of an
// episode share one table of 16-byte RunSlots, probed from run_home in
// aligned pairs.
constexpr int kRunWin = 2;
constexpr int kCkpt = 1 << kCkptLog;

__device__ __forceinline__ uint64_t run_home(uint64_t h, int32_t j, uint64_t rsmask)
{
    return (h + (uint64_t)(j + 1) * 0x9E3779B97F4A7C15ull) & rsmask & ~(uint64_t)(kRunWin - 1);
}

// chain base index (below 2^40), worker (below 256) and end (below 2^16) of a run
__device__ __forceinline__ uint64_t run_val(int64_t cb, int32_t j, int32_t end)
{
    return ((uint64_t)cb << 24) | ((uint64_t)(uint32_t)j << 16) | (uint64_t)(uint32_t)end;
}

// index entries of a run over blocks [st, P), st < P: its first block and the checkpoints past it
__device__ __forceinline__ int32_t run_entries(int32_t st, int32_t P)
{
    return 1 + ((P - 1) >> kCkptLog) - (st >> kCkptLog);
}

// chain position of entry k of the run over [st, P)
__device__ __forceinline__ int32_t run_entry_pos(int32_t st, int32_t k)
{
    return k == 0 ? st : (((st >> kCkptLog) + k) << kCkptLog);
}

__device__ __forceinline__ void load_run(const RunSlot* p, uint64_t& key, uint64_t& val)
{
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    key = (uint64_t)v.x | ((uint64_t)v.y << 32);
    val = (uint64_t)v.z | ((uint64_t)v.w << 32);
}

// Entry of worker j keyed h, whose first pair (from g) is loaded in k, v;
// false when there is none.
__device__ __forceinline__ bool run_finish(const RunSlot* rt, uint64_t rsmask, uint64_t h, int32_t j, uint64_t g,
                                           const uint64_t* k, const uint64_t* v, uint64_t& val)
{
#pragma unroll
    for (int r = 0; r < kRunWin; ++r) {
        if (k[r] == kEmpty) return false;
        if (k[r] == h && (int32_t)((v[r] >> 16) & 0xFFu) == j) {
            val = v[r];
            return true;
        }
    }
    for (uint64_t n = kRunWin; n <= rsmask; n += kRunWin) {
        g = (g + kRunWin) & rsmask;
#pragma unroll 1
        for (int r = 0; r < kRunWin; ++r) {
            uint64_t kk, vv;
            load_run(rt + g + r, kk, vv);
            if (kk == kEmpty) return false;
            if (kk == h && (int32_t)((vv >> 16) & 0xFFu) == j) {
                val = vv;
                return true;
            }
        }
    }
    return false;
}

// Add the entry (h, val) of worker j.  Each block belongs to one run and is
// entered at most once, so a slot already holding h belongs to another
// worker's run; concurrent adds claim empty slots by compare-and-swap.
__device__ __forceinline__ void run_insert(RunSlot* rt, uint64_t rsmask, uint64_t h, int32_t j, uint64_t val,
                                           int32_t* status)
{
    uint64_t g = run_home(h, j, rsmask);
    for (uint64_t n = 0; n <= rsmask; n += kRunWin) {
#pragma unroll 1
        for (int r = 0; r < kRunWin; ++r) {
            uint64_t prev = kEmpty;
            if (__hip_atomic_compare_exchange_strong(&rt[g + r].key, &prev, h, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_WORKGROUP)) {
                rt[g + r].val = val;
                return;
            }
        }
        g = (g + kRunWin) & rsmask;
    }
    atomicOr(status, RK_DEV_TABLE_FULL);
}

// Longest cached prefix for items i = threadIdx.x, + NT, ... < n on workers
// without recency; info(i, ch, P, j, h0) and put as in prefix_searches.  As
// there, a first probe of block 0 (checkpoint 0) decides the items that miss
// it and lists the others, which the full search then takes up from
// checkpoint 0 again, several per thread at most.  A step of the checkpoint search
// (CKPT) loads a run pair and the chain hashes at both checkpoints the next
// step may probe; a step of the walk inside the last interval loads the
// item's hash at its current block (HASH), a run pair (LOOK), or the two
// hashes a binary-search step compares (CMP).  lim is the first position known
// to be missing (or P).  Every item of a thread issues the same four loads, a
// run pair and two chain hashes, from addresses chosen by its mode (an item
// that needs fewer reads the index's first pair or the first chain hash
// again), so that no branch separates the KI items' loads and all of them are
// in flight together; a wavefront skips a load that none of its lanes needs.
template <class Info, class Put>
__device__ __forceinline__ void run_searches(int32_t n, const Info& info, const Put& put, const RunSlot* rt,
                                             uint64_t rsmask, const uint64_t* chains, uint16_t* list,
                                             int32_t* nlist)
{
    // first probe of every item, its block 0 (hash known): a miss decides o = 0, a hit puts the
    // item on the list that the full search then takes up, several hits per thread at most
    {
        const int lane = threadIdx.x & 63;
        __syncthreads();           // the list's previous users are done
        if (threadIdx.x == 0) *nlist = 0;
        __syncthreads();
        for (int32_t base = 0; base < n; base += NT * KI) {
            int32_t jw[KI];
            uint64_t h0[KI], x0[KI], x1[KI], y0[KI], y1[KI];
            bool own[KI];
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                const int32_t i = base + u * NT + (int32_t)threadIdx.x;
                const uint64_t* ch = chains;
                int32_t P = 0;
                jw[u] = 0;
                h0[u] = 0ull;
                own[u] = i < n && info(i, ch, P, jw[u], h0[u]);
                if (own[u] && P == 0) {
                    put(i, 0);
                    own[u] = false;
                }
                const uint64_t g = (uint64_t)(-(int64_t)own[u]) & run_home(h0[u], jw[u], rsmask);
                load_run(rt + g, x0[u], y0[u]);
                x1[u] = y1[u] = 0ull;
                if constexpr (kRunWin > 1) load_run(rt + g + 1, x1[u], y1[u]);
            }
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                const int32_t i = base + u * NT + (int32_t)threadIdx.x;
                bool hit = false;
                if (own[u]) {
                    const uint64_t kk[2] = {x0[u], x1[u]}, vv[2] = {y0[u], y1[u]};
                    uint64_t val;
                    hit = run_finish(rt, rsmask, h0[u], jw[u], run_home(h0[u], jw[u], rsmask), kk, vv, val);
                    if (!hit) put(i, 0);
                }
                const unsigned long long m = __ballot(hit);
                int32_t wb = 0;
                if (lane == 0 && m) wb = atomicAdd(nlist, (int32_t)__popcll(m));
                wb = __builtin_amdgcn_readfirstlane(wb);
                if (hit) list[wb + __popcll(m & ((1ull << lane) - 1ull))] = (uint16_t)i;
            }
        }
        __syncthreads();
        n = *nlist;
    }
    enum : int32_t { DONE = 0, HASH = 1, LOOK = 2, CMP = 3, CKPT = 4 };
    for (int32_t base = 0; base < n; base += NT * KI) {
        int64_t cb[KI], rcb[KI];     // chain bases of the item and of the run it follows
        int32_t P[KI], jw[KI], o[KI], lo[KI], hi[KI], mode[KI], km[KI], lim[KI];
        uint64_t hq[KI], qhi[KI];
        bool own[KI], qok[KI];
#pragma unroll
        for (int u = 0; u < KI; ++u) {
            const int32_t i2 = base + u * NT + (int32_t)threadIdx.x;
            const int32_t i = i2 < n ? (int32_t)list[i2] : 0;
            const uint64_t* ch = chains;
            P[u] = 0;
            jw[u] = 0;
            o[u] = 0;
            hq[u] = 0ull;
            qhi[u] = 0ull;
            qok[u] = false;
            own[u] = i2 < n && info(i, ch, P[u], jw[u], hq[u]);
            cb[u] = ch - chains;
            rcb[u] = 0;
            // checkpoints [lo, hi) undecided (those below lo cached, from hi on missing); km is
            // probed next, first checkpoint 0, whose hash is known.  While the checkpoint search
            // runs, rcb and o hold the chain and end of the run of the last cached checkpoint.
            lo[u] = 0;
            hi[u] = (P[u] + kCkpt - 1) >> kCkptLog;
            km[u] = 0;
            lim[u] = P[u];
            mode[u] = own[u] && P[u] > 0 ? CKPT : DONE;
        }
        for (;;) {
            bool any = false;
#pragma unroll
            for (int u = 0; u < KI; ++u) any |= mode[u] != DONE;
            if (!any) break;
            uint64_t x0[KI], x1[KI], y0[KI], y1[KI], hc[KI], hd[KI];
            int32_t mid[KI];
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                mid[u] = (lo[u] + hi[u]) >> 1;
                const int32_t md = mode[u];
                // all-ones masks of the item's mode: addresses by masks, not branches
                const int32_t mC = -(int32_t)(md == CKPT), mH = -(int32_t)(md == HASH), mM = -(int32_t)(md == CMP);
                const int32_t mP = -(int32_t)(md == CKPT || md == LOOK);
                // CKPT: the next probes after a hit (hc) and after a miss (hd)
                const int32_t mh = km[u] + 1 < hi[u] ? (km[u] + 1 + hi[u]) >> 1 : 0;
                const int32_t mm = lo[u] < km[u] ? (lo[u] + km[u]) >> 1 : 0;
                const int32_t ic = (mC & (mh << kCkptLog)) | (mH & o[u]) | (mM & mid[u]);
                const int32_t id = (mC & (mm << kCkptLog)) | (mM & mid[u]);
                const int64_t bc = (int64_t)(mC | mH | mM) & cb[u];
                const int64_t bd = ((int64_t)mC & cb[u]) | ((int64_t)mM & rcb[u]);
                const uint64_t g = (uint64_t)(int64_t)mP & run_home(hq[u], jw[u], rsmask);
                x0[u] = y0[u] = x1[u] = y1[u] = hc[u] = hd[u] = 0ull;
                if (__ballot(mP != 0)) {
                    load_run(rt + g, x0[u], y0[u]);
                    load_run(rt + g + 1, x1[u], y1[u]);
                }
                if (__ballot((mC | mH | mM) != 0)) hc[u] = chains[bc + ic];
                if (__ballot((mC | mM) != 0)) hd[u] = chains[bd + id];
            }
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                if (mode[u] == CKPT) {
                    const uint64_t kk[2] = {x0[u], x1[u]}, vv[2] = {y0[u], y1[u]};
                    uint64_t val = 0ull;
                    if (run_finish(rt, rsmask, hq[u], jw[u], run_home(hq[u], jw[u], rsmask), kk, vv, val)) {
                        rcb[u] = (int64_t)(val >> 24);
                        o[u] = (int32_t)(val & 0xFFFFu);
                        lo[u] = km[u] + 1;
                        hq[u] = hc[u];
                    } else {
                        hi[u] = km[u];
                        hq[u] = hd[u];
                    }
                    km[u] = (lo[u] + hi[u]) >> 1;
                    if (lo[u] >= hi[u]) {
                        if (lo[u] == 0) {
                            mode[u] = DONE;          // block 0 missing: o stays 0
                        } else {
                            // the last cached checkpoint c is held by the run at rcb, ending at o; the
                            // first miss lies in (c, c + kCkpt], or at P
                            const int32_t c = (lo[u] - 1) << kCkptLog;
                            lim[u] = min(P[u], lo[u] << kCkptLog);
                            const int32_t m = min(lim[u], o[u]);
                            lo[u] = c + 1;
                            hi[u] = m;
                            qok[u] = false;
                            if (lo[u] >= hi[u]) {
                                o[u] = m;
                                mode[u] = o[u] < lim[u] ? HASH : DONE;
                            } else {
                                mode[u] = CMP;
                            }
                        }
                    }
                } else if (mode[u] == HASH) {
                    hq[u] = hc[u];
                    mode[u] = LOOK;
                } else if (mode[u] == LOOK) {
                    const uint64_t kk[2] = {x0[u], x1[u]}, vv[2] = {y0[u], y1[u]};
                    uint64_t val = 0ull;
                    if (!run_finish(rt, rsmask, hq[u], jw[u], run_home(hq[u], jw[u], rsmask), kk, vv, val)) {
                        mode[u] = DONE;
                    } else {
                        // the entry's run holds blocks [o, end) of the chain at val >> 24
                        rcb[u] = (int64_t)(val >> 24);
                        const int32_t m = min(lim[u], (int32_t)(val & 0xFFFFu));
                        lo[u] = o[u] + 1;
                        hi[u] = m;
                        qok[u] = false;
                        if (lo[u] >= hi[u]) {
                            o[u] = m;
                            mode[u] = o[u] < lim[u] ? HASH : DONE;
                        } else {
                            mode[u] = CMP;
                        }
                    }
                } else if (mode[u] == CMP) {
                    // first block in [lo, hi) where the chains differ (hi: the run's end or lim)
                    if (hc[u] == hd[u]) {
                        lo[u] = mid[u] + 1;
                    } else {
                        hi[u] = mid[u];
                        qhi[u] = hc[u];
                        qok[u] = true;
                    }
                    if (lo[u] >= hi[u]) {
                        o[u] = lo[u];
                        if (o[u] >= lim[u]) {
                            mode[u] = DONE;
                        } else if (qok[u]) {
                            hq[u] = qhi[u];      // the item's hash at hi, loaded by the step that set hi
                            mode[u] = LOOK;
                        } else {
                            mode[u] = HASH;
                        }
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < KI; ++u) {
            const int32_t i2 = base + u * NT + (int32_t)threadIdx.x;
            if (own[u]) put((int32_t)list[i2], o[u]);
        }
    }
}

// First position k < hi of each item's chain whose block is not held at a
// stamp >= bound (not in the tier run that starts at log position bound), for
// items i = threadIdx.x, + NT, ... < n; info names the chain, hi, the worker
// table and the bound.  Binary search when the tier's blocks form a prefix of
// the chain (prefix-closed caches: stamps fall along a cached prefix), else a
// scan from block 0.
template <class Info, class Put>
__device__ __forceinline__ void tier_searches(int32_t n, bool bsearch, const Info& info, const Put& put,
                                              const Slot* slots, uint64_t S)
{
    const uint64_t smask = S - 1;
    for (int32_t base = 0; base < n; base += NT * KI) {
        int32_t lo[KI], hi[KI];
        const uint64_t* ch[KI];
        const Slot* tb[KI];
        uint32_t bound[KI];
#pragma unroll
        for (int u = 0; u < KI; ++u) {
            const int32_t i = base + u * NT + (int32_t)threadIdx.x;
            lo[u] = 0;
            hi[u] = 0;
            ch[u] = nullptr;
            tb[u] = slots;
            bound[u] = 0;
            if (i < n) {
                int32_t j;
                info(i, ch[u], hi[u], j, bound[u]);
                tb[u] = slots + (uint64_t)j * S;
            }
        }
        for (;;) {
            bool any = false;
            int32_t mid[KI];
            uint64_t hk[KI];
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                mid[u] = bsearch ? (lo[u] + hi[u]) >> 1 : lo[u];
                hk[u] = 0ull;
                if (lo[u] < hi[u]) {
                    hk[u] = ch[u][mid[u]];
                    any = true;
                }
            }
            if (!any) break;
            uint64_t kw[KI][kWin];
            uint32_t sw[KI][kWin];
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                if (lo[u] < hi[u]) {
                    const uint64_t s0 = home_slot(hk[u], smask);
#pragma unroll
                    for (int x = 0; x < kWin; ++x) load_slot(tb[u] + s0 + group_slot(hk[u], x), kw[u][x], sw[u][x]);
                }
            }
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                if (lo[u] < hi[u]) {
                    uint32_t st = 0;
                    const bool in = finish_lookup_stamp(tb[u], smask, hk[u], home_slot(hk[u], smask), kw[u], sw[u], st) &&
                                    st >= bound[u];
                    if (in) lo[u] = mid[u] + 1;
                    else hi[u] = mid[u];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < KI; ++u) {
            const int32_t i = base + u * NT + (int32_t)threadIdx.x;
            if (i < n) put(i, lo[u]);
        }
    }
}

// Offsets of the batch arrays in LDS (bytes), shared by the launch and the kernel.
struct BatchLayout {
    uint32_t rcb, rlast, rfirst, o_cur, o_tab, rc, rk, rturn, rP, rsig, rotab, rstamp, rep, rstep, rreg, revc, revd, rrnd, lcp,
        items, pairs, nxcb, nxfirst, nxP, nxo, lcp2, pval, wend, t1, t12, bytes;
};

__host__ __device__ inline BatchLayout batch_layout(int32_t NB, int32_t W, bool tiers)
{
    BatchLayout b;
    uint32_t o = 0;
    auto take = [&](uint32_t n, uint32_t al) {
        o = (o + al - 1) / al * al;
        const uint32_t r = o;
        o += n;
        return r;
    };
    const uint32_t nb = (uint32_t)NB, w = (uint32_t)W;
    b.rcb = take(nb * 8, 8);
    b.rlast = take(nb * 8, 8);
    b.rfirst = take(nb * 8, 8);
    b.o_cur = take(nb * w * 4, 4);
    b.o_tab = take(nb * w * 4, 4);
    b.rc = take(nb * 4, 4);
    b.rk = take(nb * 4, 4);
    b.rturn = take(nb * 4, 4);
    b.rP = take(nb * 4, 4);
    b.rsig = take(nb * 4, 4);
    b.rotab = take(nb * 4, 4);
    b.rstamp = take(nb * 4, 4);
    b.rep = take(nb * 4, 4);
    b.rstep = take(nb * 4, 4);
    b.rreg = take(nb * 4, 4);
    b.revc = take(nb * 4, 4);
    b.revd = take(nb * 8, 8);
    b.rrnd = take(nb * 8, 4);
    b.lcp = take(nb * nb * 2, 4);
    b.items = take(nb * w * 2, 4);
    b.pairs = take(nb * nb * 2 + 2, 4);
    b.nxcb = take(nb * 8, 8);
    b.nxfirst = take(nb * 8, 8);
    b.nxP = take(nb * 4, 4);
    b.nxo = take(nb * w * 4, 4);
    b.wend = take(nb * 4, 4);
    b.lcp2 = take(nb * nb * 2, 4);
    b.pval = take(nb * nb * 2 + 2, 4);
    b.t1 = take(tiers ? nb * w * 2 : 0, 4);
    b.t12 = take(tiers ? nb * w * 2 : 0, 4);
    b.bytes = (o + 15) / 16 * 16;
    return b;
}

// The episode queue of a launch with fewer workspaces than episodes starts at 0.
__global__ void episode_queue_init(int32_t* __restrict__ q)
{
    if (threadIdx.x == 0) *q = 0;
}

// Two waves per SIMD: two episodes share a CU (the sweep has more episodes than CUs).
// With one workspace per episode, workgroup x runs episode x.  With fewer
// workspaces (n_slots < E), workgroup x owns workspace x and takes episodes from
// the launch's queue counter in index order until none is left.  An episode
// clears what it uses of its workspace itself, so no launch needs the
// workspace cleared beforehand.
// The queued loop is a kernel of its own (Queued = true): a loop around the
// episode keeps more values live across it, and the one-episode kernel keeps
// its register allocation.
// ------------------------------------------------- the lean decision loop
// Pointers into LDS and global memory with their address spaces spelled out, for code outside
// the kernel body (a 32-bit LDS address, a global address).
template <typename T>
using lds_p = __attribute__((address_space(3))) T*;
template <typename T>
using glb_p = __attribute__((address_space(1))) T*;

template <typename T>
__device__ __forceinline__ lds_p<T> lds_at(uint32_t off)
{
    return (lds_p<T>)(uintptr_t)off;
}
template <typename T>
__device__ __forceinline__ uint32_t lds_off(T* p)
{
    return (uint32_t)(uintptr_t)(lds_p<T>)p;
}

// v, the same in every lane, as a wave-uniform value (every 32-bit word through readfirstlane):
// the arguments of a function arrive in vector registers.
template <typename T>
__device__ __forceinline__ T wave_uniform(const T& v)
{
    static_assert(sizeof(T) % 4 == 0, "32-bit words");
    T r;
    const int32_t* src = reinterpret_cast<const int32_t*>(&v);
    int32_t* dst = reinterpret_cast<int32_t*>(&r);
#pragma unroll
    for (int i = 0; i < (int)(sizeof(T) / 4); ++i) dst[i] = __builtin_amdgcn_readfirstlane(src[i]);
    return r;
}

// What the lean decision loop reads: LDS addresses of the episode's arrays, global arrays and
// the episode's parameters.
struct LeanCtx {
    uint32_t sh, s_A, s_N, s_tail, s_live, s_used, s_head, s_stamped, s_stw, s_stP, s_stc, s_stepn, s_u;
    uint32_t r_P, r_c, r_k, o_cur, o_tab, lcp, r_sig, r_wend, r_stamp, r_ep, r_otab, r_step, r_reg, r_evc, r_evd;
    glb_p<int32_t> g_hist;
    glb_p<int32_t> g_next;
    glb_p<int32_t> g_queue;
    glb_p<float> out_cost;
    glb_p<int32_t> status;
    int64_t out_base, ctrl_thr;
    uint64_t used_limit, R;
    int32_t W, NB, nb, t0, H, rps, qcap, cache, ctrl_window, ctrl_den, cap_blocks;
    float w_ov, w_act, w_sat, ctrl_w_ov, inv_cap;
};

// The routing sequence's state, carried from one call to the next.
struct LeanState {
    int32_t t, s, r_in_step, n_step, s_slot, c_pos, room_b, step_open, prev_active;
    int64_t u_sum, u_tot;
    int64_t tot[8];
};

// The decisions of wavefront 0 for an episode in prefix mode, routed by argmin under LRU,
// without memory tiers, frequency decay or the regime controller (LC: with the load
// controller), from route t up to the batch's end or a stop, as the general loop of the kernel
// takes them: the same routes, outputs and state.  It is a function of its own so that its
// registers are its own and not those of the whole episode kernel, which keeps the serial
// chain of decisions short: the batch's per-route inputs sit in registers (lane b holds route
// b's), the load release of a step is applied in registers, and the next route's overlaps are
// read from LDS while the current route's outputs are written.
template <bool LC>
__device__ __noinline__ void lean_decide(const LeanCtx c_arg, LeanState* st_arg)
{
    const int lane = (int)(threadIdx.x & 63);
    const LeanCtx c = wave_uniform(c_arg);
    LeanState* const st = wave_uniform(st_arg);
    const LeanState st0 = wave_uniform(*st);
    const lds_p<EpShared> sh = lds_at<EpShared>(c.sh);
    const lds_p<int32_t> s_A = lds_at<int32_t>(c.s_A), s_N = lds_at<int32_t>(c.s_N);
    const lds_p<uint32_t> s_tail = lds_at<uint32_t>(c.s_tail), s_head = lds_at<uint32_t>(c.s_head);
    const lds_p<int32_t> s_live = lds_at<int32_t>(c.s_live), s_used = lds_at<int32_t>(c.s_used);
    const lds_p<int32_t> s_stamped = lds_at<int32_t>(c.s_stamped);
    const lds_p<int32_t> s_stw = lds_at<int32_t>(c.s_stw), s_stP = lds_at<int32_t>(c.s_stP);
    const lds_p<int32_t> s_stc = lds_at<int32_t>(c.s_stc), s_stepn = lds_at<int32_t>(c.s_stepn);
    const lds_p<int64_t> s_u = lds_at<int64_t>(c.s_u);
    const lds_p<int32_t> r_P = lds_at<int32_t>(c.r_P), r_c = lds_at<int32_t>(c.r_c), r_k = lds_at<int32_t>(c.r_k);
    const lds_p<int32_t> o_cur = lds_at<int32_t>(c.o_cur), o_tab = lds_at<int32_t>(c.o_tab);
    const lds_p<uint16_t> l_lcp = lds_at<uint16_t>(c.lcp);
    const lds_p<int32_t> r_sig = lds_at<int32_t>(c.r_sig), r_wend = lds_at<int32_t>(c.r_wend);
    const lds_p<uint32_t> r_stamp = lds_at<uint32_t>(c.r_stamp), r_ep = lds_at<uint32_t>(c.r_ep);
    const lds_p<int32_t> r_otab = lds_at<int32_t>(c.r_otab), r_step = lds_at<int32_t>(c.r_step);
    const lds_p<int32_t> r_reg = lds_at<int32_t>(c.r_reg), r_evc = lds_at<int32_t>(c.r_evc);
    const lds_p<uint64_t> r_evd = lds_at<uint64_t>(c.r_evd);
    const int32_t W = c.W, NB = c.NB, nb = c.nb, t0 = c.t0, H = c.H, rps = c.rps;

    int32_t t = st0.t, s = st0.s, r_in_step = st0.r_in_step, n_step = st0.n_step, s_slot = st0.s_slot;
    int32_t c_pos = st0.c_pos, room_b = st0.room_b;
    bool step_open = st0.step_open != 0, prev_active = st0.prev_active != 0;
    int64_t u_sum = st0.u_sum, u_tot = st0.u_tot;
    int64_t tot0 = st0.tot[0], tot2 = st0.tot[2], tot3 = st0.tot[3], tot4 = st0.tot[4], tot5 = st0.tot[5],
            tot6 = st0.tot[6];
    int32_t event = EV_BATCH;

    // lane j < W keeps worker j's load, log tail and block counts; lane b < nb route b's inputs
    int32_t rA = 0, rlive = 0, rused = 0, rN = 0;
    uint32_t rtail = 0;
    int32_t q_head = __builtin_amdgcn_readfirstlane(sh->qhead), q_size = __builtin_amdgcn_readfirstlane(sh->qsize);
    if (lane < W) {
        rA = s_A[lane];
        rN = s_N[lane];
        rtail = s_tail[lane];
        rlive = s_live[lane];
        rused = s_used[lane];
    }
    const unsigned long long stamped_mask = __ballot(lane < W && s_stamped[lane] != 0);
    const int32_t b_start = t - t0;
    int32_t rwork = b_start > 0 ? __builtin_amdgcn_readfirstlane(r_wend[b_start - 1]) : 0;
    int32_t vP = 0, vc = 0, vk = 0;
    if (lane < nb) {
        vP = r_P[lane];
        vc = r_c[lane];
        vk = r_k[lane];
    }
    if (lane >= b_start && lane < nb) {
        r_ep[lane] = 0u;
        r_reg[lane] = 0;
        r_evc[lane] = 0;
        r_evd[lane] = 0ull;
    }
    // the overlaps of the next route (all earlier routes' raises are in)
    int32_t oj = lane < W && b_start < nb ? o_cur[b_start * W + lane] : 0;
    for (;;) {
        if (!step_open) {
            // release the routes of step s - H (their loads, in registers); queue their
            // conversations' next turns
            const int32_t slot = s_slot, sb = slot * rps;
            if (s >= H) {
                const int32_t nprev = __builtin_amdgcn_readfirstlane(s_stepn[slot]);
                const int32_t qtail = q_head + q_size;
                int32_t pushed = 0;
                int64_t rel = 0;
                for (int32_t base = 0; base < nprev; base += 64) {
                    const int32_t r = base + lane;
                    int32_t wr = 0, pr = 0, cr = 0;
                    if (r < nprev) {
                        wr = s_stw[sb + r];
                        pr = s_stP[sb + r];
                        cr = s_stc[sb + r];
                    }
                    const bool more = r < nprev && (cr & kMoreTurns) != 0;
                    const unsigned long long mb = __ballot(more);
                    if (more) {
                        const int32_t qi = qtail + pushed + __popcll(mb & ((1ull << lane) - 1ull));
                        c.g_queue[qi >= c.qcap ? qi - c.qcap : qi] = cr & ~kMoreTurns;
                    }
                    pushed += __popcll(mb);
                    const int32_t m = min(64, nprev - base);
                    for (int32_t k = 0; k < m; ++k) {
                        const int32_t wk = __builtin_amdgcn_readlane(wr, k), pk = __builtin_amdgcn_readlane(pr, k);
                        rel += pk;
                        if (lane == wk) {
                            rA -= pk;
                            rN -= 1;
                        }
                    }
                }
                u_tot -= rel;
                q_size += pushed;
            }
            int32_t inflight = 0;
            for (int32_t k = 1; k < H && k <= s; ++k)
                inflight += __builtin_amdgcn_readfirstlane(s_stepn[s_slot >= k ? s_slot - k : s_slot - k + H]);
            if (q_size == 0 && inflight == 0) {
                event = EV_DONE;
                break;
            }
            n_step = min(rps, q_size);
            if (lane == 0) s_stepn[slot] = n_step;
            if (n_step > 0) tot5 = s + 1;
            r_in_step = 0;
            step_open = true;
        }
        if (r_in_step >= n_step) {
            ++s;
            s_slot = s_slot + 1 == H ? 0 : s_slot + 1;
            step_open = false;
            continue;
        }
        const int32_t b = t - t0;
        if (b >= nb) break;
        // one route: controller, cost of every worker, argmin
        const int32_t sb = s_slot * rps;
        bool active = false;
        if (LC && t >= c.ctrl_window) active = (int64_t)c.ctrl_den * u_sum > c.ctrl_thr;
        const float w = active ? fminf(c.w_ov, c.ctrl_w_ov) : c.w_ov;
        const int32_t P = __builtin_amdgcn_readlane(vP, b);
        const int64_t row = c.out_base + (int64_t)t;
        uint32_t bits = 0xFFFFFFFFu;
        if (lane < W) {
            const float cj = route_cost_ep(w, c.w_act, c.w_sat, c.cap_blocks, c.inv_cap, P, oj, rA);
            if (c.out_cost) c.out_cost[row * W + lane] = cj;
            bits = __float_as_uint(__fadd_rn(cj, 0.0f));
        }
        const uint32_t mn = ep_wave_min_u32(bits);
        const int32_t sg = __ffsll(__ballot(lane < W && bits == mn)) - 1;
        const int32_t osg = __builtin_amdgcn_readlane(oj, sg);
        const int32_t live_after = __builtin_amdgcn_readlane(rlive, sg) + P - osg;
        const uint32_t base = (uint32_t)__builtin_amdgcn_readlane((int)rtail, sg);
        const bool flush = live_after > c.cache;
        const bool stamped = ((stamped_mask >> sg) & 1ull) != 0;
        // a worker that keeps recency needs log records for the route's P touches and slots for
        // its new blocks: without room, stop before the route and compact that worker
        if (__builtin_expect(stamped, 0)) {
            const uint32_t head = __builtin_amdgcn_readfirstlane(s_head[sg]);
            const uint64_t add = (uint64_t)(P - osg);
            if ((uint64_t)(uint32_t)__builtin_amdgcn_readlane(rused, sg) + add > c.used_limit ||
                (uint64_t)(base - head) + (uint64_t)P > c.R || (uint64_t)base + (uint64_t)P > 0x40000000u) {
                if (room_b == t) {
                    if (lane == 0) atomicOr((int32_t*)c.status, RK_DEV_TABLE_FULL);
                } else {
                    room_b = t;
                    if (lane == 0) sh->ev_b = sg;
                    event = EV_ROOM;
                    break;
                }
            }
        }
        if (active) {
            tot3 += 1;
            if (!prev_active) tot4 += 1;
        }
        prev_active = active;
        const int32_t rc = __builtin_amdgcn_readlane(vc, b);
        if (lane == sg) {
            rA += P;
            rN += 1;
            rtail = base + (uint32_t)P;
            rlive = live_after;
            rused += P - osg;
        }
        rwork += stamped ? P : (osg < P ? run_entries(osg, P) : 0);
        // later requests of the batch now find this chain on sg; then the next route's overlaps
        const int32_t b2 = b + 1 + lane;
        if (b2 < nb) {
            const int32_t l = l_lcp[b * NB + b2];
            if (l > o_cur[b2 * W + sg]) o_cur[b2 * W + sg] = l;
        }
        oj = lane < W && b + 1 < nb ? o_cur[(b + 1) * W + lane] : 0;
        if (lane == 0) {
            r_sig[b] = sg;
            r_wend[b] = rwork;
            r_stamp[b] = base;
            r_otab[b] = o_tab[b * W + sg];
            s_stw[sb + r_in_step] = sg;
            s_stP[sb + r_in_step] = P;
            s_stc[sb + r_in_step] = rc;
            r_step[b] = s;
            c.g_hist[2 * t] = rc & ~kMoreTurns;
            c.g_hist[2 * t + 1] = P | (sg << 16);
            c.g_next[rc & ~kMoreTurns] = __builtin_amdgcn_readlane(vk, b) + 1;
            if (flush) {
                sh->ev_b = b;
                sh->ev_row = row;
            }
        }
        u_tot += P;
        q_head = q_head + 1 == c.qcap ? 0 : q_head + 1;
        q_size -= 1;
        if (LC) {
            const int32_t pos = c_pos;
            c_pos = c_pos + 1 == c.ctrl_window ? 0 : c_pos + 1;
            if (t >= c.ctrl_window) {
                const int64_t old = s_u[pos];
                u_sum -= (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int32_t)(old >> 32)) << 32) |
                                   (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)old));
            }
            if (lane == 0) s_u[pos] = u_tot;
            u_sum += u_tot;
        }
        tot0 += P - osg;
        tot2 += P;
        tot6 += osg;
        ++t;
        ++r_in_step;
        ep_wave_sync();
        if (lane == 0) __hip_atomic_store(&sh->decided, b + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (__builtin_expect(flush, 0)) {
            event = EV_FLUSH;
            break;
        }
    }
    if (lane < W) {
        s_A[lane] = rA;
        s_N[lane] = rN;
        s_tail[lane] = rtail;
        s_live[lane] = rlive;
        s_used[lane] = rused;
    }
    if (lane == 0) {
        sh->qhead = q_head;
        sh->qsize = q_size;
        sh->event = event;
        sh->tdone = t;
        __hip_atomic_store(&sh->stop, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
    st->t = t;
    st->s = s;
    st->r_in_step = r_in_step;
    st->n_step = n_step;
    st->s_slot = s_slot;
    st->c_pos = c_pos;
    st->room_b = room_b;
    st->step_open = step_open;
    st->prev_active = prev_active;
    st->u_sum = u_sum;
    st->u_tot = u_tot;
    st->tot[0] = tot0;
    st->tot[2] = tot2;
    st->tot[3] = tot3;
    st->tot[4] = tot4;
    st->tot[5] = tot5;
    st->tot[6] = tot6;
}

template <bool Queued>
__global__ __launch_bounds__(NT, 2) void episode_kernel(EpArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ EpShared sh;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    unsigned char* const ws = a.ws + (size_t)blockIdx.x * a.L.per_episode;
    for (int32_t it = 0;; ++it) {
    int32_t e = (int32_t)blockIdx.x;
    if constexpr (Queued) {
        if (tid == 0)
            sh.next_e = __hip_atomic_fetch_add((int32_t*)(a.ws + a.L.off_ctl), 1, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
        e = sh.next_e;
        __syncthreads();
        if (e >= a.E) break;
    } else if (it > 0) {
        break;
    }
    [&]() {
    const rk_episode_params prm = a.params[e];
    const int32_t W = a.W, NB = a.NB;
    const bool scan = a.probe_mode == RK_PROBE_SCAN;

    // per-worker state
    int32_t* s_A = (int32_t*)(smem + a.lds_w);
    uint32_t* s_head = (uint32_t*)(s_A + W);
    uint32_t* s_tail = s_head + W;
    int32_t* s_live = (int32_t*)(s_tail + W);
    int32_t* s_used = s_live + W;
    int32_t* s_N = s_used + W;                              // requests in flight per worker
    uint32_t* s_b1 = (uint32_t*)(s_N + W);                  // memory tiers: G1's boundary in the log,
    uint32_t* s_b2 = s_b1 + W;                              //   G1 u G2's boundary,
    int32_t* s_n1 = (int32_t*)(s_b2 + W);                   //   live records from each boundary on
    int32_t* s_n2 = s_n1 + W;
    int32_t* s_stamped = s_n2 + W;                          // recency kept (else insert-only until the first eviction)
    // in-flight routes of the last H steps, by step slot
    int32_t* s_stw = (int32_t*)(smem + a.lds_inflight);   // worker
    int32_t* s_stP = s_stw + a.max_inflight;               // prompt blocks
    int32_t* s_stc = s_stP + a.max_inflight;               // conversation (| kMoreTurns)
    int32_t* s_stepn = s_stc + a.max_inflight;             // routes per step slot
    int64_t* s_u = (int64_t*)(smem + a.lds_u);             // controller load samples
    int32_t* s_roff = (int32_t*)(smem + a.lds_roff);       // recency rebuild: first touch of each route
    // the batch
    const BatchLayout BL = batch_layout(NB, W, a.tiers != 0);
    unsigned char* bb = smem + a.lds_batch;
    int64_t* r_cb = (int64_t*)(bb + BL.rcb);               // chain base
    uint64_t* r_last = (uint64_t*)(bb + BL.rlast);         // h_{P-1}
    uint64_t* r_first = (uint64_t*)(bb + BL.rfirst);       // h_0
    int32_t* o_cur = (int32_t*)(bb + BL.o_cur);            // [b][j] overlap as of now
    int32_t* o_tab = (int32_t*)(bb + BL.o_tab);            // [b][j] overlap found in the table
    int32_t* r_c = (int32_t*)(bb + BL.rc);                 // conversation (| kMoreTurns)
    int32_t* r_k = (int32_t*)(bb + BL.rk);                 // turn of the conversation
    int32_t* r_turn = (int32_t*)(bb + BL.rturn);           // global turn index
    int32_t* r_P = (int32_t*)(bb + BL.rP);                 // prompt blocks
    int32_t* r_sig = (int32_t*)(bb + BL.rsig);             // chosen worker
    int32_t* r_otab = (int32_t*)(bb + BL.rotab);           // blocks known cached in sigma's table
    uint32_t* r_stamp = (uint32_t*)(bb + BL.rstamp);       // stamp of the last block
    uint32_t* r_ep = (uint32_t*)(bb + BL.rep);             // decay epoch (frequency eviction)
    int32_t* r_step = (int32_t*)(bb + BL.rstep);           // per-route outputs, written out at the end
    int32_t* r_reg = (int32_t*)(bb + BL.rreg);             //   of the batch: step, regime, evictions
    int32_t* r_evc = (int32_t*)(bb + BL.revc);             //   and their digest
    uint64_t* r_evd = (uint64_t*)(bb + BL.revd);
    uint32_t* r_rnd = (uint32_t*)(bb + BL.rrnd);           // the route's two random words
    uint16_t* l_lcp = (uint16_t*)(bb + BL.lcp);            // [b2][b], b2 < b: common prefix (a row per earlier route)
    uint16_t* nx_lcp = (uint16_t*)(bb + BL.lcp2);          //   the same for the next batch (the two swap)
    uint16_t* l_pval = (uint16_t*)(bb + BL.pval);          // common prefix of each listed pair
    uint16_t* l_items = (uint16_t*)(bb + BL.items);        // search items left after a first probe
    uint16_t* l_pairs = (uint16_t*)(bb + BL.pairs);        // batch pairs whose common prefix is searched
    int64_t* nx_cb = (int64_t*)(bb + BL.nxcb);             // the next batch, its overlaps computed while
    uint64_t* nx_first = (uint64_t*)(bb + BL.nxfirst);     //   this batch is decided: chain base, h_0, P
    int32_t* nx_P = (int32_t*)(bb + BL.nxP);
    int32_t* nx_o = (int32_t*)(bb + BL.nxo);               //   and [b][j] overlaps
    int32_t* r_wend = (int32_t*)(bb + BL.wend);            // writes of the batch's routes up to b, inclusive
    uint16_t* t1_tab = (uint16_t*)(bb + BL.t1);            // [b][j] leading blocks in G1 (tiers)
    uint16_t* t12_tab = (uint16_t*)(bb + BL.t12);          // [b][j] leading blocks in G1 u G2 (tiers)

    const int32_t H = prm.hold_steps, rps = prm.routes_per_step, n_conv = prm.n_conv;
    const bool bad = H < 1 || rps < 1 || rps > a.max_rps || (int64_t)H * rps > a.max_inflight ||
                     n_conv < 0 || n_conv > a.max_conv || prm.cap_blocks < 1 ||
                     (prm.controller == 1 && (prm.ctrl_window < 1 || prm.ctrl_window > a.max_ctrl_window ||
                                              prm.ctrl_den < 1 || prm.ctrl_num < 0));
    if (bad) {
        if (tid == 0) atomicOr(a.status, RK_DEV_TOO_LARGE);
        return;
    }
    const int32_t policy = prm.policy;
    const float tau = prm.tau;
    const bool regime_ctl = prm.controller == 2;
    const rk_regime_params& rg = a.regime;
    bool rg_ok = true, rg_draws = false;
    if (regime_ctl) {
        rg_ok = rg.alpha > 0.0 && rg.alpha <= 1.0 && rg.theta1 <= rg.theta2 && rg.eps >= 0.0 && rg.k >= 1 &&
                rg.beta >= 1 && rg.beta <= 8 && rg.n_sat >= 1;
        for (int r = 0; r < 3; ++r) {
            rg_ok = rg_ok && rg.tau[r] >= 0.0f && rg.w_ov[r] >= 0.0f;
            rg_draws = rg_draws || rg.tau[r] > 0.0f;
        }
    }
    const bool draws = rg_draws || (!regime_ctl && (policy == RK_POLICY_SOFTMAX || policy == RK_POLICY_RANDOM ||
                                                    policy == RK_POLICY_P2C));
    if (a.turn_off[prm.conv_begin + n_conv] - a.turn_off[prm.conv_begin] > (int64_t)a.max_routes) {
        if (tid == 0) atomicOr(a.status, RK_DEV_TOO_LARGE);
        return;
    }
    const bool freq = prm.evict_policy == RK_EVICT_FREQ;
    const int32_t dsteps = prm.decay_steps;
    const bool tiers = prm.tier_g1 > 0;
    const int32_t K1 = prm.tier_g1, K12 = prm.tier_g1 + prm.tier_g2;
    const bool tiers_ok = prm.tier_g1 >= 0 && prm.tier_g2 >= 0 && (int64_t)prm.tier_g1 + prm.tier_g2 <= a.cache &&
                          (!tiers || (a.tiers != 0 && !freq && prm.tier_w[0] >= 0.0f && prm.tier_w[1] >= 0.0f &&
                                      prm.tier_w[2] >= 0.0f));
    // negative or NaN weights would break the argmin on cost bits (unsigned order is float order only
    // for costs >= 0)
    const bool weights_ok = prm.w_ov >= 0.0f && prm.w_act >= 0.0f && prm.w_sat >= 0.0f && prm.ctrl_w_ov >= 0.0f;
    if (prm.controller < 0 || prm.controller > 2 || !rg_ok || !tiers_ok || !weights_ok ||
        (prm.evict_policy != RK_EVICT_LRU && !freq) || (freq && dsteps < 1) ||
        (!regime_ctl && (policy < RK_POLICY_ARGMIN || policy > RK_POLICY_P2C ||
                         (policy == RK_POLICY_SOFTMAX && !(tau > 0.0f)))) ||
        (draws && !a.route_rand)) {
        if (tid == 0) atomicOr(a.status, RK_DEV_BAD_PARAMS);
        return;
    }
    const int64_t gc0 = prm.conv_begin;
    const bool lean = !scan && policy == RK_POLICY_ARGMIN && prm.controller == 0 && !freq && !tiers;
    const bool lean_ctrl = !scan && policy == RK_POLICY_ARGMIN && prm.controller == 1 && !freq && !tiers;

    Slot* g_slots = (Slot*)(ws + a.L.off_slots);
    uint32_t* g_log = (uint32_t*)(ws + a.L.off_log);
    uint64_t* g_scratch = (uint64_t*)(ws + a.L.off_scratch);
    uint32_t* g_scratch_f = (uint32_t*)(ws + a.L.off_scratch_f);
    int32_t* g_queue = (int32_t*)(ws + a.L.off_queue);
    int32_t* g_next = (int32_t*)(ws + a.L.off_next);
    int32_t* g_hist = (int32_t*)(ws + a.L.off_hist);       // per route: conversation, P | worker << 16
    RunSlot* g_runs = (RunSlot*)(ws + a.L.off_runs);       // run index of the workers without recency
    const uint64_t S = a.L.slots, smask = S - 1, R = a.L.ring, rmask = R - 1, rsmask = a.L.runs - 1;
    const uint64_t used_limit = S - S / 4;
    const uint64_t scratch_cap = (uint64_t)a.cache + (uint64_t)a.max_blocks;

    // ---- initial state: empty caches, idle workers, every first turn queued.  The run index is
    //      cleared here; a worker's block table when the worker starts keeping recency (here for
    //      episodes that keep it from the start, at its first eviction for the others).
    const bool eager = freq || tiers || scan;
    auto clear_tables = [&](int32_t j_lo, int32_t j_hi) {
        uint4* z = reinterpret_cast<uint4*>(g_slots + (uint64_t)j_lo * S);
        const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
        const uint64_t n16 = (uint64_t)(j_hi - j_lo) * S;
        for (uint64_t k = tid; k < n16; k += NT) z[k] = zero;
    };
    {
        uint4* z = reinterpret_cast<uint4*>(g_runs);
        const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
        for (uint64_t k = tid; k <= rsmask; k += NT) z[k] = zero;
        if (eager) clear_tables(0, W);
    }
    if (tid < W) {
        s_A[tid] = 0;
        s_N[tid] = 0;
        s_b1[tid] = 0;
        s_b2[tid] = 0;
        s_n1[tid] = 0;
        s_n2[tid] = 0;
        s_stamped[tid] = eager;     // frequencies, tier runs and scans of any cached sets need every touch
        s_head[tid] = 0;
        s_tail[tid] = 0;
        s_live[tid] = 0;
        s_used[tid] = 0;
    }
    for (int32_t i = tid; i < a.max_inflight; i += NT) s_stepn[i] = 0;
    int32_t qn = 0;
    int32_t turns2 = 0;   // some conversation of the episode has a second turn
    for (int32_t base = 0; base < n_conv; base += NT) {
        const int32_t c = base + tid;
        bool has = false;
        if (c < n_conv) {
            g_next[c] = 0;
            has = a.turn_off[gc0 + c + 1] > a.turn_off[gc0 + c];
            turns2 |= a.turn_off[gc0 + c + 1] - a.turn_off[gc0 + c] > 1 ? 1 : 0;
        }
        int32_t total;
        const int32_t rank = block_scan(has, sh.wtot, total);
        if (has) g_queue[qn + rank] = c;
        qn += total;
    }
    const bool multi_turn = __syncthreads_or(turns2) != 0;
    if (tid == 0) {
        sh.qhead = 0;
        sh.qsize = qn;
        sh.ins = 0;
        sh.h1 = 0;
        sh.h2 = 0;
        sh.ev_total = 0;
        sh.tdone = 0;
    }
    __syncthreads();
    const int32_t qcap = n_conv + 1;

    // ---- compaction of worker j: re-stamp its live records in order into a cleared table (all threads)
    auto rebuild = [&](int32_t j) {
        Slot* tk = g_slots + (uint64_t)j * S;
        uint32_t* tl = g_log + (uint64_t)j * R;
        const uint32_t head = s_head[j], tail = s_tail[j];
        int32_t cnt = 0;
        for (uint32_t base = head; base < tail; base += NT) {
            const uint32_t pos = base + (uint32_t)tid;
            bool live = false;
            uint64_t key = 0;
            uint32_t fk = 0;
            if (pos < tail) {
                const uint32_t sl = tl[pos & rmask];
                if (sl < S) {
                    uint32_t st;
                    load_slot(tk + sl, key, st, fk);
                    live = st == pos;
                }
            }
            int32_t total;
            const int32_t rank = block_scan(live, sh.wtot, total);
            if (live && (uint64_t)(cnt + rank) < scratch_cap) {
                g_scratch[cnt + rank] = key;
                g_scratch_f[cnt + rank] = fk;
            }
            cnt += total;
        }
        if ((uint64_t)cnt > scratch_cap) {
            if (tid == 0) atomicOr(a.status, RK_DEV_TABLE_FULL);
            cnt = (int32_t)scratch_cap;
        }
        __syncthreads();
        {
            uint4* z = reinterpret_cast<uint4*>(tk);
            const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
            for (uint64_t i = tid; i < S; i += NT) z[i] = zero;
        }
        __syncthreads();
        for (int32_t q = tid; q < cnt; q += NT) {
            int ins;
            const uint64_t sl = insert_or_touch(tk, smask, g_scratch[q], ins, a.status);
            if (sl != ~0ull) {
                tk[sl].stamp = (uint32_t)q;
                tk[sl].fkey = g_scratch_f[q];
            }
            tl[(uint32_t)q & rmask] = (uint32_t)sl;
        }
        __syncthreads();
        if (tid == 0) {
            s_head[j] = 0;
            s_tail[j] = (uint32_t)cnt;
            s_live[j] = cnt;
            s_used[j] = cnt;
            // the live records keep their order: a tier's run is now the last n of them
            s_n1[j] = min(s_n1[j], cnt);
            s_n2[j] = min(s_n2[j], cnt);
            s_b1[j] = (uint32_t)(cnt - s_n1[j]);
            s_b2[j] = (uint32_t)(cnt - s_n2[j]);
        }
        __syncthreads();
    };

    // ---- waves 1-3 while wavefront 0 decides (and wavefront 0 once it stops): claim the next
    //      128 writes of the decided routes (sh.claimed counts writes, r_wend numbers them; a
    //      compare-and-swap) and apply them with the wave's 64 lanes, two each; stop once
    //      wavefront 0 has stopped and every decided write is claimed.  sh.decided and
    //      sh.claimed only grow until the workgroup synchronizes.
    auto writer = [&]() {
        int my_ins = 0, my_h1 = 0, my_h2 = 0;
        for (;;) {
            const int32_t c = __builtin_amdgcn_readfirstlane(
                __hip_atomic_load(&sh.claimed, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP));
            const int32_t d = __builtin_amdgcn_readfirstlane(
                __hip_atomic_load(&sh.decided, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP));
            const int32_t wd = d > 0 ? __builtin_amdgcn_readfirstlane(r_wend[d - 1]) : 0;
            if (c < wd) {
                // work items [c, hi): the decided routes' writes numbered in order, route b's
                // [r_wend[b - 1], r_wend[b]).  A route on a worker that keeps no recency yet adds
                // the entries of one run to the run index (the blocks past its decided overlap,
                // which counts the common prefixes with the batch's earlier routes on that
                // worker); a route on a worker that keeps recency touches all of its blocks.
                const int32_t hi = min(wd, c + 128);
                int32_t won = 0;
                if (lane == 0) {
                    int32_t expect = c;
                    won = __hip_atomic_compare_exchange_strong(&sh.claimed, &expect, hi, __ATOMIC_ACQ_REL,
                                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                }
                if (!__builtin_amdgcn_readfirstlane(won)) continue;
                int32_t b0 = 0, bh = d - 1;    // the route of item c
                while (b0 < bh) {
                    const int32_t mid = (b0 + bh) >> 1;
                    if (r_wend[mid] > c) bh = mid;
                    else b0 = mid + 1;
                }
                // two items per lane, their chain hashes, claims and group loads in flight together
                int32_t bq[2], kq[2], sgq[2], stq[2];
                bool v[2], lazy[2];
                int64_t hoff[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const int32_t w = c + lane + 64 * u;
                    v[u] = w < hi;
                    int32_t b = b0;
                    while (v[u] && r_wend[b] <= w) ++b;
                    bq[u] = b;
                    kq[u] = w - (b > 0 ? r_wend[b - 1] : 0);
                    sgq[u] = v[u] ? r_sig[b] : 0;
                    lazy[u] = v[u] && !s_stamped[sgq[u]];
                    stq[u] = lazy[u] ? o_cur[b * W + sgq[u]] : 0;
                    const int32_t pos = lazy[u] ? run_entry_pos(stq[u], kq[u]) : kq[u];
                    hoff[u] = v[u] ? r_cb[b] + pos : 0;
                }
                uint64_t h[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) h[u] = a.chains[hoff[u]];
                Slot* tk[2];
                bool hint[2], act[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    if (lazy[u])
                        run_insert(g_runs, rsmask, h[u], sgq[u], run_val(r_cb[bq[u]], sgq[u], r_P[bq[u]]),
                                   a.status);
                    tk[u] = g_slots + (uint64_t)sgq[u] * S;
                    act[u] = v[u] && !lazy[u];
                    hint[u] = kq[u] < r_otab[bq[u]];
                }
                if (__ballot(act[0] || act[1]) == 0ull) continue;
                uint64_t sl[2];
                int ins[2];
                touch_hinted2(tk, smask, h, hint, act, sl, ins, a.status);
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    if (!act[u]) continue;
                    const int32_t b = bq[u], sg = sgq[u];
                    const uint32_t stamp = r_stamp[b] + (uint32_t)(r_P[b] - 1 - kq[u]);
                    // routes of one worker that share a block touch it concurrently: the latest stamp wins
                    if (sl[u] != ~0ull) {
                        const uint32_t old = __hip_atomic_fetch_max(&tk[u][sl[u]].stamp, stamp, __ATOMIC_RELAXED,
                                                                    __HIP_MEMORY_SCOPE_WORKGROUP);
                        if (freq) freq_touch(&tk[u][sl[u]].fkey, ins[u] != 0, r_ep[b]);
                        if (tiers && !ins[u]) {       // a hit whose old record lay in a tier's run
                            my_h1 += old >= s_b1[sg];
                            my_h2 += old >= s_b2[sg];
                        }
                    }
                    g_log[(uint64_t)sg * R + (stamp & rmask)] = (uint32_t)sl[u];   // a failed insert logs an out-of-range slot
                    my_ins += ins[u];
                }
                continue;
            }
            if (__builtin_amdgcn_readfirstlane(
                    __hip_atomic_load(&sh.stop, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP))) {
                const int32_t c2 = __builtin_amdgcn_readfirstlane(
                    __hip_atomic_load(&sh.claimed, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP));
                const int32_t d2 = __builtin_amdgcn_readfirstlane(
                    __hip_atomic_load(&sh.decided, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP));
                const int32_t wd2 = d2 > 0 ? __builtin_amdgcn_readfirstlane(r_wend[d2 - 1]) : 0;
                if (c2 >= wd2) break;
                continue;
            }
            __builtin_amdgcn_s_sleep(2);
        }
        if (my_ins) atomicAdd(&sh.ins, my_ins);
        if (my_h1) atomicAdd(&sh.h1, my_h1);
        if (my_h2) atomicAdd(&sh.h2, my_h2);
    };

    // ---- memory tiers: move worker j's boundary bk forward until the run from it holds at most K
    //      live records (all threads)
    auto advance = [&](uint32_t* bk, int32_t* nk, int32_t K, int32_t j) {
        const Slot* tk = g_slots + (uint64_t)j * S;
        const uint32_t* tl = g_log + (uint64_t)j * R;
        uint32_t b = bk[j];
        int32_t n = nk[j];
        const uint32_t tail = s_tail[j];
        while (n > K) {
            if (b >= tail) {
                if (tid == 0) atomicOr(a.status, RK_DEV_TABLE_FULL);
                n = K;
                break;
            }
            const uint32_t pos = b + (uint32_t)tid;
            bool live = false;
            if (pos < tail) {
                const uint32_t sl = tl[pos & rmask];
                if (sl < S) {
                    uint64_t key;
                    uint32_t st;
                    load_slot(tk + sl, key, st);
                    live = st == pos;
                }
            }
            int32_t total;
            const int32_t rank = block_scan(live, sh.wtot, total);
            const int32_t need = n - K;
            if (total >= need) {
                if (live && rank == need - 1) sh.adv = pos + 1;
                __syncthreads();
                b = sh.adv;
                n = K;
            } else {
                n -= total;
                b = min(b + (uint32_t)NT, tail);
            }
        }
        __syncthreads();
        if (tid == 0) {
            bk[j] = b;
            nk[j] = n;
        }
        __syncthreads();
    };

    // ---- recency of worker j rebuilt from the episode's routes [0, t_end) (all threads): pass 1
    //      gives every block the stamp of its last touch (routes in order, a route's blocks from last
    //      to first, stamps counting up from 0), pass 2 keeps the touch that set each block's stamp
    //      and lays the live records down in the log in that order, re-stamped 0, 1, ...
    auto replay = [&](int32_t j, int32_t t_end) {
        Slot* tk = g_slots + (uint64_t)j * S;
        uint32_t* tl = g_log + (uint64_t)j * R;
        int64_t* r_cbs = (int64_t*)(ws + a.L.off_replay);     // per chunk of routes, the worker's: chain
        int32_t* r_off = s_roff;                              // base (global), first touch index (LDS)
                                                              // and P (global)
        int32_t* r_Ps = (int32_t*)(r_cbs + NT) + NT;
        for (int pass = 0; pass < 2; ++pass) {
            int64_t stamp0 = 0;      // original stamp of the chunk's first touch
            int32_t live = 0;        // pass 2: live records laid down so far
            for (int32_t base = 0; base < t_end; base += NT) {
                const int32_t r = base + tid;
                int32_t P = 0;
                int64_t cb = 0;
                if (r < t_end) {
                    const int32_t pw = g_hist[2 * r + 1];
                    if ((pw >> 16) == j) {
                        P = pw & 0xFFFF;
                        cb = a.chain_off[gc0 + g_hist[2 * r]];
                    }
                }
                int32_t n_r, ptot;
                const int32_t rank = block_scan(P > 0, sh.wtot, n_r);
                const int32_t off = block_excl_sum(P, sh.wtot, ptot);
                if (P > 0) {
                    r_off[rank] = off;
                    r_cbs[rank] = cb;
                    r_Ps[rank] = P;
                }
                __syncthreads();
                // kRU touches per thread at a time, their memory operations issued together
                for (int32_t i0 = 0; i0 < ptot; i0 += NT * kRU) {
                    uint64_t h[kRU], sl[kRU];
                    uint32_t st[kRU];
                    bool last[kRU];
#pragma unroll
                    for (int u = 0; u < kRU; ++u) {
                        const int32_t i = i0 + u * NT + tid;
                        h[u] = kEmpty;
                        st[u] = 0;
                        sl[u] = ~0ull;
                        last[u] = false;
                        if (i < ptot) {
                            int32_t lo = 0, hi = n_r - 1;     // the route holding touch i
                            while (lo < hi) {
                                const int32_t mid = (lo + hi + 1) >> 1;
                                if (r_off[mid] <= i) lo = mid;
                                else hi = mid - 1;
                            }
                            const int32_t q = i - r_off[lo];            // touches go from the last block
                            const int32_t k = r_Ps[lo] - 1 - q;         // to the first
                            st[u] = (uint32_t)(stamp0 + r_off[lo] + q);
                            h[u] = a.chains[r_cbs[lo] + k];
                        }
                    }
                    if (pass == 0) {
                        // every block into the table (it starts empty), the latest touch's stamp kept
                        touch_batch(tk, smask, h, sl, a.status);
#pragma unroll
                        for (int u = 0; u < kRU; ++u)
                            if (sl[u] != ~0ull)
                                __hip_atomic_fetch_max(&tk[sl[u]].stamp, st[u], __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_WORKGROUP);
                    } else {
                        find_batch(tk, smask, h, sl, st, last);
                        // every thread has read its slots' stamps before any is rewritten; the
                        // live records keep the order of their touches
#pragma unroll
                        for (int u = 0; u < kRU; ++u) {
                            int32_t nl;
                            const int32_t lr = block_scan(last[u], sh.wtot, nl);
                            if (last[u]) {
                                const uint32_t ns = (uint32_t)(live + lr);
                                tk[sl[u]].stamp = ns;
                                tl[ns & rmask] = (uint32_t)sl[u];
                            }
                            live += nl;
                        }
                    }
                }
                stamp0 += ptot;
                __syncthreads();
            }
            __syncthreads();
            if (pass == 1 && tid == 0) {
                if (live != s_live[j]) atomicOr(a.status, RK_DEV_TABLE_FULL);
                s_head[j] = 0;
                s_tail[j] = (uint32_t)live;
                s_stamped[j] = 1;
            }
            if (pass == 0 && stamp0 >= 0x40000000ll) {
                if (tid == 0) atomicOr(a.status, RK_DEV_TOO_LARGE);
            }
        }
        __syncthreads();
    };

    // ---- recency of worker j rebuilt in one pass when the touches of its routes [0, t_end) fit the
    //      log (all threads; false, with nothing written, when they do not).  The touches keep
    //      their stamps (route after route, a route's blocks from last to first, counting up from
    //      0), so every touch has its own log position: each touch that may be a block's latest
    //      writes its record there and raises the block's stamp to its own, and a record is live
    //      iff the block's stamp is its position, as in the eager upkeep.  The log positions of
    //      all touches are cleared first.  Routes go newest first, so a touch that finds its
    //      block already stamped by a later touch does nothing more.  Every turn of a
    //      conversation reads the leading blocks of the conversation's one chain, so the first
    //      D blocks of a route are touched again by any later route of its conversation on j
    //      with D blocks: those touches are skipped outright (their log positions stay clear,
    //      as a record that is not live), and only the route's last P - min(P, D) blocks are
    //      looked up, D the most blocks of such a route in the chunks done before (any D up to
    //      the most blocks of a later route gives the same result; the skips need none).
    auto materialize = [&](int32_t j, int32_t t_end) -> bool {
        Slot* tk = g_slots + (uint64_t)j * S;
        uint32_t* tl = g_log + (uint64_t)j * R;
        int64_t* r_cbs = (int64_t*)(ws + a.L.off_replay);     // per chunk, the routes on j: chain base,
        int32_t* r_sb = (int32_t*)(r_cbs + NT);               //   stamp of the route's last block within
        int32_t* r_Ps = r_sb + NT;                            //   the chunk, P (global) and the first of
        int32_t* r_off = s_roff;                              //   its looked-up touches (LDS)
        int32_t* m_P = (int32_t*)(ws + a.L.off_later);        // per conversation: most blocks of a route
        if (multi_turn)                                       //   on j in the chunks done so far
            for (int32_t c = tid; c < n_conv; c += NT) m_P[c] = 0;
        auto route_of = [&](int32_t r, int32_t& P, int64_t& cb, int32_t& cv) {
            P = 0;
            cb = 0;
            cv = 0;
            if (r < t_end) {
                const int32_t pw = g_hist[2 * r + 1];
                if ((pw >> 16) == j) {
                    P = pw & 0xFFFF;
                    cv = g_hist[2 * r];
                    cb = a.chain_off[gc0 + cv];
                }
            }
        };
        int64_t T = 0;     // touches of the worker's routes
        for (int32_t base = 0; base < t_end; base += NT) {
            int32_t P, cv;
            int64_t cb;
            route_of(base + tid, P, cb, cv);
            int32_t ptot;
            block_excl_sum(P, sh.wtot, ptot);
            T += ptot;
        }
        if (T > (int64_t)R) return false;
        for (int64_t p = tid; p < T; p += NT) tl[p] = 0xFFFFFFFFu;
        __syncthreads();
        int64_t end = T;   // stamp after the last touch of the chunks done so far
        const int32_t nchunk = (t_end + NT - 1) / NT;
        for (int32_t c = nchunk - 1; c >= 0; --c) {
            int32_t P, cv;
            int64_t cb;
            route_of(c * NT + tid, P, cb, cv);
            int32_t n_r, ptot, ltot;
            const int32_t rank = block_scan(P > 0, sh.wtot, n_r);
            const int32_t D = multi_turn && P > 0 ? m_P[cv] : 0;   // blocks touched again later
            const int32_t off = block_excl_sum(P, sh.wtot, ptot);
            int32_t loff = off;
            ltot = ptot;
            if (multi_turn) loff = block_excl_sum(P - min(P, D), sh.wtot, ltot);
            if (P > 0) {
                r_off[rank] = loff;
                r_cbs[rank] = cb;
                r_sb[rank] = off;
                r_Ps[rank] = P;
            }
            __syncthreads();
            const int64_t stamp0 = end - ptot;
            // kRU looked-up touches per thread, each step's memory operations issued for all of
            // them before any result is used (addresses by masks: an empty touch reads chain hash
            // 0 and the table's first group).  A route's looked-up touches are its last blocks, so
            // the q-th of them is the route's q-th touch.
            for (int32_t i0 = 0; i0 < ltot; i0 += NT * kRU) {
                uint64_t h[kRU], k[kRU][kWin];
                uint32_t st[kRU], stv[kRU][kWin];
                int64_t hoff[kRU];
                bool v[kRU];
#pragma unroll
                for (int u = 0; u < kRU; ++u) {
                    const int32_t i = ltot - 1 - (i0 + u * NT + tid);    // the chunk's newest touches first
                    v[u] = i >= 0;
                    const int32_t ii = v[u] ? i : 0;
                    int32_t lo = 0, hi = n_r - 1;     // the route holding touch ii (the last of equal
                    while (lo < hi) {                 // offsets: a route with none shares the next's)
                        const int32_t mid = (lo + hi + 1) >> 1;
                        if (r_off[mid] <= ii) lo = mid;
                        else hi = mid - 1;
                    }
                    const int32_t q = ii - r_off[lo];            // touches go from the last block
                    const int32_t kb = r_Ps[lo] - 1 - q;         // to the first
                    st[u] = (uint32_t)(stamp0 + r_sb[lo] + q);
                    hoff[u] = (-(int64_t)v[u]) & (r_cbs[lo] + kb);
                }
#pragma unroll
                for (int u = 0; u < kRU; ++u) h[u] = a.chains[hoff[u]];
#pragma unroll
                for (int u = 0; u < kRU; ++u) {
                    const Slot* g = tk + ((uint64_t)(-(int64_t)v[u]) & home_slot(h[u], smask));
                    load_slot(g + group_slot(h[u], 0), k[u][0], stv[u][0]);
                }
#pragma unroll
                for (int u = 0; u < kRU; ++u) {
                    const bool more = v[u] && k[u][0] != h[u] && k[u][0] != kEmpty;
#pragma unroll
                    for (int r = 1; r < kWin; ++r) {
                        k[u][r] = kEmpty;
                        stv[u][r] = 0;
                    }
                    if (more) {
                        const Slot* g = tk + home_slot(h[u], smask);
#pragma unroll
                        for (int r = 1; r < kWin; ++r) load_slot(g + group_slot(h[u], r), k[u][r], stv[u][r]);
                    }
                }
                // the key's slot in its first group, or the first empty slot there to claim
                uint64_t sl[kRU], prev[kRU];
                int32_t claim[kRU];
#pragma unroll
                for (int u = 0; u < kRU; ++u) {
                    const uint64_t s0 = home_slot(h[u], smask);
                    sl[u] = ~0ull;
                    claim[u] = -1;
                    bool later = false, stop = false;
#pragma unroll
                    for (int r = 0; r < kWin; ++r) {
                        if (!stop) {
                            if (k[u][r] == h[u]) {
                                sl[u] = s0 + group_slot(h[u], r);
                                later = stv[u][r] > st[u];
                                stop = true;
                            } else if (k[u][r] == kEmpty) {
                                claim[u] = r;
                                stop = true;
                            }
                        }
                    }
                    if (!v[u] || later) {         // a later touch of the block was stamped already
                        sl[u] = ~0ull;
                        claim[u] = -2;
                    }
                    prev[u] = kEmpty;
                }
                // the claims return the slots' previous keys; nothing reads them before all are issued
#pragma unroll
                for (int u = 0; u < kRU; ++u) {
                    if (claim[u] >= 0) {
                        const uint64_t si = home_slot(h[u], smask) + group_slot(h[u], claim[u]);
                        prev[u] = atomicCAS(reinterpret_cast<unsigned long long*>(&tk[si].key), kEmpty, h[u]);
                    }
                }
#pragma unroll
                for (int u = 0; u < kRU; ++u) {
                    if (claim[u] >= 0) {
                        if (prev[u] == kEmpty || prev[u] == h[u])
                            sl[u] = home_slot(h[u], smask) + group_slot(h[u], claim[u]);
                    }
                    if (claim[u] != -2 && sl[u] == ~0ull) {    // a full first group or a lost claim
                        int ins;
                        sl[u] = insert_or_touch(tk, smask, h[u], ins, a.status);
                    }
                }
#pragma unroll
                for (int u = 0; u < kRU; ++u) {
                    if (sl[u] == ~0ull) continue;
                    __hip_atomic_fetch_max(&tk[sl[u]].stamp, st[u], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                    tl[st[u] & rmask] = (uint32_t)sl[u];
                }
            }
            if (multi_turn && P > 0) atomicMax(&m_P[cv], P);     // later routes for the chunks before
            end = stamp0;
            __syncthreads();
        }
        if (tid == 0) {
            s_head[j] = 0;
            s_tail[j] = (uint32_t)T;
            s_stamped[j] = 1;
        }
        __syncthreads();
        return true;
    };

    // ---- evict blocks of worker sg down to the capacity (all threads): live log records in log
    //      (recency) order, under frequency eviction only those at frequency 1 in epoch ep; the
    //      head moves to the first record left live
    auto evict = [&](int32_t sg, uint32_t ep) {
        Slot* tk = g_slots + (uint64_t)sg * S;
        uint32_t* tl = g_log + (uint64_t)sg * R;
        uint32_t head = s_head[sg];
        while (sh.remaining > 0) {
            const uint32_t tail = s_tail[sg];
            const int32_t rem = sh.remaining;
            if (head >= tail) {
                __syncthreads();
                if (tid == 0) {
                    atomicOr(a.status, RK_DEV_TABLE_FULL);
                    s_head[sg] = min(sh.first_kept, tail);
                    sh.remaining = 0;
                }
                __syncthreads();
                break;
            }
            const uint32_t pos = head + (uint32_t)tid;
            uint32_t sl = 0;
            bool live = false, cand = false;
            uint64_t key = 0;
            if (pos < tail) {
                sl = tl[pos & rmask];
                if (sl < S) {
                    uint32_t st, fk;
                    load_slot(tk + sl, key, st, fk);
                    live = st == pos;
                    cand = live && (!freq || fk <= ep + 1u);
                }
            }
            int32_t total;
            const int32_t rank = block_scan(cand, sh.wtot, total);
            const bool gone = cand && rank < rem;
            if (gone) {
                tk[sl].stamp = kTomb;
                atomicAdd(&sh.digest, (unsigned long long)mix64(key));
                if (rank == rem - 1) sh.new_head = pos + 1;
            }
            if (live && !gone) atomicMin(&sh.first_kept, pos);
            __syncthreads();
            if (tid == 0) {
                if (total >= rem) {
                    s_head[sg] = min(sh.first_kept, sh.new_head);
                    sh.ev += rem;
                    s_live[sg] -= rem;
                    sh.remaining = 0;
                } else {
                    sh.ev += total;
                    s_live[sg] -= total;
                    sh.remaining = rem - total;
                }
            }
            head = min(head + (uint32_t)NT, tail);
            __syncthreads();
        }
    };

    // overlaps of batch routes b in [b_lo, nb) on worker j (j < 0: every worker), into o_tab and o_cur
    auto search = [&](int32_t b_lo, int32_t nb, int32_t j) {
        if (!scan) {
            const int32_t per = j < 0 ? W : 1;
            const int32_t n = (nb - b_lo) * per;
            auto put = [&](int32_t i, int32_t o) {
                const int32_t b = b_lo + i / per;
                const int32_t jj = j < 0 ? i % per : j;
                o_tab[b * W + jj] = o;
                o_cur[b * W + jj] = o;
            };
            // workers that keep recency: binary search in their block tables; the others: the
            // run walk
            const unsigned long long st = __ballot(lane < W && s_stamped[lane] != 0 && (j < 0 || lane == j));
            const unsigned long long lz = __ballot(lane < W && s_stamped[lane] == 0 && (j < 0 || lane == j));
            if (st)
                prefix_searches(
                    n,
                    [&](int32_t i, const uint64_t*& ch, int32_t& P, int32_t& jj, uint64_t& h0) {
                        const int32_t b = b_lo + i / per;
                        jj = j < 0 ? i % per : j;
                        ch = a.chains + r_cb[b];
                        P = r_P[b];
                        h0 = r_first[b];
                        return s_stamped[jj] != 0;
                    },
                    put, g_slots, S, a.chains, l_items, &sh.nlist);
            if (lz)
                run_searches(
                    n,
                    [&](int32_t i, const uint64_t*& ch, int32_t& P, int32_t& jj, uint64_t& h0) {
                        const int32_t b = b_lo + i / per;
                        jj = j < 0 ? i % per : j;
                        ch = a.chains + r_cb[b];
                        P = r_P[b];
                        h0 = r_first[b];
                        return s_stamped[jj] == 0;
                    },
                    put, g_runs, rsmask, a.chains, l_items, &sh.nlist);
        } else {
            for (int32_t b = b_lo + wave; b < nb; b += NW) {
                const uint64_t* ch = a.chains + r_cb[b];
                if (j < 0) {
                    for (int32_t jb = 0; jb < W; jb += 4)
                        wave_overlaps<4>(ch, r_P[b], jb, 1, min(W, jb + 4), g_slots, S, RK_PROBE_SCAN, o_tab + b * W,
                                         -1, 0);
                } else {
                    wave_overlaps<1>(ch, r_P[b], j, 1, j + 1, g_slots, S, RK_PROBE_SCAN, o_tab + b * W, -1, 0);
                }
            }
            __syncthreads();
            const int32_t per = j < 0 ? W : 1;
            for (int32_t i = tid; i < (nb - b_lo) * per; i += NT) {
                const int32_t b = b_lo + i / per;
                const int32_t jj = j < 0 ? i % per : j;
                o_cur[b * W + jj] = o_tab[b * W + jj];
            }
        }
        __syncthreads();
    };

    // overlaps of batch routes b in [b_lo, nb) on worker j after j evicted (prefix mode): the
    // caches stay prefix-closed, so an eviction can only cut a suffix off a route's cached prefix,
    // and with every decided route's writes in, the table holds exactly o_cur[b][j] leading blocks
    // before it.  One lookup of the last of them decides the usual case; otherwise a binary search
    // within it finds the first block no longer live.
    auto research = [&](int32_t b_lo, int32_t nb, int32_t j) {
        const Slot* tj = g_slots + (uint64_t)j * S;
        for (int32_t b = b_lo + tid; b < nb; b += NT) {
            int32_t hi = o_cur[b * W + j];
            if (hi > 0) {
                const uint64_t* ch = a.chains + r_cb[b];
                auto live = [&](int32_t k) {
                    const uint64_t h = ch[k];
                    const uint64_t s0 = home_slot(h, smask);
                    uint64_t kw[kWin];
                    uint32_t sw[kWin];
#pragma unroll
                    for (int x = 0; x < kWin; ++x) load_slot(tj + s0 + group_slot(h, x), kw[x], sw[x]);
                    return finish_lookup(tj, smask, h, s0, kw, sw);
                };
                if (!live(hi - 1)) {
                    int32_t lo = 0;
                    --hi;
                    while (lo < hi) {
                        const int32_t mid = (lo + hi) >> 1;
                        if (live(mid)) lo = mid + 1;
                        else hi = mid;
                    }
                    hi = lo;
                }
            }
            o_tab[b * W + j] = hi;
            o_cur[b * W + j] = hi;
        }
        __syncthreads();
    };

    // tier overlaps of batch routes b in [b_lo, nb) on worker j (j < 0: every worker): o12 within
    // the cached prefix o_tab, then o1 within o12
    auto tier_search = [&](int32_t b_lo, int32_t nb, int32_t j) {
        const int32_t per = j < 0 ? W : 1;
        const int32_t n = (nb - b_lo) * per;
        tier_searches(
            n, !scan,
            [&](int32_t i, const uint64_t*& ch, int32_t& hi, int32_t& jj, uint32_t& bound) {
                const int32_t b = b_lo + i / per;
                jj = j < 0 ? i % per : j;
                ch = a.chains + r_cb[b];
                hi = o_tab[b * W + jj];
                bound = s_b2[jj];
            },
            [&](int32_t i, int32_t v) {
                const int32_t b = b_lo + i / per;
                t12_tab[b * W + (j < 0 ? i % per : j)] = (uint16_t)v;
            },
            g_slots, S);
        __syncthreads();
        tier_searches(
            n, !scan,
            [&](int32_t i, const uint64_t*& ch, int32_t& hi, int32_t& jj, uint32_t& bound) {
                const int32_t b = b_lo + i / per;
                jj = j < 0 ? i % per : j;
                ch = a.chains + r_cb[b];
                hi = t12_tab[b * W + jj];
                bound = s_b1[jj];
            },
            [&](int32_t i, int32_t v) {
                const int32_t b = b_lo + i / per;
                t1_tab[b * W + (j < 0 ? i % per : j)] = (uint16_t)v;
            },
            g_slots, S);
        __syncthreads();
    };

    // state of the routing sequence, kept by wavefront 0
    int32_t t = 0, s = 0, r_in_step = 0, n_step = 0;
    int32_t s_slot = 0;                            // s % H
    int32_t c_pos = 0;                             // t % ctrl_window (load controller)
    int32_t room_b = -1;                           // route last stopped for a compaction
    const float inv_cap = (prm.cap_blocks & (prm.cap_blocks - 1)) == 0 ? 1.0f / (float)prm.cap_blocks : 0.0f;
    bool step_open = false, prev_active = false;
    int64_t tot[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    int64_t u_sum = 0, u_tot = 0;
    double rg_ewma = 0.0;                          // regime controller: smoothed latency, regime,
    int32_t rg_r = 0, rg_up = 0, rg_down = 0;      // hysteresis counters

    // Longest common prefix of npair pairs of chains (all threads): pair(q, ca, cb, m, b1, b2)
    // names pair q's chain bases, the lesser length and two indices for store(q, b1, b2, lcp).
    // Pairs whose first blocks differ (or that have at most one block in common) are stored at
    // once; the others are listed and searched KP at a time per thread, each group in the depth
    // of one binary search on equal hashes.  npair <= NB * NB.
    auto pair_lcps = [&](int32_t npair, const auto& pair, const auto& store) {
        if (tid == 0) sh.nlist = 0;
        __syncthreads();
        for (int32_t q0 = 0; q0 < npair; q0 += NT) {
            const int32_t q = q0 + tid;
            bool srch = false;
            if (q < npair) {
                int64_t ca, cc;
                int32_t m, b1, b2;
                const bool same = pair(q, ca, cc, m, b1, b2);
                srch = same && m > 1;
                if (!srch) store(q, b1, b2, same && m > 0 ? 1 : 0);
            }
            const unsigned long long mb = __ballot(srch);
            int32_t wb = 0;
            if (lane == 0 && mb) wb = atomicAdd(&sh.nlist, (int32_t)__popcll(mb));
            wb = __builtin_amdgcn_readfirstlane(wb);
            if (srch) l_pairs[wb + __popcll(mb & ((1ull << lane) - 1ull))] = (uint16_t)q;
        }
        __syncthreads();
        const int32_t nsrch = sh.nlist;
        for (int32_t grp = 0; grp * KP * NT < nsrch; ++grp) {
            int32_t lo[KP], hi[KP], qq[KP], p1[KP], p2[KP];
            int64_t ca[KP], cc[KP];
#pragma unroll
            for (int k = 0; k < KP; ++k) {
                const int32_t i = tid + (grp * KP + k) * NT;
                lo[k] = 0;
                hi[k] = 0;
                qq[k] = -1;
                ca[k] = 0;
                cc[k] = 0;
                p1[k] = p2[k] = 0;
                if (i < nsrch) {
                    qq[k] = l_pairs[i];
                    int32_t m;
                    pair(qq[k], ca[k], cc[k], m, p1[k], p2[k]);
                    lo[k] = 1;                 // block 0 is common
                    hi[k] = m;
                }
            }
            for (;;) {
                bool any = false;
#pragma unroll
                for (int k = 0; k < KP; ++k) any |= lo[k] < hi[k];
                if (!any) break;
                // addresses by masks (a closed search reads the first chain hash), so that the KP
                // pairs' loads are in flight together
                int32_t mid[KP];
                uint64_t va[KP], vb[KP];
#pragma unroll
                for (int k = 0; k < KP; ++k) {
                    mid[k] = (lo[k] + hi[k]) >> 1;
                    const int64_t mk = -(int64_t)(lo[k] < hi[k]);
                    va[k] = a.chains[mk & (ca[k] + mid[k])];
                    vb[k] = a.chains[mk & (cc[k] + mid[k])];
                }
#pragma unroll
                for (int k = 0; k < KP; ++k) {
                    if (lo[k] < hi[k]) {
                        if (va[k] == vb[k]) lo[k] = mid[k] + 1;
                        else hi[k] = mid[k];
                    }
                }
            }
#pragma unroll
            for (int k = 0; k < KP; ++k)
                if (qq[k] >= 0) store(qq[k], p1[k], p2[k], lo[k]);
        }
        __syncthreads();
    };
    // pair q of the batch: routes b1 > b2 (q = b1 (b1 - 1) / 2 + b2)
    auto batch_pair = [&](int32_t q, int64_t& ca, int64_t& cc, int32_t& m, int32_t& b1, int32_t& b2) {
        b1 = (int32_t)((1.0f + sqrtf(1.0f + 8.0f * (float)q)) * 0.5f);
        while (b1 > 1 && b1 * (b1 - 1) / 2 > q) --b1;
        while ((b1 + 1) * b1 / 2 <= q) ++b1;
        b2 = q - b1 * (b1 - 1) / 2;
        ca = r_cb[b1];
        cc = r_cb[b2];
        m = min(r_P[b1], r_P[b2]);
        return m > 0 && r_first[b1] == r_first[b2];
    };

    // the request at queue position qi: conversation, turn, prompt blocks and chain base
    auto queued = [&](int32_t qi, int32_t& c, int32_t& k, int64_t& turn, int32_t& P, int64_t& cb, bool& more) {
        c = g_queue[qi >= qcap ? qi - qcap : qi];
        k = g_next[c];
        const int64_t g = gc0 + c;
        const int64_t tb0 = a.turn_off[g], tb1 = a.turn_off[g + 1];
        turn = tb0 + k;
        P = a.turn_blocks[turn];
        cb = a.chain_off[g];
        const int64_t ce = a.chain_off[g + 1];
        if (P < 0 || (int64_t)P > ce - cb) {
            atomicOr(a.status, RK_DEV_SHORT_INPUT);
            P = P < 0 ? 0 : (int32_t)max((int64_t)0, ce - cb);
        }
        if (cb < 0 || cb >= (1ll << 40)) {     // a run keeps 40 bits of its chain's base
            atomicOr(a.status, RK_DEV_BAD_OFFSETS);
            P = 0;
        }
        if (P > a.max_blocks) {
            atomicOr(a.status, RK_DEV_TOO_LARGE);
            P = a.max_blocks;
        }
        more = (int64_t)k + 1 < tb1 - tb0;
    };
    int32_t nb_cur = 0;            // routes of the batch being decided
    // Waves 1-3: every (request, worker) overlap of the next batch (all workers add runs), by the
    // run-index search of run_searches: a first probe of block 0 settles the misses and lists the
    // rest; once the three waves have listed theirs, the listed items are searched with KI slots
    // per thread, each slot taking the next listed item when its search ends.
    auto job_search_part = [&]() {
        enum : int32_t { DONE = 0, HASH = 1, LOOK = 2, CMP = 3, CKPT = 4 };
        constexpr int NJ = NT - 128;                 // the searching threads
        const int32_t tj = tid - 64;
        const int32_t n = NB * W;
        for (int32_t base = 0; base < n; base += NJ * KI) {
            int32_t jw[KI];
            uint64_t h0[KI], x0[KI], x1[KI], y0[KI], y1[KI];
            bool own[KI];
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                const int32_t i = base + u * NJ + tj;
                const int32_t b = i / W;
                jw[u] = i - b * W;
                own[u] = i < n && nx_P[b < NB ? b : 0] > 0;
                if (i < n && !own[u]) nx_o[i] = 0;
                h0[u] = own[u] ? nx_first[b] : 0ull;
                const uint64_t g = (uint64_t)(-(int64_t)own[u]) & run_home(h0[u], jw[u], rsmask);
                load_run(g_runs + g, x0[u], y0[u]);
                load_run(g_runs + g + 1, x1[u], y1[u]);
            }
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                const int32_t i = base + u * NJ + tj;
                bool hit = false;
                if (own[u]) {
                    const uint64_t kk[2] = {x0[u], x1[u]}, vv[2] = {y0[u], y1[u]};
                    uint64_t val;
                    hit = run_finish(g_runs, rsmask, h0[u], jw[u], run_home(h0[u], jw[u], rsmask), kk, vv, val);
                    if (!hit) nx_o[i] = 0;
                }
                const unsigned long long m = __ballot(hit);
                int32_t wb = 0;
                if (lane == 0 && m) wb = atomicAdd(&sh.jn, (int32_t)__popcll(m));
                wb = __builtin_amdgcn_readfirstlane(wb);
                if (hit) l_items[wb + __popcll(m & ((1ull << lane) - 1ull))] = (uint16_t)i;
            }
        }
        // barrier of the searching waves: their lists are complete
        ep_wave_sync();
        if (lane == 0) __hip_atomic_fetch_add(&sh.jsync, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP);
        while (__builtin_amdgcn_readfirstlane(
                   __hip_atomic_load(&sh.jsync, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP)) < NW - 2)
            __builtin_amdgcn_s_sleep(1);
        const int32_t n2 = __hip_atomic_load(&sh.jn, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
        const uint64_t* chains = a.chains;
        int64_t cb[KI], rcb[KI];
        int32_t P[KI], jw[KI], o[KI], lo[KI], hi[KI], mode[KI], km[KI], lim[KI], item[KI];
        uint64_t hq[KI], qhi[KI];
        bool qok[KI];
        // slot u takes listed item idx (or none)
        auto take = [&](int u, int32_t idx) {
            item[u] = -1;
            mode[u] = DONE;
            if (idx >= n2) return;
            const int32_t i = l_items[idx];
            const int32_t b = i / W;
            item[u] = i;
            jw[u] = i - b * W;
            cb[u] = nx_cb[b];
            P[u] = nx_P[b];
            hq[u] = nx_first[b];
            rcb[u] = 0;
            o[u] = 0;
            qhi[u] = 0ull;
            qok[u] = false;
            lo[u] = 0;
            hi[u] = (P[u] + kCkpt - 1) >> kCkptLog;
            km[u] = 0;
            lim[u] = P[u];
            mode[u] = CKPT;
        };
#pragma unroll
        for (int u = 0; u < KI; ++u) {
            cb[u] = rcb[u] = 0;
            P[u] = jw[u] = o[u] = lo[u] = hi[u] = km[u] = lim[u] = 0;
            hq[u] = qhi[u] = 0ull;
            qok[u] = false;
            take(u, atomicAdd(&sh.jnext, 1));
        }
        for (;;) {
            bool any = false;
#pragma unroll
            for (int u = 0; u < KI; ++u) any |= mode[u] != DONE;
            if (!any) break;
            uint64_t x0[KI], x1[KI], y0[KI], y1[KI], hc[KI], hd[KI];
            int32_t mid[KI];
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                mid[u] = (lo[u] + hi[u]) >> 1;
                const int32_t md = mode[u];
                const int32_t mC = -(int32_t)(md == CKPT), mH = -(int32_t)(md == HASH), mM = -(int32_t)(md == CMP);
                const int32_t mP = -(int32_t)(md == CKPT || md == LOOK);
                const int32_t mh = km[u] + 1 < hi[u] ? (km[u] + 1 + hi[u]) >> 1 : 0;
                const int32_t mm = lo[u] < km[u] ? (lo[u] + km[u]) >> 1 : 0;
                const int32_t ic = (mC & (mh << kCkptLog)) | (mH & o[u]) | (mM & mid[u]);
                const int32_t id = (mC & (mm << kCkptLog)) | (mM & mid[u]);
                const int64_t bc = (int64_t)(mC | mH | mM) & cb[u];
                const int64_t bd = ((int64_t)mC & cb[u]) | ((int64_t)mM & rcb[u]);
                const uint64_t g = (uint64_t)(int64_t)mP & run_home(hq[u], jw[u], rsmask);
                x0[u] = y0[u] = x1[u] = y1[u] = hc[u] = hd[u] = 0ull;
                if (__ballot(mP != 0)) {
                    load_run(g_runs + g, x0[u], y0[u]);
                    load_run(g_runs + g + 1, x1[u], y1[u]);
                }
                if (__ballot((mC | mH | mM) != 0)) hc[u] = chains[bc + ic];
                if (__ballot((mC | mM) != 0)) hd[u] = chains[bd + id];
            }
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                if (mode[u] == CKPT) {
                    const uint64_t kk[2] = {x0[u], x1[u]}, vv[2] = {y0[u], y1[u]};
                    uint64_t val = 0ull;
                    if (run_finish(g_runs, rsmask, hq[u], jw[u], run_home(hq[u], jw[u], rsmask), kk, vv, val)) {
                        rcb[u] = (int64_t)(val >> 24);
                        o[u] = (int32_t)(val & 0xFFFFu);
                        lo[u] = km[u] + 1;
                        hq[u] = hc[u];
                    } else {
                        hi[u] = km[u];
                        hq[u] = hd[u];
                    }
                    km[u] = (lo[u] + hi[u]) >> 1;
                    if (lo[u] >= hi[u]) {
                        if (lo[u] == 0) {
                            mode[u] = DONE;
                        } else {
                            const int32_t c = (lo[u] - 1) << kCkptLog;
                            lim[u] = min(P[u], lo[u] << kCkptLog);
                            const int32_t m = min(lim[u], o[u]);
                            lo[u] = c + 1;
                            hi[u] = m;
                            qok[u] = false;
                            if (lo[u] >= hi[u]) {
                                o[u] = m;
                                mode[u] = o[u] < lim[u] ? HASH : DONE;
                            } else {
                                mode[u] = CMP;
                            }
                        }
                    }
                } else if (mode[u] == HASH) {
                    hq[u] = hc[u];
                    mode[u] = LOOK;
                } else if (mode[u] == LOOK) {
                    const uint64_t kk[2] = {x0[u], x1[u]}, vv[2] = {y0[u], y1[u]};
                    uint64_t val = 0ull;
                    if (!run_finish(g_runs, rsmask, hq[u], jw[u], run_home(hq[u], jw[u], rsmask), kk, vv, val)) {
                        mode[u] = DONE;
                    } else {
                        rcb[u] = (int64_t)(val >> 24);
                        const int32_t m = min(lim[u], (int32_t)(val & 0xFFFFu));
                        lo[u] = o[u] + 1;
                        hi[u] = m;
                        qok[u] = false;
                        if (lo[u] >= hi[u]) {
                            o[u] = m;
                            mode[u] = o[u] < lim[u] ? HASH : DONE;
                        } else {
                            mode[u] = CMP;
                        }
                    }
                } else if (mode[u] == CMP) {
                    if (hc[u] == hd[u]) {
                        lo[u] = mid[u] + 1;
                    } else {
                        hi[u] = mid[u];
                        qhi[u] = hc[u];
                        qok[u] = true;
                    }
                    if (lo[u] >= hi[u]) {
                        o[u] = lo[u];
                        if (o[u] >= lim[u]) {
                            mode[u] = DONE;
                        } else if (qok[u]) {
                            hq[u] = qhi[u];
                            mode[u] = LOOK;
                        } else {
                            mode[u] = HASH;
                        }
                    }
                }
                if (mode[u] == DONE && item[u] >= 0) {
                    nx_o[item[u]] = o[u];
                    take(u, atomicAdd(&sh.jnext, 1));
                }
            }
        }
    };
    auto job_pair_part = [&]() {
        // ---- common prefixes of pairs (pair(q, ...) as for pair_lcps): direct(q, b1, b2, same, m)
        //      stores a pair's prefix at once or returns true to list the pair; the listed pairs are
        //      searched with KP slots per thread, each taking the next listed pair when its search
        //      ends, store(listed index, q, prefix)
        auto job_pairs = [&](int32_t npair, int32_t* cnt, int32_t* next, const auto& pair, const auto& direct,
                             const auto& store) {
            for (int32_t q0 = 0; q0 < npair; q0 += 64) {
                const int32_t q = q0 + lane;
                bool lst = false;
                if (q < npair) {
                    int64_t ca, cc;
                    int32_t m, b1, b2;
                    const bool same = pair(q, ca, cc, m, b1, b2);
                    lst = direct(q, b1, b2, same, m);
                }
                const unsigned long long mb = __ballot(lst);
                int32_t wb = 0;
                if (lane == 0 && mb) wb = atomicAdd(cnt, (int32_t)__popcll(mb));
                wb = __builtin_amdgcn_readfirstlane(wb);
                if (lst) l_pairs[wb + __popcll(mb & ((1ull << lane) - 1ull))] = (uint16_t)q;
            }
            ep_wave_sync();
            const int32_t nl = __builtin_amdgcn_readfirstlane(
                __hip_atomic_load(cnt, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP));
            int32_t lo[KP], hi[KP], it[KP];
            int64_t ca[KP], cc[KP];
            auto takep = [&](int k, int32_t idx) {
                it[k] = -1;
                lo[k] = hi[k] = 0;
                ca[k] = cc[k] = 0;
                if (idx >= nl) return;
                int32_t m, b1, b2;
                it[k] = idx;
                pair(l_pairs[idx], ca[k], cc[k], m, b1, b2);
                lo[k] = 1;                 // block 0 is common
                hi[k] = m;
            };
#pragma unroll
            for (int k = 0; k < KP; ++k) takep(k, atomicAdd(next, 1));
            for (;;) {
                bool any = false;
#pragma unroll
                for (int k = 0; k < KP; ++k) any |= it[k] >= 0;
                if (!any) break;
                int32_t mid[KP];
                uint64_t va[KP], vb[KP];
#pragma unroll
                for (int k = 0; k < KP; ++k) {
                    mid[k] = (lo[k] + hi[k]) >> 1;
                    const int64_t mk = -(int64_t)(lo[k] < hi[k]);
                    va[k] = a.chains[mk & (ca[k] + mid[k])];
                    vb[k] = a.chains[mk & (cc[k] + mid[k])];
                }
#pragma unroll
                for (int k = 0; k < KP; ++k) {
                    if (lo[k] < hi[k]) {
                        if (va[k] == vb[k]) lo[k] = mid[k] + 1;
                        else hi[k] = mid[k];
                    }
                    if (it[k] >= 0 && lo[k] >= hi[k]) {
                        store(it[k], (int32_t)l_pairs[it[k]], lo[k]);
                        takep(k, atomicAdd(next, 1));
                    }
                }
            }
        };
        // within the next batch, into nx_lcp
        job_pairs(
            NB * (NB - 1) / 2, &sh.jp, &sh.jpnext,
            [&](int32_t q, int64_t& ca, int64_t& cc, int32_t& m, int32_t& b1, int32_t& b2) {
                b1 = (int32_t)((1.0f + sqrtf(1.0f + 8.0f * (float)q)) * 0.5f);
                while (b1 > 1 && b1 * (b1 - 1) / 2 > q) --b1;
                while ((b1 + 1) * b1 / 2 <= q) ++b1;
                b2 = q - b1 * (b1 - 1) / 2;
                ca = nx_cb[b1];
                cc = nx_cb[b2];
                m = min(nx_P[b1], nx_P[b2]);
                return m > 0 && nx_first[b1] == nx_first[b2];
            },
            [&](int32_t q, int32_t b1, int32_t b2, bool same, int32_t m) {
                if (same && m > 1) return true;
                nx_lcp[b2 * NB + b1] = (uint16_t)(same && m > 0 ? 1 : 0);
                return false;
            },
            [&](int32_t idx, int32_t q, int32_t l) {
                int32_t b1 = (int32_t)((1.0f + sqrtf(1.0f + 8.0f * (float)q)) * 0.5f);
                while (b1 > 1 && b1 * (b1 - 1) / 2 > q) --b1;
                while ((b1 + 1) * b1 / 2 <= q) ++b1;
                nx_lcp[(q - b1 * (b1 - 1) / 2) * NB + b1] = (uint16_t)l;
            });
        ep_wave_sync();            // the within-batch list is no longer read
        // between the next batch's routes and this batch's (nb routes), every pair whose first
        // blocks agree listed, its prefix in l_pval: the overlaps rise by them at the next batch
        const int32_t nbc = nb_cur;
        job_pairs(
            NB * nbc, &sh.jq, &sh.jqnext,
            [&](int32_t q, int64_t& ca, int64_t& cc, int32_t& m, int32_t& b1, int32_t& b2) {
                b1 = q / nbc;
                b2 = q - b1 * nbc;
                ca = nx_cb[b1];
                cc = r_cb[b2];
                m = min(nx_P[b1], r_P[b2]);
                return m > 0 && nx_first[b1] == r_first[b2];
            },
            [&](int32_t q, int32_t b1, int32_t b2, bool same, int32_t m) { return same; },
            [&](int32_t idx, int32_t q, int32_t l) { l_pval[idx] = (uint16_t)l; });
    };
    // The job's two parts run side by side: waves 1 .. NW-2 search the run index, the last wave
    // takes the common prefixes of the batch pairs.
    auto next_batch_job = [&]() {
        if (wave == NW - 1) {
            job_pair_part();
        } else {
            __builtin_amdgcn_s_setprio(2);   // the searches end the job: ahead of writers and pairs
            job_search_part();
            __builtin_amdgcn_s_setprio(0);
        }
    };

    // the next batch's overlaps, computed by waves 1-3 while wavefront 0 decides this batch
    // (run-index searches against the caches as this batch found them); nx_ready: they are
    // complete and this batch had no eviction, compaction or epoch stop, so the caches grew by
    // this batch's chains only
    bool nx_ready = false;
    int32_t nb_prev = 0;
    for (;;) {
        // ---- A. the batch: the next nb queued requests (queue order is routing order)
        const int32_t qh0 = sh.qhead;
        const int32_t tb0 = sh.tdone;        // routes decided before this batch
        int32_t nb = min(NB, sh.qsize);
        const bool pre = nx_ready && nb == NB;
        if (pre) {
            // the precomputed batch's common prefixes become the batch's; a route of the batch just
            // decided added its chain to its worker's cache, so the precomputed overlap of a next
            // route on that worker rises to their common prefix (the decided batch's arrays are
            // still in place)
            uint16_t* tl = l_lcp;
            l_lcp = nx_lcp;
            nx_lcp = tl;
            const int32_t nxl = sh.jq;
            for (int32_t i = tid; i < nxl; i += NT) {
                const int32_t q = l_pairs[i], l = l_pval[i];
                const int32_t b1 = q / nb_prev, b2 = q - b1 * nb_prev;
                if (l > 0) atomicMax(&nx_o[b1 * W + r_sig[b2]], l);
            }
            __syncthreads();
        }
        for (int32_t b = tid; b < nb; b += NT) {
            int32_t c, k, P;
            int64_t turn, cb;
            bool more;
            queued(qh0 + b, c, k, turn, P, cb, more);
            r_c[b] = c | (more ? kMoreTurns : 0);
            r_k[b] = k;
            r_turn[b] = (int32_t)turn;
            r_P[b] = P;
            r_cb[b] = cb;
            r_last[b] = P > 0 ? a.chains[cb + P - 1] : 0ull;
            r_first[b] = P > 0 ? a.chains[cb] : 0ull;
            const int64_t row = prm.out_base + (int64_t)sh.tdone + b;
            r_rnd[2 * b] = draws ? a.route_rand[2 * row] : 0u;
            r_rnd[2 * b + 1] = draws ? a.route_rand[2 * row + 1] : 0u;
        }
        __syncthreads();
        // room in a worker's table and log is checked route by route when the route is decided
        if (tid == 0) sh.nb = nb;
        if (tid == 0) {
            sh.decided = 0;
            sh.claimed = 0;
            sh.stop = 0;
        }
        __syncthreads();
        nb = sh.nb;
        if (pre) {
            // the overlaps computed during the previous batch, raised above
            for (int32_t i = tid; i < nb * W; i += NT) o_tab[i] = o_cur[i] = nx_o[i];
            __syncthreads();
        } else {
            // every (request, worker) overlap against the caches as they stand
            search(0, nb, -1);
            if (tiers) tier_search(0, nb, -1);
            if (!scan) pair_lcps(nb * (nb - 1) / 2, batch_pair, [&](int32_t q, int32_t b1, int32_t b2, int32_t l) {
                l_lcp[b2 * NB + b1] = (uint16_t)l;
            });
        }
        // the next batch is searched during this batch's decisions when every worker still adds
        // runs (no recency kept: the run index is all the searches read) and the queue already
        // holds all of the next batch
        bool job = false;
        if (lean || lean_ctrl) {
            bool stamped_any = false;
            for (int32_t j = 0; j < W; ++j) stamped_any |= s_stamped[j] != 0;
            job = !stamped_any && sh.qsize >= nb + NB;
        }
        if (job) {
            for (int32_t b = tid; b < NB; b += NT) {
                int32_t c, k, P;
                int64_t turn, cb;
                bool more;
                queued(qh0 + nb + b, c, k, turn, P, cb, more);
                nx_cb[b] = cb;
                nx_P[b] = P;
                nx_first[b] = P > 0 ? a.chains[cb] : 0ull;
            }
            if (tid == 0) {
                sh.jn = 0;
                sh.jsync = 0;
                sh.jnext = 0;
                sh.jp = 0;
                sh.jpnext = 0;
                sh.jq = 0;
                sh.jqnext = 0;
            }
            __syncthreads();
        }

        // ---- B. routing decisions in order (wavefront 0); stops for a flush, a new batch or the end
        const int32_t t0 = t;
        int32_t event = EV_BATCH;
        // ---- B. the decisions of wavefront 0 (below).  LN: the episode runs in prefix
        // mode, routed by argmin under LRU, without memory tiers or the regime controller
        // (LC: with the load controller, else without); those copies of the decision loop
        // are compiled with the other features switched off, which shortens the serial
        // decision chain.
        auto decide = [&](auto lean_tag) {
            constexpr bool LN = decltype(lean_tag)::value != 0;
            constexpr bool LC = decltype(lean_tag)::value == 2;
            const bool freq_d = !LN && freq, tiers_d = !LN && tiers, regime_d = !LN && regime_ctl, scan_d = !LN && scan;
            const bool ctrl1_d = LC || (!LN && prm.controller == 1);
            const int32_t policy_d = LN ? RK_POLICY_ARGMIN : policy;
            event = EV_BATCH;
            // lane j < W keeps worker j's load, log tail and block counts in registers
            int32_t rA = 0, rlive = 0, rused = 0, rN = 0;
            uint32_t rtail = 0;
            int32_t run_ep = -1;   // decay epoch of the routes decided since the last sync
            int32_t q_head = sh.qhead, q_size = sh.qsize;   // the ready queue, kept in registers
            if (lane < W) {
                rA = s_A[lane];
                rN = s_N[lane];
                rtail = s_tail[lane];
                rlive = s_live[lane];
                rused = s_used[lane];
            }
            // workers that keep recency (write log records)
            const unsigned long long stamped_mask = __ballot(lane < W && s_stamped[lane] != 0);
            // writes of the batch's routes decided so far (run-index entries or touches; the
            // decisions go on in the same batch after a stop)
            int32_t rwork = t > t0 ? r_wend[t - t0 - 1] : 0;
            for (;;) {
                if (!step_open) {
                    // release the routes of step s - H; queue their conversations' next turns
                    const int32_t slot = s_slot, sb = slot * rps;
                    if (s >= H) {
                        if (lane < W) {
                            s_A[lane] = rA;
                            s_N[lane] = rN;
                        }
                        ep_wave_sync();
                        const int32_t nprev = s_stepn[slot];
                        const int32_t qtail = q_head + q_size;
                        int32_t pushed = 0, rel = 0;
                        for (int32_t base = 0; base < nprev; base += 64) {
                            const int32_t r = base + lane;
                            bool more = false;
                            int32_t c = 0;
                            if (r < nprev) {
                                const int32_t cc = s_stc[sb + r];
                                c = cc & ~kMoreTurns;
                                more = (cc & kMoreTurns) != 0;
                                rel += s_stP[sb + r];
                                atomicSub(&s_A[s_stw[sb + r]], s_stP[sb + r]);
                                atomicSub(&s_N[s_stw[sb + r]], 1);
                            }
                            const unsigned long long mb = __ballot(more);
                            if (more) {
                                int32_t qi = qtail + pushed + __popcll(mb & ((1ull << lane) - 1ull));
                                g_queue[qi >= qcap ? qi - qcap : qi] = c;
                            }
                            pushed += __popcll(mb);
                        }
                        u_tot -= wave_sum_i32(rel);
                        ep_wave_sync();
                        q_size += pushed;
                        if (lane < W) {
                            rA = s_A[lane];
                            rN = s_N[lane];
                        }
                        ep_wave_sync();
                    }
                    int32_t inflight = 0;
                    for (int32_t k = 1; k < H && k <= s; ++k) inflight += s_stepn[s_slot >= k ? s_slot - k : s_slot - k + H];
                    const int32_t qs = q_size;
                    if (qs == 0 && inflight == 0) {
                        event = EV_DONE;
                        break;
                    }
                    n_step = min(rps, qs);
                    if (lane == 0) s_stepn[slot] = n_step;
                    if (n_step > 0) tot[5] = s + 1;
                    r_in_step = 0;
                    step_open = true;
                    ep_wave_sync();
                }
                if (r_in_step >= n_step) {
                    ++s;
                    s_slot = s_slot + 1 == H ? 0 : s_slot + 1;
                    step_open = false;
                    continue;
                }
                const int32_t b = t - t0;
                if (b >= nb) break;
                if (__builtin_expect(freq_d, 0)) {
                    // a new decay epoch waits until the earlier epoch's cache writes are in
                    const int32_t ep = s / dsteps;
                    if (run_ep >= 0 && ep != run_ep) {
                        event = EV_EPOCH;
                        break;
                    }
                    run_ep = ep;
                }
                // one route: controller, cost of every worker, argmin
                const int32_t slot = s_slot, sb = slot * rps;
                bool active = false;
                if (__builtin_expect(ctrl1_d && t >= prm.ctrl_window, 0))
                    active = (int64_t)prm.ctrl_den * u_sum >
                             (int64_t)prm.ctrl_num * prm.ctrl_window * W * (int64_t)prm.cap_blocks;
                float w = prm.w_ov;
                if (active) w = fminf(prm.w_ov, prm.ctrl_w_ov);
                int32_t pol = policy_d;
                float tau_r = tau;
                if (__builtin_expect(regime_d, 0)) {
                    w = rg.w_ov[rg_r];
                    tau_r = rg.tau[rg_r];
                    pol = tau_r > 0.0f ? RK_POLICY_SOFTMAX : RK_POLICY_ARGMIN;
                }
                const int32_t P = r_P[b];
                const int64_t row = prm.out_base + (int64_t)t;
                uint32_t bits = 0xFFFFFFFFu;
                int32_t oj = 0;
                float cj = 0.0f;
                if (lane < W) {
                    oj = o_cur[b * W + lane];
                    if (__builtin_expect(tiers_d, 0)) {
                        const int32_t o1 = t1_tab[b * W + lane], o12 = t12_tab[b * W + lane];
                        cj = route_cost_tiers(w, prm.w_act, prm.w_sat, prm.cap_blocks, P, oj, o1, o12,
                                              prm.tier_w, rA);
                        if (a.out.tier_overlap) {
                            a.out.tier_overlap[(row * W + lane) * 2] = o1;
                            a.out.tier_overlap[(row * W + lane) * 2 + 1] = o12;
                        }
                    } else {
                        cj = route_cost_ep(w, prm.w_act, prm.w_sat, prm.cap_blocks, inv_cap, P, oj, rA);
                    }
                    if (a.out.cost) a.out.cost[row * W + lane] = cj;
                    bits = __float_as_uint(__fadd_rn(cj, 0.0f));
                }
                int32_t sg;
                if (__builtin_expect(pol == RK_POLICY_ARGMIN, 1)) {
                    const uint32_t mn = ep_wave_min_u32(bits);
                    sg = __ffsll(__ballot(lane < W && bits == mn)) - 1;
                } else if (pol == RK_POLICY_SOFTMAX) {
                    // weights exp((c_min - c_j) / tau); running sums in worker order
                    const float cmin = __uint_as_float(ep_wave_min_u32(bits));
                    const float ej = lane < W ? exp_neg_f32(__fdiv_rn(__fsub_rn(cmin, cj), tau_r)) : 0.0f;
                    float total = 0.0f;
                    for (int32_t j = 0; j < W; ++j)
                        total = __fadd_rn(total, __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ej), j)));
                    const float u = __fmul_rn((float)(r_rnd[2 * b] >> 8), 5.9604644775390625e-8f);
                    const float thr = __fmul_rn(u, total);
                    float run = 0.0f;
                    int32_t last = 0;
                    sg = -1;
                    for (int32_t j = 0; j < W && sg < 0; ++j) {
                        const float e = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ej), j));
                        run = __fadd_rn(run, e);
                        if (e > 0.0f) last = j;
                        if (run > thr) sg = j;
                    }
                    if (sg < 0) sg = last;
                } else if (pol == RK_POLICY_ROUND_ROBIN) {
                    sg = t % W;
                } else {
                    const int32_t ca = (int32_t)(((uint64_t)r_rnd[2 * b] * (uint64_t)W) >> 32);
                    sg = ca;
                    if (pol == RK_POLICY_P2C && W > 1) {
                        int32_t cb2 = (int32_t)(((uint64_t)r_rnd[2 * b + 1] * (uint64_t)(W - 1)) >> 32);
                        if (cb2 >= ca) ++cb2;
                        const float fa = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cj), ca));
                        const float fb = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cj), cb2));
                        if (fb < fa || (fb == fa && cb2 < ca)) sg = cb2;
                    }
                }
                const int32_t osg = __builtin_amdgcn_readlane(oj, sg);
                const int32_t live_after = __builtin_amdgcn_readlane(rlive, sg) + (scan_d ? 0 : P - osg);
                const uint32_t base = (uint32_t)__builtin_amdgcn_readlane((int)rtail, sg);
                const bool flush = scan_d || tiers_d || live_after > a.cache;
                // a worker that keeps recency needs log records for the route's P touches and slots
                // for its new blocks: without room, stop before the route and compact that worker
                // (the cached sets and loads stay as they are, so the route is decided again alike)
                if (__builtin_expect((stamped_mask >> sg) & 1ull, 0)) {
                    const uint32_t head = s_head[sg];
                    const uint64_t add = scan_d ? (uint64_t)P : (uint64_t)(P - osg);
                    if ((uint64_t)(uint32_t)__builtin_amdgcn_readlane(rused, sg) + add > used_limit ||
                        (uint64_t)(base - head) + (uint64_t)P > R || (uint64_t)base + (uint64_t)P > 0x40000000u) {
                        if (room_b == t) {
                            // still no room right after a compaction (the workspace layout always
                            // leaves room for one route): report it and go on
                            if (lane == 0) atomicOr(a.status, RK_DEV_TABLE_FULL);
                        } else {
                            room_b = t;
                            if (lane == 0) sh.ev_b = sg;
                            event = EV_ROOM;
                            break;
                        }
                    }
                }
                if (active) {
                    tot[3] += 1;
                    if (!prev_active) tot[4] += 1;
                }
                prev_active = active;
                if (regime_d && rg_r > 0) tot[3] += 1;
                const int32_t rc = r_c[b];
                if (lane == sg) {
                    rA += P;
                    rN += 1;
                    rtail = base + (uint32_t)P;
                    if (!scan_d) {
                        rlive = live_after;
                        rused += P - osg;
                    }
                }
                rwork += ((stamped_mask >> sg) & 1ull) ? P : (osg < P ? run_entries(osg, P) : 0);
                if (lane == 0) {
                    r_sig[b] = sg;
                    r_wend[b] = rwork;
                    r_stamp[b] = base;
                    r_ep[b] = freq_d ? (uint32_t)run_ep : 0u;
                    g_hist[2 * t] = rc & ~kMoreTurns;
                    g_hist[2 * t + 1] = P | (sg << 16);
                    r_otab[b] = o_tab[b * W + sg];
                    s_stw[sb + r_in_step] = sg;
                    s_stP[sb + r_in_step] = P;
                    s_stc[sb + r_in_step] = rc;
                    g_next[rc & ~kMoreTurns] = r_k[b] + 1;
                    r_step[b] = (int32_t)s;
                    r_reg[b] = regime_d ? rg_r : 0;
                    r_evc[b] = 0;
                    r_evd[b] = 0ull;
                    if (flush) {
                        sh.ev_b = b;
                        sh.ev_row = row;
                    }
                }
                u_tot += P;
                q_head = q_head + 1 == qcap ? 0 : q_head + 1;
                q_size -= 1;
                if (__builtin_expect(regime_d, 0)) {
                    // the chosen worker's latency with the new request (already counted in
                    // lane sg's rN) stands in for TTFT (fp64)
                    const int32_t n_sg = __builtin_amdgcn_readlane(rN, sg);
                    double gap = (double)(rg.n_sat - n_sg);
                    gap = gap < 1.0 ? 1.0 : gap;
                    double pw = gap;
                    for (int32_t i = 1; i < rg.beta; ++i) pw = __dmul_rn(pw, gap);
                    const double lat = __dadd_rn(__dadd_rn(__dmul_rn(rg.a, (double)n_sg), rg.b), __ddiv_rn(rg.d, pw));
                    rg_ewma = t == 0 ? lat
                                     : __dadd_rn(__dmul_rn(rg.alpha, lat), __dmul_rn(__dsub_rn(1.0, rg.alpha), rg_ewma));
                    if (rg_r == 0) {
                        rg_up = rg_ewma > rg.theta1 ? rg_up + 1 : 0;
                        if (rg_up >= rg.k) {
                            rg_r = 1;
                            rg_up = rg_down = 0;
                            tot[4] += 1;
                        }
                    } else if (rg_r == 1) {
                        rg_up = rg_ewma >= rg.theta2 ? rg_up + 1 : 0;
                        rg_down = rg_ewma < __dsub_rn(rg.theta1, rg.eps) ? rg_down + 1 : 0;
                        if (rg_up >= rg.k) {
                            rg_r = 2;
                            rg_up = rg_down = 0;
                            tot[4] += 1;
                        } else if (rg_down >= rg.k) {
                            rg_r = 0;
                            rg_up = rg_down = 0;
                        }
                    } else {
                        rg_down = rg_ewma < __dsub_rn(rg.theta2, rg.eps) ? rg_down + 1 : 0;
                        if (rg_down >= rg.k) {
                            rg_r = 1;
                            rg_up = rg_down = 0;
                        }
                    }
                }
                if (__builtin_expect(ctrl1_d, 0)) {
                    const int32_t pos = c_pos;
                    c_pos = c_pos + 1 == prm.ctrl_window ? 0 : c_pos + 1;
                    if (t >= prm.ctrl_window) u_sum -= s_u[pos];
                    ep_wave_sync();
                    if (lane == 0) s_u[pos] = u_tot;
                    u_sum += u_tot;
                }
                tot[0] += P - osg;
                tot[2] += P;
                tot[6] += osg;
                // later requests of the batch now find this chain on sg
                if (!scan_d) {
                    const int32_t b2 = b + 1 + lane;
                    if (b2 < nb) {
                        const int32_t l = l_lcp[b * NB + b2];
                        if (l > o_cur[b2 * W + sg]) o_cur[b2 * W + sg] = l;
                    }
                }
                ++t;
                ++r_in_step;
                ep_wave_sync();
                if (lane == 0)
                    __hip_atomic_store(&sh.decided, b + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
                if (__builtin_expect(flush, 0)) {
                    event = EV_FLUSH;
                    break;
                }
            }
            if (lane < W) {
                s_A[lane] = rA;
                s_N[lane] = rN;
                s_tail[lane] = rtail;
                s_live[lane] = rlive;
                s_used[lane] = rused;
            }
            if (lane == 0) {
                sh.qhead = q_head;
                sh.qsize = q_size;
                sh.event = event;
                sh.tdone = t;
                __hip_atomic_store(&sh.stop, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
            }
        };
        nb_cur = nb;
        bool had_stop = false;      // an eviction, compaction or epoch stop in this batch
        bool job_ran = false;
        for (;;) {
            if (wave == 0) {
                // the serial chain of decisions goes first on its SIMD
                __builtin_amdgcn_s_setprio(3);
                if (!Queued && (lean || lean_ctrl) && t == t0) {
                    // a batch's first decisions in the one-episode kernel: the lean loop as a function
                    // of its own (the queued kernel, and the decisions after a stop, keep the copy
                    // inside the kernel and spare the call's register saves)
                    LeanCtx lc;
                    lc.sh = lds_off(&sh);
                    lc.s_A = lds_off(s_A);
                    lc.s_N = lds_off(s_N);
                    lc.s_tail = lds_off(s_tail);
                    lc.s_live = lds_off(s_live);
                    lc.s_used = lds_off(s_used);
                    lc.s_head = lds_off(s_head);
                    lc.s_stamped = lds_off(s_stamped);
                    lc.s_stw = lds_off(s_stw);
                    lc.s_stP = lds_off(s_stP);
                    lc.s_stc = lds_off(s_stc);
                    lc.s_stepn = lds_off(s_stepn);
                    lc.s_u = lds_off(s_u);
                    lc.r_P = lds_off(r_P);
                    lc.r_c = lds_off(r_c);
                    lc.r_k = lds_off(r_k);
                    lc.o_cur = lds_off(o_cur);
                    lc.o_tab = lds_off(o_tab);
                    lc.lcp = lds_off(l_lcp);
                    lc.r_sig = lds_off(r_sig);
                    lc.r_wend = lds_off(r_wend);
                    lc.r_stamp = lds_off(r_stamp);
                    lc.r_ep = lds_off(r_ep);
                    lc.r_otab = lds_off(r_otab);
                    lc.r_step = lds_off(r_step);
                    lc.r_reg = lds_off(r_reg);
                    lc.r_evc = lds_off(r_evc);
                    lc.r_evd = lds_off(r_evd);
                    lc.g_hist = (glb_p<int32_t>)g_hist;
                    lc.g_next = (glb_p<int32_t>)g_next;
                    lc.g_queue = (glb_p<int32_t>)g_queue;
                    lc.out_cost = (glb_p<float>)a.out.cost;
                    lc.status = (glb_p<int32_t>)a.status;
                    lc.out_base = prm.out_base;
                    lc.ctrl_thr = (int64_t)prm.ctrl_num * prm.ctrl_window * W * (int64_t)prm.cap_blocks;
                    lc.used_limit = used_limit;
                    lc.R = R;
                    lc.W = W;
                    lc.NB = NB;
                    lc.nb = nb;
                    lc.t0 = t0;
                    lc.H = H;
                    lc.rps = rps;
                    lc.qcap = qcap;
                    lc.cache = a.cache;
                    lc.ctrl_window = prm.ctrl_window;
                    lc.ctrl_den = prm.ctrl_den;
                    lc.cap_blocks = prm.cap_blocks;
                    lc.w_ov = prm.w_ov;
                    lc.w_act = prm.w_act;
                    lc.w_sat = prm.w_sat;
                    lc.ctrl_w_ov = prm.ctrl_w_ov;
                    lc.inv_cap = inv_cap;
                    LeanState ls;
                    ls.t = t;
                    ls.s = s;
                    ls.r_in_step = r_in_step;
                    ls.n_step = n_step;
                    ls.s_slot = s_slot;
                    ls.c_pos = c_pos;
                    ls.room_b = room_b;
                    ls.step_open = step_open;
                    ls.prev_active = prev_active;
                    ls.u_sum = u_sum;
                    ls.u_tot = u_tot;
                    for (int k = 0; k < 8; ++k) ls.tot[k] = tot[k];
                    if (lean_ctrl) lean_decide<true>(lc, &ls);
                    else lean_decide<false>(lc, &ls);
                    t = ls.t;
                    s = ls.s;
                    r_in_step = ls.r_in_step;
                    n_step = ls.n_step;
                    s_slot = ls.s_slot;
                    c_pos = ls.c_pos;
                    room_b = ls.room_b;
                    step_open = ls.step_open != 0;
                    prev_active = ls.prev_active != 0;
                    u_sum = ls.u_sum;
                    u_tot = ls.u_tot;
                    for (int k = 0; k < 8; ++k) tot[k] = ls.tot[k];
                } else if (lean) {
                    decide(LeanTag<1>{});
                } else if (lean_ctrl) {
                    decide(LeanTag<2>{});
                } else {
                    decide(LeanTag<0>{});
                }
                __builtin_amdgcn_s_setprio(0);
                writer();           // the decided routes not yet claimed
            } else {
                if (job) next_batch_job();
                writer();
            }
            job_ran = job_ran || job;
            job = false;
            __syncthreads();
            event = sh.event;
            if (event != EV_BATCH && event != EV_DONE) had_stop = true;
            if (event == EV_ROOM) {
                // every decided route's writes are in: compact the route's worker, then decide on
                rebuild(sh.ev_b);
                if (tid == 0) sh.stop = 0;
                __syncthreads();
                continue;
            }
            if (event == EV_EPOCH) {
                if (tid == 0) sh.stop = 0;
                __syncthreads();
                continue;
            }
            if (event != EV_FLUSH) break;
            // the route's worker (every decided route's writes are in): evict, search the pending
            // requests again
            const int32_t b = sh.ev_b;
            const int32_t sg = r_sig[b];
            if (tid == 0) {
                sh.stop = 0;
                if (scan) {
                    s_live[sg] += sh.ins;
                    s_used[sg] += sh.ins;
                }
                sh.ins = 0;
                sh.remaining = max(0, s_live[sg] - a.cache);
                sh.ev = 0;
                sh.digest = 0ull;
                sh.first_kept = 0xFFFFFFFFu;
            }
            __syncthreads();
            if (tiers) {
                // the route's P records joined both tier runs; its hits left them where their old
                // records lay inside
                if (tid == 0) {
                    s_n1[sg] += r_P[b] - sh.h1;
                    s_n2[sg] += r_P[b] - sh.h2;
                    sh.h1 = 0;
                    sh.h2 = 0;
                }
                __syncthreads();
                advance(s_b1, s_n1, K1, sg);
                advance(s_b2, s_n2, K12, sg);
            }
            if (!s_stamped[sg] && sh.remaining > 0) {
                // the worker's first eviction: its blocks go into its (cleared) block table with
                // the recency of its routes
                clear_tables(sg, sg + 1);
                __syncthreads();
                if (!materialize(sg, sh.tdone)) replay(sg, sh.tdone);
            }
            evict(sg, r_ep[b]);
            if (tiers) {
                // evictions take the oldest records: a run keeps at most the live count
                if (tid == 0) {
                    s_n1[sg] = min(s_n1[sg], s_live[sg]);
                    s_n2[sg] = min(s_n2[sg], s_live[sg]);
                    s_b1[sg] = max(s_b1[sg], s_head[sg]);
                    s_b2[sg] = max(s_b2[sg], s_head[sg]);
                }
                __syncthreads();
            }
            if (!scan && !tiers) research(b + 1, nb, sg);
            else search(b + 1, nb, sg);
            if (tiers) tier_search(b + 1, nb, sg);
            if (tid == 0) {
                r_evc[sh.ev_b] = sh.ev;
                r_evd[sh.ev_b] = sh.digest;
                sh.ev_total += sh.ev;
            }
            __syncthreads();
        }

        // the batch's per-route outputs, from LDS, by the whole workgroup
        {
            const int32_t nd = sh.tdone - tb0;
            const int64_t row0 = prm.out_base + (int64_t)tb0;
            for (int32_t b = tid; b < nd; b += NT) {
                const int64_t row = row0 + b;
                if (a.out.route_turn) a.out.route_turn[row] = r_turn[b];
                if (a.out.route_worker) a.out.route_worker[row] = r_sig[b];
                if (a.out.route_step) a.out.route_step[row] = r_step[b];
                if (a.out.route_blocks) a.out.route_blocks[row] = r_P[b];
                if (a.out.last_hash) a.out.last_hash[row] = r_last[b];
                if (a.out.route_regime) a.out.route_regime[row] = r_reg[b];
                if (a.out.evict_count) a.out.evict_count[row] = r_evc[b];
                if (a.out.evict_digest) a.out.evict_digest[row] = r_evd[b];
            }
            if (a.out.overlap)
                for (int32_t i = tid; i < nd * W; i += NT) a.out.overlap[row0 * W + i] = o_cur[i];
        }
        if (tid == 0) sh.ins = 0;
        __syncthreads();
        nx_ready = job_ran && !had_stop && event == EV_BATCH;
        nb_prev = nb;
        if (event == EV_DONE) break;
    }
    if (tid == 0 && a.out.totals) {
        int64_t cachedsum = 0;
        for (int32_t j = 0; j < W; ++j) cachedsum += s_live[j];
        tot[1] = sh.ev_total;
        tot[7] = cachedsum;
        for (int k = 0; k < 8; ++k) a.out.totals[(int64_t)e * 8 + k] = tot[k];
    }
    }();
    __syncthreads();
    }
}

}  // namespace rk

using namespace rk;

extern "C" size_t rk_simulate_workspace_size(int32_t E, int32_t W, int32_t cache_blocks, int32_t max_blocks,
                                             int32_t max_conv, int32_t max_routes)
{
    if (E < 0 || W < 1 || cache_blocks < 1 || max_blocks < 1 || max_conv < 0 || max_routes < 0) return 0;
    const EpisodeLayout L = episode_layout(W, cache_blocks, max_blocks, max_conv, max_routes);
    return L.per_episode * (size_t)E;
}

// Shape fields of a batch.
static int check_batch_shape(const char* who, const rk_episode_batch* b)
{
    if (b->E < 0) return fail(RK_EINVAL, "%s: E < 0", who);
    if (b->W < 1 || b->W > 64) return fail(RK_EUNSUPPORTED, "%s: W outside 1..64", who);
    if (b->cache_blocks < 1) return fail(RK_EINVAL, "%s: cache_blocks < 1", who);
    if (b->max_blocks < 1 || b->max_blocks > 8192) return fail(RK_EUNSUPPORTED, "%s: max_blocks outside 1..8192", who);
    if (b->max_conv < 0 || b->max_conv > (1 << 28)) return fail(RK_EINVAL, "%s: max_conv", who);
    if (b->max_inflight < 1 || b->max_inflight > 8192)
        return fail(RK_EUNSUPPORTED, "%s: max_inflight outside 1..8192", who);
    if (b->max_routes_per_step < 1 || b->max_routes_per_step > b->max_inflight)
        return fail(RK_EINVAL, "%s: max_routes_per_step outside 1..max_inflight", who);
    if (b->max_ctrl_window < 1 || b->max_ctrl_window > 4096)
        return fail(RK_EUNSUPPORTED, "%s: max_ctrl_window outside 1..4096", who);
    if (b->probe_mode != RK_PROBE_PREFIX && b->probe_mode != RK_PROBE_SCAN)
        return fail(RK_EINVAL, "%s: unknown probe_mode", who);
    if ((int64_t)b->cache_blocks + b->max_blocks > (1ll << 29)) return fail(RK_EUNSUPPORTED, "%s: cache too large", who);
    if (b->max_routes < 0) return fail(RK_EINVAL, "%s: max_routes < 0", who);
    if (b->flags != 0) return fail(RK_EINVAL, "%s: unknown flags %#x", who, (unsigned)b->flags);
    if (b->ws_slots < 0 || b->ws_pad != 0) return fail(RK_EINVAL, "%s: ws_slots < 0 or ws_pad != 0", who);
    return RK_OK;
}

// Episode workspaces a batch uses: one per episode, or ws_slots when fewer.
static int32_t batch_slots(const rk_episode_batch* b)
{
    return b->ws_slots > 0 && b->ws_slots < b->E ? b->ws_slots : b->E;
}

extern "C" int rk_simulate_episodes(const rk_episode_batch* b, const rk_episode_outputs* out, void* workspace,
                                    size_t ws_bytes, void* stream)
{
    if (!b || !out) return fail(RK_EINVAL, "rk_simulate_episodes: NULL batch or outputs");
    int rc = check_batch_shape("rk_simulate_episodes", b);
    if (rc) return rc;
    if (b->E == 0) return RK_OK;
    if (!b->params || !b->turn_off || !b->turn_blocks || !b->chain_off || !b->chains || !workspace)
        return fail(RK_EINVAL, "rk_simulate_episodes: NULL array");
    const EpisodeLayout L = episode_layout(b->W, b->cache_blocks, b->max_blocks, b->max_conv, b->max_routes);
    const int32_t n_slots = batch_slots(b);
    const size_t need = L.per_episode * (size_t)n_slots;
    if (ws_bytes < need)
        return fail(RK_ENOMEM, "rk_simulate_episodes: workspace %zu bytes < %zu needed", ws_bytes, need);
    int32_t* st = status_word();
    if (!st) return fail(RK_EHIP, "rk_simulate_episodes: no status word");

    EpArgs a;
    a.E = b->E;
    a.W = b->W;
    a.cache = b->cache_blocks;
    a.max_blocks = b->max_blocks;
    a.max_conv = b->max_conv;
    a.max_inflight = b->max_inflight;
    a.max_rps = b->max_routes_per_step;
    a.max_ctrl_window = b->max_ctrl_window;
    a.probe_mode = b->probe_mode;
    a.tiers = b->tiers;
    a.max_routes = b->max_routes;
    a.n_slots = n_slots;
    a.flags = b->flags;
    a.params = b->params;
    a.turn_off = b->turn_off;
    a.turn_blocks = b->turn_blocks;
    a.chain_off = b->chain_off;
    a.chains = b->chains;
    a.route_rand = b->route_rand;
    a.regime = b->regime;
    a.out = *out;
    a.ws = (unsigned char*)workspace;
    a.L = L;
    a.status = st;
    // LDS: worker state, in-flight routes, controller window, then the batch arrays of the largest
    // batch that fits in 76 KiB (two episodes can then share a CU)
    size_t o = 0;
    a.lds_w = 0;
    o = align_up(o + (size_t)b->W * 11 * 4, 16);
    a.lds_inflight = (uint32_t)o;
    o = align_up(o + (size_t)b->max_inflight * 4 * 4, 16);
    a.lds_u = (uint32_t)o;
    o = align_up(o + (size_t)b->max_ctrl_window * 8, 16);
    a.lds_roff = (uint32_t)o;
    o = align_up(o + (size_t)kEpisodeThreads * 4, 16);
    a.lds_batch = (uint32_t)o;
    const size_t limit = 76 * 1024;
    int32_t NB = kMaxBatch;
    const bool tiers = b->tiers != 0;
    while (NB > 1 && o + batch_layout(NB, b->W, tiers).bytes > limit) NB /= 2;
    if (o + batch_layout(NB, b->W, tiers).bytes > limit)
        return fail(RK_EUNSUPPORTED, "rk_simulate_episodes: %zu bytes of LDS per episode exceed 76 KiB",
                    o + (size_t)batch_layout(NB, b->W, tiers).bytes);
    a.NB = NB;
    const size_t lds = o + batch_layout(NB, b->W, tiers).bytes;
    hipStream_t s = (hipStream_t)stream;
    if (n_slots < b->E) {
        hipLaunchKernelGGL(episode_queue_init, dim3(1), dim3(64), 0, s,
                           (int32_t*)((unsigned char*)workspace + L.off_ctl));
        rc = hip_check(hipGetLastError(), "rk_simulate_episodes queue init");
        if (rc) return rc;
    }
    if (n_slots < b->E) hipLaunchKernelGGL(episode_kernel<true>, dim3((unsigned)n_slots), dim3(NT), lds, s, a);
    else hipLaunchKernelGGL(episode_kernel<false>, dim3((unsigned)n_slots), dim3(NT), lds, s, a);
    return hip_check(hipGetLastError(), "rk_simulate_episodes launch");
}
