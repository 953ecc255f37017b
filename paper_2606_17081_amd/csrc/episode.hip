// episode.hip -- independent sequential routing episodes, one workgroup each.
//
// Per episode the workgroup (256 threads, 4 wavefronts) keeps in LDS the
// worker loads A_j, the LRU bookkeeping of every worker, the in-flight routes
// of the last H steps, the controller's load window and the current and next
// prompt chains.  Each worker's cached blocks live in HBM as an
// open-addressing table of 16-byte slots (key, stamp) plus a ring log of
// touches:
//   - a touch of a block at stamp p writes slot.stamp = p and log[p] = slot,
//     so stamps are log positions and recency order is log order;
//   - a log record p is live iff the stamp of slot log[p] still equals p;
//     eviction pops the log head, skipping stale records, and tombstones the
//     slot (stamp kTomb);
//   - when tombstones or the log fill up, the live records are compacted,
//     re-stamped in order and re-inserted into a cleared table.
// A route: every wavefront finds the longest cached prefix of the chain on
// its workers (all of its workers' probes in flight together; a round probes
// 64 spread positions, the next round the sub-interval holding the first
// miss); wavefront 0 turns the overlaps into fp32 costs and takes the min of
// packed (cost, worker) keys; all threads touch/insert the chosen worker's P
// blocks in parallel (stamps in reverse block order) and evict the oldest live
// records.  The next route's chain is loaded into registers while the current
// route runs.
#include <hip/hip_runtime.h>

#include "rk_internal.h"

namespace rk {

constexpr int NT = 256;
constexpr int NW = NT / 64;
constexpr int PF = 8;      // chain blocks per thread prefetched for the next route

struct EpArgs {
    int32_t E, W, cache, max_blocks, max_conv, max_inflight, max_rps, max_ctrl_window, probe_mode, prefetch;
    const rk_episode_params* params;
    const int64_t* turn_off;
    const int32_t* turn_blocks;
    const int64_t* chain_off;
    const uint64_t* chains;
    rk_episode_outputs out;
    unsigned char* ws;
    EpisodeLayout L;
    int32_t* status;
    uint32_t lds_chain0, lds_chain1, lds_w, lds_key, lds_inflight, lds_step, lds_u;
};

struct EpShared {
    int32_t n_route, done, sigma, P, rebuild, ins, remaining, ev, qhead, qsize, pop_base, lcp;
    uint32_t new_head;
    float w_eff;
    int64_t cbase;
    unsigned long long digest;
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

__device__ __forceinline__ void load_slot(const Slot* p, uint64_t& key, uint32_t& stamp)
{
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    key = (uint64_t)v.x | ((uint64_t)v.y << 32);
    stamp = v.z;
}

constexpr int kWin = 4;    // slots read by one lookup (a run of this length is rare at load <= 0.5)

// Membership test finishing a walk whose first kWin slots (from s) are loaded.
__device__ __forceinline__ bool finish_lookup(const Slot* t, uint64_t smask, uint64_t h, uint64_t s,
                                              const uint64_t* k, const uint32_t* st)
{
#pragma unroll
    for (int i = 0; i < kWin; ++i) {
        if (k[i] == kEmpty) return false;
        if (k[i] == h && st[i] != kTomb) return true;
    }
    s = (s + kWin) & smask;
    for (uint64_t n = kWin; n <= smask; ++n) {
        uint64_t kk;
        uint32_t ss;
        load_slot(t + s, kk, ss);
        if (kk == kEmpty) return false;
        if (kk == h && ss != kTomb) return true;
        s = (s + 1) & smask;
    }
    return false;
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
                sh0[jj] = hk[jj] & smask;
#pragma unroll
                for (int i = 0; i < kWin; ++i) load_slot(t + ((sh0[jj] + i) & smask), kw[jj][i], sw[jj][i]);
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

// Find the live slot of h, or claim an empty slot for it.  Concurrent callers
// insert distinct keys; a failed claim moves on along the probe sequence.
__device__ __forceinline__ uint64_t insert_or_touch(Slot* __restrict__ t, uint64_t smask, uint64_t h, int& inserted,
                                                   int32_t* status)
{
    inserted = 0;
    uint64_t s = h & smask;
    for (uint64_t n = 0; n <= smask; ++n) {
        const uint64_t k = __hip_atomic_load(&t[s].key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        const uint32_t st = t[s].stamp;
        if (k == h) {
            if (st != kTomb) return s;
        } else if (k == kEmpty) {
            uint64_t prev = kEmpty;
            if (__hip_atomic_compare_exchange_strong(&t[s].key, &prev, h, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_WORKGROUP)) {
                inserted = 1;
                return s;
            }
            if (prev == h) return s;
        }
        s = (s + 1) & smask;
    }
    atomicOr(status, RK_DEV_TABLE_FULL);
    return ~0ull;
}

// Same result as insert_or_touch, in one memory round trip in the usual
// case.  A block the overlap search found cached is looked up in a window of
// kWin slots.  For a block past the overlap, the claim of its home slot is
// issued together with the loads of the next kWin-1 slots: slots never return
// to empty between compactions, so an empty home slot proves the key absent,
// and an occupied one usually leaves a free slot in the window.  Anything else
// falls back to the full walk.
__device__ __forceinline__ uint64_t touch_hinted(Slot* __restrict__ t, uint64_t smask, uint64_t h, bool cached_hint,
                                                 int& inserted, int32_t* status)
{
    const uint64_t s = h & smask;
    inserted = 0;
    uint64_t k[kWin];
    uint32_t st[kWin];
    if (cached_hint) {
#pragma unroll
        for (int i = 0; i < kWin; ++i) load_slot(t + ((s + i) & smask), k[i], st[i]);
#pragma unroll
        for (int i = 0; i < kWin; ++i)
            if (k[i] == h && st[i] != kTomb) return (s + i) & smask;
    } else {
        uint64_t prev = kEmpty;
        const bool won = __hip_atomic_compare_exchange_strong(&t[s].key, &prev, h, __ATOMIC_RELAXED,
                                                              __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
#pragma unroll
        for (int i = 1; i < kWin; ++i) load_slot(t + ((s + i) & smask), k[i], st[i]);
        if (won) {
            inserted = 1;
            return s;
        }
        if (prev != h) {           // home holds another key: look further in the window
#pragma unroll
            for (int i = 1; i < kWin; ++i) {
                const uint64_t si = (s + i) & smask;
                if (k[i] == h) {
                    if (st[i] != kTomb) return si;
                    continue;
                }
                if (k[i] != kEmpty) continue;
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

template <int JPW>
__global__ __launch_bounds__(NT) void episode_kernel(EpArgs a)
{
    constexpr bool kPipe = JPW <= 4;      // two wavefronts then search up to 8 workers each
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ EpShared sh;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int e = blockIdx.x;
    const rk_episode_params prm = a.params[e];
    const int32_t W = a.W;

    uint64_t* s_cur = (uint64_t*)(smem + a.lds_chain0);     // chain of the current route
    uint64_t* s_nxt = (uint64_t*)(smem + a.lds_chain1);     // chain of the next route (prefetched)
    int32_t* s_A = (int32_t*)(smem + a.lds_w);
    uint32_t* s_head = (uint32_t*)(s_A + W);
    uint32_t* s_tail = s_head + W;
    int32_t* s_live = (int32_t*)(s_tail + W);
    int32_t* s_used = s_live + W;
    int32_t* s_ovc = s_used + W;                          // overlaps of the current route
    int32_t* s_ovn = s_ovc + W;                            // overlaps of the next route (lookahead)
    uint64_t* s_key = (uint64_t*)(smem + a.lds_key);       // packed (cost, worker) per worker
    int32_t* s_stw = (int32_t*)(smem + a.lds_inflight);   // in-flight routes: worker
    int32_t* s_stP = s_stw + a.max_inflight;               //                   prompt blocks
    int32_t* s_stc = s_stP + a.max_inflight;               //                   conversation
    int32_t* s_stepn = s_stc + a.max_inflight;             // routes per step slot
    int64_t* s_stcb = (int64_t*)(smem + a.lds_step);       // this step: chain base
    int32_t* s_stt = (int32_t*)(s_stcb + a.max_rps);       //            global turn
    int64_t* s_u = (int64_t*)(smem + a.lds_u);             // controller load samples

    const int32_t H = prm.hold_steps, rps = prm.routes_per_step, n_conv = prm.n_conv;
    const bool bad = H < 1 || rps < 1 || rps > a.max_rps || (int64_t)H * rps > a.max_inflight ||
                     n_conv < 0 || n_conv > a.max_conv || prm.cap_blocks < 1 ||
                     (prm.controller && (prm.ctrl_window < 1 || prm.ctrl_window > a.max_ctrl_window ||
                                         prm.ctrl_den < 1 || prm.ctrl_num < 0));
    if (bad) {
        if (tid == 0) atomicOr(a.status, RK_DEV_TOO_LARGE);
        return;
    }
    const int64_t gc0 = prm.conv_begin;

    unsigned char* ws = a.ws + (size_t)e * a.L.per_episode;
    Slot* g_slots = (Slot*)(ws + a.L.off_slots);
    uint32_t* g_log = (uint32_t*)(ws + a.L.off_log);
    uint64_t* g_scratch = (uint64_t*)(ws + a.L.off_scratch);
    int32_t* g_queue = (int32_t*)(ws + a.L.off_queue);
    int32_t* g_next = (int32_t*)(ws + a.L.off_next);
    const uint64_t S = a.L.slots, smask = S - 1, R = a.L.ring, rmask = R - 1;
    const uint64_t used_limit = S - S / 4;
    const uint64_t scratch_cap = (uint64_t)a.cache + (uint64_t)a.max_blocks;

    // ---- initial state: empty caches, idle workers, every first turn queued
    {
        uint4* z = reinterpret_cast<uint4*>(g_slots);
        const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
        for (uint64_t i = tid; i < (uint64_t)W * S; i += NT) z[i] = zero;
    }
    if (tid < W) {
        s_A[tid] = 0;
        s_head[tid] = 0;
        s_tail[tid] = 0;
        s_live[tid] = 0;
        s_used[tid] = 0;
    }
    for (int32_t i = tid; i < a.max_inflight; i += NT) s_stepn[i] = 0;
    int32_t qn = 0;
    for (int32_t base = 0; base < n_conv; base += NT) {
        const int32_t c = base + tid;
        bool has = false;
        if (c < n_conv) {
            g_next[c] = 0;
            has = a.turn_off[gc0 + c + 1] > a.turn_off[gc0 + c];
        }
        int32_t total;
        const int32_t rank = block_scan(has, sh.wtot, total);
        if (has) g_queue[qn + rank] = c;
        qn += total;
    }
    if (tid == 0) {
        sh.qhead = 0;
        sh.qsize = qn;
        sh.ins = 0;
        sh.digest = 0;
    }
    __syncthreads();

    const int32_t qcap = n_conv + 1;
    int32_t t = 0;                                 // routes done (uniform)
    int64_t tot[8] = {0, 0, 0, 0, 0, 0, 0, 0};     // thread 0
    int64_t u_sum = 0;                             // thread 0
    bool prev_active = false;                      // thread 0

    // thread 0: prompt, chain base and effective overlap weight of route r of the step
    auto setup = [&](int32_t sbase, int32_t r) {
        bool active = false;
        if (prm.controller && t >= prm.ctrl_window)
            active = (int64_t)prm.ctrl_den * u_sum >
                     (int64_t)prm.ctrl_num * prm.ctrl_window * W * (int64_t)prm.cap_blocks;
        float w = prm.w_ov;
        if (active) {
            w = fminf(prm.w_ov, prm.ctrl_w_ov);
            tot[3] += 1;
            if (!prev_active) tot[4] += 1;
        }
        prev_active = active;
        sh.w_eff = w;
        sh.P = s_stP[sbase + r];
        sh.cbase = s_stcb[r];
    };

    for (int32_t s = 0;; ++s) {
        const int32_t slot = s % H;
        const int32_t sb = slot * rps;
        // ---- release the routes of step s - H; queue their conversations' next turns
        if (s >= H) {
            const int32_t nprev = s_stepn[slot];
            const int32_t qend = sh.qhead + sh.qsize;
            int32_t pushed = 0;
            for (int32_t base = 0; base < nprev; base += NT) {
                const int32_t r = base + tid;
                bool more = false;
                int32_t c = 0;
                if (r < nprev) {
                    c = s_stc[sb + r];
                    atomicSub(&s_A[s_stw[sb + r]], s_stP[sb + r]);
                    more = g_next[c] < (int32_t)(a.turn_off[gc0 + c + 1] - a.turn_off[gc0 + c]);
                }
                int32_t total;
                const int32_t rank = block_scan(more, sh.wtot, total);
                if (more) g_queue[(qend + pushed + rank) % qcap] = c;
                pushed += total;
            }
            if (tid == 0 && pushed) sh.qsize += pushed;
            __syncthreads();
        }
        // ---- how many requests this step routes
        if (tid == 0) {
            int64_t inflight = 0;
            for (int32_t k = 1; k < H && k <= s; ++k) inflight += s_stepn[(s - k) % H];
            sh.done = sh.qsize == 0 && inflight == 0;
            sh.n_route = sh.done ? 0 : min(rps, sh.qsize);
            s_stepn[slot] = sh.n_route;
            if (sh.n_route > 0) tot[5] = s + 1;
            sh.pop_base = sh.qhead;
            sh.qhead = (sh.qhead + sh.n_route) % qcap;
            sh.qsize -= sh.n_route;
        }
        __syncthreads();
        if (sh.done) break;
        const int32_t n = sh.n_route;
        // ---- pop the step's requests from the queue head (in parallel)
        for (int32_t r = tid; r < n; r += NT) {
            const int32_t c = g_queue[(sh.pop_base + r) % qcap];
            const int32_t k = g_next[c];
            g_next[c] = k + 1;
            const int64_t g = gc0 + c;
            const int64_t turn = a.turn_off[g] + k;
            int32_t P = a.turn_blocks[turn];
            const int64_t cb = a.chain_off[g], ce = a.chain_off[g + 1];
            if (P < 0 || (int64_t)P > ce - cb) {
                atomicOr(a.status, RK_DEV_SHORT_INPUT);
                P = P < 0 ? 0 : (int32_t)max((int64_t)0, ce - cb);
            }
            if (P > a.max_blocks) {
                atomicOr(a.status, RK_DEV_TOO_LARGE);
                P = a.max_blocks;
            }
            s_stc[sb + r] = c;
            s_stP[sb + r] = P;
            s_stt[r] = (int32_t)turn;
            s_stcb[r] = cb;
        }
        __syncthreads();
        if (tid == 0 && n > 0) setup(sb, 0);
        __syncthreads();
        // Pipelining: while worker sigma_r absorbs route r's blocks, waves 2-3
        // already search route r+1's cached prefixes.  Workers other than
        // sigma_r are unchanged by route r.  On sigma_r, route r+1's blocks
        // shared with route r's chain (their common prefix) are cached after
        // the update, and its later blocks are chained hashes route r cannot
        // insert, so a search over those positions only is exact while the
        // update runs.  Evictions by route r are corrected by a new search.
        const bool can_pipe = kPipe && a.probe_mode == RK_PROBE_PREFIX;
        bool nxt_ready = false;    // s_nxt holds route r+1's chain (uniform)
        bool have_ov = false;      // s_ovc holds route r's overlaps (uniform)
        {
            const uint64_t* gch = a.chains + sh.cbase;
            for (int32_t k = tid; k < sh.P; k += NT) s_cur[k] = gch[k];
            __syncthreads();
        }

        for (int32_t r = 0; r < n; ++r) {
            const int32_t P = sh.P;
            const int32_t Pn = r + 1 < n ? s_stP[sb + r + 1] : 0;
            uint64_t last_h = 0;    // thread 0: h_{P-1} of route r
            if (r + 1 < n && !nxt_ready) {
                const uint64_t* gch = a.chains + s_stcb[r + 1];
                for (int32_t k = tid; k < Pn; k += NT) s_nxt[k] = gch[k];
            }
            // ---- prefetch the chain of route r+2 into registers
            uint64_t pf[PF];
            int32_t P2 = 0;
            bool prefetch = false;
            if (a.prefetch && r + 2 < n) {
                P2 = s_stP[sb + r + 2];
                prefetch = P2 <= NT * PF;
                if (prefetch) {
                    const uint64_t* gch = a.chains + s_stcb[r + 2];
#pragma unroll
                    for (int i = 0; i < PF; ++i) {
                        const int32_t k = tid + i * NT;
                        pf[i] = k < P2 ? gch[k] : 0ull;
                    }
                }
            }
            // ---- longest cached prefix of route r on every worker (unless already known)
            if (!have_ov) {
                wave_overlaps<JPW>(s_cur, P, wave, NW, W, g_slots, S, a.probe_mode, s_ovc, -1, 0);
            }
            __syncthreads();
            const bool pipe = can_pipe && r + 1 < n;
            // ---- cost of every worker and argmin (wavefront 0); common prefix with route r+1 (wavefront 1)
            const int64_t row = prm.out_base + (int64_t)t;
            if (wave == 0) {
                if (lane < W) {
                    const float c = route_cost(sh.w_eff, prm.w_act, prm.w_sat, prm.cap_blocks, P, s_ovc[lane],
                                               s_A[lane]);
                    if (a.out.overlap) a.out.overlap[row * W + lane] = s_ovc[lane];
                    if (a.out.cost) a.out.cost[row * W + lane] = c;
                    s_key[lane] = argmin_key(c, lane);
                }
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
                if (lane == 0) {
                    uint64_t key = s_key[0];
                    for (int32_t j = 1; j < W; ++j) {
                        const uint64_t kj = s_key[j];
                        key = kj < key ? kj : key;
                    }
                    const int32_t sg = (int32_t)(uint32_t)(key & 0xffffffffu);
                    sh.sigma = sg;
                    last_h = P > 0 ? s_cur[P - 1] : 0ull;   // read before the buffer is reused
                    const uint64_t ins_max = (uint64_t)(P - s_ovc[sg]);
                    sh.rebuild = ((uint64_t)s_used[sg] + ins_max > used_limit) ||
                                 ((uint64_t)(s_tail[sg] - s_head[sg]) + (uint64_t)P > R) ||
                                 (s_tail[sg] > 0x40000000u);
                }
            } else if (wave == 1 && pipe) {
                const int32_t m = min(P, Pn);
                int32_t l = m;
                for (int32_t base = 0; base < m; base += 64) {
                    const int32_t k = base + lane;
                    const unsigned long long d = __ballot(k < m && s_cur[k] != s_nxt[k]);
                    if (d) {
                        l = base + __ffsll(d) - 1;
                        break;
                    }
                }
                if (lane == 0) sh.lcp = l;
            }
            __syncthreads();
            const int32_t sg = sh.sigma;
            Slot* tk = g_slots + (uint64_t)sg * S;
            uint32_t* tl = g_log + (uint64_t)sg * R;

            // ---- compaction: re-stamp the live records in order into a cleared table
            if (sh.rebuild) {
                const uint32_t head = s_head[sg], tail = s_tail[sg];
                int32_t cnt = 0;
                for (uint32_t base = head; base < tail; base += NT) {
                    const uint32_t pos = base + (uint32_t)tid;
                    bool live = false;
                    uint64_t key = 0;
                    if (pos < tail) {
                        const uint32_t sl = tl[pos & rmask];
                        if (sl < S) {
                            uint32_t st;
                            load_slot(tk + sl, key, st);
                            live = st == pos;
                        }
                    }
                    int32_t total;
                    const int32_t rank = block_scan(live, sh.wtot, total);
                    if (live && (uint64_t)(cnt + rank) < scratch_cap) g_scratch[cnt + rank] = key;
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
                    if (sl != ~0ull) tk[sl].stamp = (uint32_t)q;
                    tl[(uint32_t)q & rmask] = (uint32_t)sl;
                }
                __syncthreads();
                if (tid == 0) {
                    s_head[sg] = 0;
                    s_tail[sg] = (uint32_t)cnt;
                    s_live[sg] = cnt;
                    s_used[sg] = cnt;
                }
                __syncthreads();
            }

            // ---- touch route r's blocks (block k gets stamp tail + P-1-k), inserting misses;
            //      with pipelining, waves 2-3 meanwhile search route r+1's overlaps
            {
                const int32_t nupd = pipe ? NT / 2 : NT;
                if (tid < nupd) {
                    const uint32_t tail = s_tail[sg];
                    const int32_t o_sg = s_ovc[sg];
                    int my_ins = 0;
                    for (int32_t k = tid; k < P; k += nupd) {
                        int ins;
                        const uint32_t stamp = tail + (uint32_t)(P - 1 - k);
                        const uint64_t sl = touch_hinted(tk, smask, s_cur[k], k < o_sg, ins, a.status);
                        if (sl != ~0ull) tk[sl].stamp = stamp;
                        tl[stamp & rmask] = (uint32_t)sl;    // a failed insert logs an out-of-range slot
                        my_ins += ins;
                    }
                    if (my_ins) atomicAdd(&sh.ins, my_ins);
                } else if constexpr (kPipe) {
                    wave_overlaps<2 * JPW>(s_nxt, Pn, wave - NW / 2, NW / 2, W, g_slots, S, RK_PROBE_PREFIX, s_ovn,
                                           sg, sh.lcp);
                }
            }
            __syncthreads();
            if (tid == 0) {
                s_tail[sg] += (uint32_t)P;
                s_live[sg] += sh.ins;
                s_used[sg] += sh.ins;
                sh.remaining = max(0, s_live[sg] - a.cache);
                sh.ins = 0;
                sh.ev = 0;
                sh.digest = 0ull;
            }
            __syncthreads();
            // ---- evict least recently used blocks down to the capacity
            while (sh.remaining > 0) {
                const uint32_t head = s_head[sg], tail = s_tail[sg];
                const int32_t rem = sh.remaining;
                if (head >= tail) {
                    if (tid == 0) atomicOr(a.status, RK_DEV_TABLE_FULL);
                    break;
                }
                const uint32_t pos = head + (uint32_t)tid;
                uint32_t sl = 0;
                bool live = false;
                uint64_t key = 0;
                if (pos < tail) {
                    sl = tl[pos & rmask];
                    if (sl < S) {
                        uint32_t st;
                        load_slot(tk + sl, key, st);
                        live = st == pos;
                    }
                }
                int32_t total;
                const int32_t rank = block_scan(live, sh.wtot, total);
                if (live && rank < rem) {
                    tk[sl].stamp = kTomb;
                    atomicAdd(&sh.digest, (unsigned long long)mix64(key));
                    if (rank == rem - 1) sh.new_head = pos + 1;
                }
                __syncthreads();
                if (tid == 0) {
                    if (total >= rem) {
                        s_head[sg] = sh.new_head;
                        sh.ev += rem;
                        s_live[sg] -= rem;
                        sh.remaining = 0;
                    } else {
                        s_head[sg] = min(head + (uint32_t)NT, tail);
                        sh.ev += total;
                        s_live[sg] -= total;
                        sh.remaining = rem - total;
                    }
                }
                __syncthreads();
            }
            // ---- the lookahead search of sigma_r is void if route r evicted: search again
            if (pipe && sh.ev > 0) {
                if (wave == 0)
                    wave_overlaps<1>(s_nxt, Pn, sg, 1, sg + 1, g_slots, S, RK_PROBE_PREFIX, s_ovn, -1, 0);
                __syncthreads();
            }
            // ---- load, controller sample, outputs; set up the next route
            if (tid == 0) {
                s_A[sg] += P;
                s_stw[sb + r] = sg;
                if (prm.controller) {
                    int64_t u = 0;
                    for (int32_t j = 0; j < W; ++j) u += s_A[j];
                    const int32_t pos = t % prm.ctrl_window;
                    if (t >= prm.ctrl_window) u_sum -= s_u[pos];
                    s_u[pos] = u;
                    u_sum += u;
                }
                if (a.out.route_turn) a.out.route_turn[row] = s_stt[r];
                if (a.out.route_worker) a.out.route_worker[row] = sg;
                if (a.out.route_step) a.out.route_step[row] = (int32_t)s;
                if (a.out.route_blocks) a.out.route_blocks[row] = P;
                if (a.out.evict_count) a.out.evict_count[row] = sh.ev;
                if (a.out.evict_digest) a.out.evict_digest[row] = sh.digest;
                if (a.out.last_hash) a.out.last_hash[row] = last_h;
                tot[0] += P - s_ovc[sg];
                tot[1] += sh.ev;
                tot[2] += P;
                tot[6] += s_ovc[sg];
                ++t;
                if (r + 1 < n) setup(sb, r + 1);
            } else {
                ++t;
            }
            // route r's chain buffer now takes route r+2's chain; rotate the buffers
            if (prefetch) {
#pragma unroll
                for (int i = 0; i < PF; ++i) {
                    const int32_t k = tid + i * NT;
                    if (k < P2) s_cur[k] = pf[i];
                }
            }
            {
                uint64_t* x = s_cur;
                s_cur = s_nxt;
                s_nxt = x;
                int32_t* y = s_ovc;
                s_ovc = s_ovn;
                s_ovn = y;
            }
            nxt_ready = prefetch;
            have_ov = pipe;
            __syncthreads();
        }
    }
    if (tid == 0 && a.out.totals) {
        int64_t cachedsum = 0;
        for (int32_t j = 0; j < W; ++j) cachedsum += s_live[j];
        tot[7] = cachedsum;
        for (int k = 0; k < 8; ++k) a.out.totals[(int64_t)e * 8 + k] = tot[k];
    }
}

}  // namespace rk

using namespace rk;

extern "C" size_t rk_simulate_workspace_size(int32_t E, int32_t W, int32_t cache_blocks, int32_t max_blocks,
                                             int32_t max_conv)
{
    if (E < 0 || W < 1 || cache_blocks < 1 || max_blocks < 1 || max_conv < 0) return 0;
    const EpisodeLayout L = episode_layout(W, cache_blocks, max_blocks, max_conv);
    return L.per_episode * (size_t)E;
}

extern "C" int rk_simulate_episodes(const rk_episode_batch* b, const rk_episode_outputs* out, void* workspace,
                                    size_t ws_bytes, void* stream)
{
    if (!b || !out) return fail(RK_EINVAL, "rk_simulate_episodes: NULL batch or outputs");
    if (b->E < 0) return fail(RK_EINVAL, "rk_simulate_episodes: E < 0");
    if (b->W < 1 || b->W > 64) return fail(RK_EUNSUPPORTED, "rk_simulate_episodes: W outside 1..64");
    if (b->cache_blocks < 1) return fail(RK_EINVAL, "rk_simulate_episodes: cache_blocks < 1");
    if (b->max_blocks < 1 || b->max_blocks > 8192)
        return fail(RK_EUNSUPPORTED, "rk_simulate_episodes: max_blocks outside 1..8192");
    if (b->max_conv < 0 || b->max_conv > (1 << 28)) return fail(RK_EINVAL, "rk_simulate_episodes: max_conv");
    if (b->max_inflight < 1 || b->max_inflight > 8192)
        return fail(RK_EUNSUPPORTED, "rk_simulate_episodes: max_inflight outside 1..8192");
    if (b->max_routes_per_step < 1 || b->max_routes_per_step > b->max_inflight)
        return fail(RK_EINVAL, "rk_simulate_episodes: max_routes_per_step outside 1..max_inflight");
    if (b->max_ctrl_window < 1 || b->max_ctrl_window > 4096)
        return fail(RK_EUNSUPPORTED, "rk_simulate_episodes: max_ctrl_window outside 1..4096");
    if (b->probe_mode != RK_PROBE_PREFIX && b->probe_mode != RK_PROBE_SCAN)
        return fail(RK_EINVAL, "rk_simulate_episodes: unknown probe_mode");
    if ((int64_t)b->cache_blocks + b->max_blocks > (1ll << 29))
        return fail(RK_EUNSUPPORTED, "rk_simulate_episodes: cache too large");
    if (b->E == 0) return RK_OK;
    if (!b->params || !b->turn_off || !b->turn_blocks || !b->chain_off || !b->chains || !workspace)
        return fail(RK_EINVAL, "rk_simulate_episodes: NULL array");
    const EpisodeLayout L = episode_layout(b->W, b->cache_blocks, b->max_blocks, b->max_conv);
    const size_t need = L.per_episode * (size_t)b->E;
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
    a.params = b->params;
    a.turn_off = b->turn_off;
    a.turn_blocks = b->turn_blocks;
    a.chain_off = b->chain_off;
    a.chains = b->chains;
    a.out = *out;
    a.ws = (unsigned char*)workspace;
    a.L = L;
    a.status = st;
    const size_t chain_bytes = align_up((size_t)b->max_blocks * 8, 16);
    size_t rest = 0;
    rest = align_up(rest + (size_t)b->W * 7 * 4, 16);
    const size_t off_key = rest;
    rest = align_up(rest + (size_t)b->W * 8, 16);
    const size_t off_inflight = rest;
    rest = align_up(rest + (size_t)b->max_inflight * 4 * 4, 16);
    const size_t off_step = rest;
    rest = align_up(rest + (size_t)b->max_routes_per_step * 12, 16);
    const size_t off_u = rest;
    rest = align_up(rest + (size_t)b->max_ctrl_window * 8, 16);
    const size_t limit = 60 * 1024;
    a.prefetch = 2 * chain_bytes + rest <= limit;
    const size_t chains_total = (a.prefetch ? 2 : 1) * chain_bytes;
    if (chains_total + rest > limit)
        return fail(RK_EUNSUPPORTED, "rk_simulate_episodes: %zu bytes of LDS per episode exceed 60 KiB",
                    chains_total + rest);
    a.lds_chain0 = 0;
    a.lds_chain1 = a.prefetch ? (uint32_t)chain_bytes : 0;
    a.lds_w = (uint32_t)chains_total;
    a.lds_key = (uint32_t)(chains_total + off_key);
    a.lds_inflight = (uint32_t)(chains_total + off_inflight);
    a.lds_step = (uint32_t)(chains_total + off_step);
    a.lds_u = (uint32_t)(chains_total + off_u);
    const size_t lds = chains_total + rest;
    const int jpw = (b->W + NW - 1) / NW;
    hipStream_t s = (hipStream_t)stream;
    if (jpw <= 1) hipLaunchKernelGGL(episode_kernel<1>, dim3((unsigned)b->E), dim3(NT), lds, s, a);
    else if (jpw <= 2) hipLaunchKernelGGL(episode_kernel<2>, dim3((unsigned)b->E), dim3(NT), lds, s, a);
    else if (jpw <= 4) hipLaunchKernelGGL(episode_kernel<4>, dim3((unsigned)b->E), dim3(NT), lds, s, a);
    else if (jpw <= 8) hipLaunchKernelGGL(episode_kernel<8>, dim3((unsigned)b->E), dim3(NT), lds, s, a);
    else hipLaunchKernelGGL(episode_kernel<16>, dim3((unsigned)b->E), dim3(NT), lds, s, a);
    return hip_check(hipGetLastError(), "rk_simulate_episodes launch");
}
