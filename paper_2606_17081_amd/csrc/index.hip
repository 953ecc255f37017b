// index.hip -- the router's global block index (block hash -> set of workers
// caching that block) and batched routing-cost evaluation against it.
//
// The router the paper studies answers "which workers hold this prefix" from
// one index over all workers (the global radix tree of the Smart Router in the
// Dynamo architecture background section, queried by best_worker in
// Alg. adaptive-router).  Chained block hashes name prefixes uniquely, so the radix tree
// becomes one open-addressing table of 16-byte slots (key, worker mask) and a
// single probe answers membership on all W <= 64 workers at once.  Scoring a
// request then costs a few lane-parallel probe rounds per request instead of
// a search per (request, worker) pair:
//   - PREFIX mode (every worker's set is prefix-closed along the chains):
//     worker masks along a chain only lose bits.  A coarse round (16
//     samples) bounds the region [0, U) where any worker may still hold the
//     chain, a second round samples it with 64 lanes (every position when
//     U <= 64), and a third probes the inside of the sample intervals where
//     some worker's bit disappears.  Worker j's overlap is the first
//     position whose mask lacks bit j.
//   - SCAN mode (any sets): positions from block 0 in rounds of 64; a
//     running AND of the masks gives each worker's first miss exactly, and
//     the scan stops once no worker is left.
// One wavefront scores two consecutive requests; lane j owns worker j's
// overlap and cost.
#include <hip/hip_runtime.h>

#include "rk_internal.h"

namespace rk {

struct __align__(16) IndexSlot {
    uint64_t key;
    uint64_t mask;
};

__device__ __forceinline__ void load_slot(const IndexSlot* t, uint64_t s, uint64_t& k, uint64_t& m)
{
    const uint4 v = *reinterpret_cast<const uint4*>(t + s);
    k = (uint64_t)v.x | ((uint64_t)v.y << 32);
    m = (uint64_t)v.z | ((uint64_t)v.w << 32);
}

// Worker mask of block hash h (0 when no worker holds it): linear probing
// one 16-byte slot per access from the home slot h & smask.  At the loads the
// index is sized for, the home slot settles almost every lookup, and one slot
// costs the smallest read the memory system serves; wider windows (an aligned
// 32- or 64-byte group per access) moved more bytes per lookup and ran slower.
__device__ __forceinline__ uint64_t index_lookup(const IndexSlot* __restrict__ t, uint64_t smask, uint64_t h)
{
    uint64_t s = h & smask;
    for (uint64_t n = 0; n <= smask; ++n) {
        uint64_t k, m;
        load_slot(t, s, k, m);
        if (k == h) return m;
        if (k == kEmpty) return 0ull;
        s = (s + 1) & smask;
    }
    return 0ull;
}

// First index in [lo, hi) whose mask lacks bit j, for masks in which bit j
// never comes back once cleared; hi if none.
__device__ __forceinline__ int32_t first_clear(const uint64_t* m, int32_t lo, int32_t hi, int32_t j)
{
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        if ((m[mid] >> j) & 1ull) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

__device__ __forceinline__ uint32_t next_pow2_dev(uint32_t x)
{
    return x <= 1u ? 1u : 1u << (32 - __clz((int)(x - 1u)));
}

// LDS writes of one wavefront made visible to the other lanes of that wavefront.
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

constexpr int kRPW = 2;           // requests per wavefront: their offsets and chains are loaded together
constexpr int kRound1Min = 64;    // chains longer than this get the coarse first round
constexpr int kStage = 256;       // leading chain blocks staged in LDS, read in one coalesced pass
constexpr int kStageRegs = kStage / 64;

struct IdxLds {
    uint64_t ch[kRPW][kStage];   // the first kStage chain hashes of each of the wavefront's requests
    uint64_t m[64];              // masks of the current round (prefix ANDs in rounds 1-2)
    int32_t ioff[65];            // start of each sample interval's positions in the third round
};

constexpr int kFewBounds = 8;     // boundaries handled by a scalar loop; more take the LDS search
constexpr int kDppWaveShr1 = 0x138;   // DPP: every lane takes lane - 1's value (lane 0 keeps old)

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v)
{
    auto mn = [](uint32_t a, uint32_t b) { return b < a ? b : a; };
    v = mn(v, dpp32<kDppQuadSwap1>(v, v));
    v = mn(v, dpp32<kDppQuadSwap2>(v, v));
    v = mn(v, dpp32<kDppRowHalfMirror>(v, v));
    v = mn(v, dpp32<kDppRowMirror>(v, v));
    const auto rl = [&](int l) { return (uint32_t)__builtin_amdgcn_readlane((int)v, l); };
    return mn(mn(rl(0), rl(16)), mn(rl(32), rl(48)));
}

// The router cost (Section 2.2, Eq. router-cost) in the operation order of
// route_cost; when cap is a power of two, (A + P) / cap is the exact product
// with 1 / cap.
__device__ __forceinline__ float index_route_cost(const rk_cost_params& p, float inv_cap, int32_t P, int32_t o,
                                                  int32_t A)
{
    const float t1 = __fmul_rn(p.w_ov, (float)(P - o));
    const float t2 = __fmul_rn(p.w_act, (float)A);
    const float L = (float)((int64_t)A + (int64_t)P);
    const float r = inv_cap != 0.0f ? __fmul_rn(L, inv_cap) : __fdiv_rn(L, (float)p.cap_blocks);
    const float x = fmaxf(__fsub_rn(r, 1.0f), 0.0f);
    const float t3 = __fmul_rn(p.w_sat, __fmul_rn(x, x));
    return __fadd_rn(__fadd_rn(t1, t2), t3);
}

// Position of second-round sample k: every position when the round is exact,
// else the power-of-two grid of step st2, clamped to U - 1.
__device__ __forceinline__ int32_t round2_pos(int32_t k, bool exact, int64_t st2, int32_t U)
{
    return exact ? k : (int32_t)min((int64_t)(k + 1) * st2, (int64_t)U) - 1;
}

// One wavefront scores kRPW consecutive requests; lane j owns worker j.  The
// requests' chain offsets come in one load and their leading chain blocks in
// one coalesced pass into LDS, so only the first request waits for them.
template <int MODE>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(8))) void score_index_kernel(
    int32_t B, int32_t W, const uint64_t* __restrict__ chains, const int64_t* __restrict__ chain_off,
    const IndexSlot* __restrict__ index, int32_t log2_slots, const int32_t* __restrict__ active, rk_cost_params p,
    int32_t* __restrict__ ov_out, float* __restrict__ cost_out, int32_t* __restrict__ am_out, int32_t* status)
{
    __shared__ IdxLds L;
    const int32_t lane = threadIdx.x & 63;
    const uint64_t smask = (1ull << log2_slots) - 1;
    const int32_t A = lane < W ? active[lane] : 0;
    const uint64_t all = W == 64 ? ~0ull : ((1ull << W) - 1ull);
    const float inv_cap = (p.cap_blocks & (p.cap_blocks - 1)) == 0 ? 1.0f / (float)p.cap_blocks : 0.0f;
    const int64_t npairs = ((int64_t)B + kRPW - 1) / kRPW;

    // Workgroups are handed to the 8 XCDs round-robin; renumber them so each
    // XCD walks one contiguous range of requests (gridDim.x is a multiple of 8).
    const uint32_t nb8 = gridDim.x >> 3;
    const uint32_t lb = (blockIdx.x & 7u) * nb8 + (blockIdx.x >> 3);
    for (int64_t g = lb; g < npairs; g += gridDim.x) {
        const int64_t i0 = g * kRPW;
        const int32_t nr = (int32_t)min((int64_t)kRPW, (int64_t)B - i0);
        const int64_t offv = lane <= nr ? chain_off[i0 + lane] : 0;
        int64_t c[kRPW + 1];
#pragma unroll
        for (int r = 0; r <= kRPW; ++r) c[r] = (int64_t)readlane64((uint64_t)offv, r);
        int32_t Pr[kRPW];
#pragma unroll
        for (int r = 0; r < kRPW; ++r) {
            Pr[r] = 0;
            if (r < nr) {
                if (c[r + 1] < c[r] || c[r + 1] - c[r] > 0x7fffffff) {
                    if (lane == 0) atomicOr(status, RK_DEV_BAD_OFFSETS);
                } else {
                    Pr[r] = (int32_t)(c[r + 1] - c[r]);
                }
            }
        }
        wave_sync();   // the previous requests' reads of L.ch are done
        {
            uint64_t v[kRPW][kStageRegs];
#pragma unroll
            for (int r = 0; r < kRPW; ++r) {
                const int32_t n = min(Pr[r], kStage);
                const uint64_t* __restrict__ hg = chains + c[r];
#pragma unroll
                for (int k = 0; k < kStageRegs; ++k) v[r][k] = lane + 64 * k < n ? hg[lane + 64 * k] : 0ull;
            }
#pragma unroll
            for (int r = 0; r < kRPW; ++r)
#pragma unroll
                for (int k = 0; k < kStageRegs; ++k) L.ch[r][lane + 64 * k] = v[r][k];
        }
        wave_sync();

        for (int32_t r = 0; r < nr; ++r) {
            const int64_t i = i0 + r;
            const int32_t P = Pr[r];
            const uint64_t* __restrict__ hg = chains + c[r];
            const uint64_t* ch = L.ch[r];
            auto h = [&](int32_t x) -> uint64_t { return x < kStage ? ch[x] : hg[x]; };
            int32_t o = 0;   // lane j: overlap on worker j

            if (MODE == RK_PROBE_SCAN) {
                uint64_t carry = all;
                bool done = false;
                for (int32_t base = 0; base < P && carry != 0ull; base += 64) {
                    const int32_t n = min(64, P - base);
                    const uint64_t m = lane < n ? index_lookup(index, smask, h(base + lane)) : 0ull;
                    const uint64_t pa = wave_scan_and_u64(m) & carry;
                    L.m[lane] = pa;
                    wave_sync();
                    if (lane < W && !done) {
                        const int32_t f = first_clear(L.m, 0, n, lane);
                        o += f;
                        done = f < n;
                    }
                    carry = readlane64(pa, n - 1);
                    wave_sync();
                }
            } else {
                // ---- round 1: every worker's first miss lies in [0, U).  Sample
                // positions sit on a power-of-two grid (clamped to the chain's end)
                // so requests of one prefix group probe the same index slots.
                // Masks along a chain only lose bits, so the first sample with an
                // empty mask bounds every worker.
                int32_t U = P;
                if (P > kRound1Min) {
                    const int64_t st1 = (int64_t)next_pow2_dev((uint32_t)P) >> 4;
                    const int32_t q1 = (int32_t)min((int64_t)(lane + 1) * st1, (int64_t)P) - 1;
                    const uint64_t m1 = lane < 16 ? index_lookup(index, smask, h(q1)) & all : all;
                    const uint64_t z = __ballot(m1 == 0ull);
                    if (z) U = __builtin_amdgcn_readlane(q1, __ffsll((unsigned long long)z) - 1) + 1;
                }
                // ---- round 2: every position of [0, U) when U <= 64, else 64 samples
                // on the power-of-two grid of step next_pow2(U) / 64, clamped to U - 1.
                // Sample k is a boundary when its mask lacks bits its predecessor's
                // had (all W bits before sample 0); worker j's first missing sample
                // t is the boundary that drops bit j.  A request has few boundaries
                // (one per distinct overlap), so a loop over them costs a few scalar
                // steps; many boundaries fall back to a search per worker in LDS.
                const bool exact = U <= 64;
                const int32_t nq = exact ? U : 64;
                const int64_t st2 = (int64_t)next_pow2_dev((uint32_t)U) >> 6;
                const int32_t q = round2_pos(lane, exact, st2, U);
                const uint64_t m = lane < nq ? index_lookup(index, smask, h(q)) & all : 0ull;
                const uint64_t mp = dpp64<kDppWaveShr1>(all, m);   // sample lane - 1's mask
                const uint64_t bnd = __ballot(lane < nq && mp != m);
                const bool few = __popcll(bnd) <= kFewBounds;
                int32_t t = nq;
                if (few) {
                    for (uint64_t b = bnd; b; b &= b - 1) {
                        const int k = __ffsll((unsigned long long)b) - 1;
                        if ((((readlane64(mp, k) & ~readlane64(m, k)) >> lane) & 1ull)) t = k;
                    }
                } else {
                    L.m[lane] = m;
                    wave_sync();
                    if (lane < W) t = first_clear(L.m, 0, nq, lane);
                    wave_sync();
                }
                if (exact) {
                    o = t;   // t == U only when U == P: every position is cached
                } else {
                    // ---- round 3: worker j's first miss is in (q[t-1], q[t]]; probe the
                    // inside of the boundary intervals, laid out one after another.
                    const int32_t qprev = (int32_t)dpp32<kDppWaveShr1>(0xffffffffu, (uint32_t)q);
                    const bool mine = lane < W && t < 64;
                    o = mine ? round2_pos(t, false, st2, U) : P;
                    int32_t pos = -1, a0 = 0, a1 = 0, pb = 0, nb3 = 0;
                    uint64_t pstart = 0ull;   // the mask before the lane's position when it opens an interval
                    bool opens = false;
                    if (few) {
                        for (uint64_t b = bnd; b; b &= b - 1) {
                            const int k = __ffsll((unsigned long long)b) - 1;
                            const int32_t qk = __builtin_amdgcn_readlane(q, k), qpk = __builtin_amdgcn_readlane(qprev, k);
                            const int32_t w = max(qk - qpk - 1, 0);
                            if (lane >= nb3 && lane < nb3 + w) pos = qpk + 1 + (lane - nb3);
                            if (w > 0 && lane == nb3) {
                                opens = true;
                                pstart = readlane64(mp, k);
                            }
                            if (t == k) {
                                a0 = nb3;
                                a1 = nb3 + w;
                                pb = qpk + 1;
                            }
                            nb3 += w;
                        }
                    }
                    if (few && nb3 <= 64) {
                        const uint64_t mm = pos >= 0 ? index_lookup(index, smask, h(pos)) & all : 0ull;
                        // the shift runs on every lane (a lane whose source lane sat out
                        // would receive the fill value), then the lanes that open an
                        // interval take the mask before it instead
                        const uint64_t left = dpp64<kDppWaveShr1>(all, mm);
                        const uint64_t pv = opens ? pstart : left;
                        const uint64_t b3 = __ballot(pos >= 0 && pv != mm);
                        if (__popcll(b3) <= kFewBounds) {
                            for (uint64_t b = b3; b; b &= b - 1) {
                                const int x = __ffsll((unsigned long long)b) - 1;
                                if ((((readlane64(pv, x) & ~readlane64(mm, x)) >> lane) & 1ull))
                                    o = __builtin_amdgcn_readlane(pos, x);
                            }
                        } else {
                            L.m[lane] = mm;
                            wave_sync();
                            if (mine && a1 > a0) {
                                const int32_t f = first_clear(L.m, a0, a1, lane);
                                if (f < a1) o = pb + (f - a0);
                            }
                            wave_sync();
                        }
                    } else {
                        // many boundaries or more than 64 positions: chunks of 64
                        // positions, each lane finding its interval by binary search
                        const int32_t width = ((bnd >> lane) & 1ull) ? max(q - qprev - 1, 0) : 0;
                        int32_t total;
                        const int32_t off = wave_excl_sum_dpp(width, total);
                        L.ioff[lane] = off;
                        if (lane == 63) L.ioff[64] = total;
                        wave_sync();
                        const int32_t c0 = mine ? L.ioff[t] : 0, c1 = mine ? L.ioff[t + 1] : 0;
                        const int32_t pbase = mine ? (t == 0 ? 0 : round2_pos(t - 1, false, st2, U) + 1) : 0;
                        bool found = !mine;
                        for (int32_t b3 = 0; b3 < total; b3 += 64) {
                            const int32_t idx = b3 + lane;
                            uint64_t mm = 0ull;
                            if (idx < total) {
                                int32_t lo = 0, hi = 63;   // largest k with ioff[k] <= idx
                                while (lo < hi) {
                                    const int32_t mid = (lo + hi + 1) >> 1;
                                    if (L.ioff[mid] <= idx) lo = mid;
                                    else hi = mid - 1;
                                }
                                const int32_t p3 = (lo == 0 ? 0 : round2_pos(lo - 1, false, st2, U) + 1) +
                                                   (idx - L.ioff[lo]);
                                mm = index_lookup(index, smask, h(p3)) & all;
                            }
                            wave_sync();   // the previous chunk's masks have been read
                            L.m[lane] = mm;
                            wave_sync();
                            if (!found) {
                                const int32_t lo = max(c0, b3), hi = min(c1, b3 + 64);
                                if (lo < hi) {
                                    const int32_t x = first_clear(L.m, lo - b3, hi - b3, lane) + b3;
                                    if (x < hi) {
                                        o = pbase + (x - c0);
                                        found = true;
                                    }
                                }
                            }
                        }
                        wave_sync();   // L.m and L.ioff are free for the next request
                    }
                }
            }

            // cost per worker; argmin = the lowest worker among those of minimal
            // cost (non-negative floats order as their bit patterns)
            uint32_t cb = 0xffffffffu;
            if (lane < W) {
                const float cst = index_route_cost(p, inv_cap, P, o, A);
                if (ov_out) ov_out[i * W + lane] = o;
                if (cost_out) cost_out[i * W + lane] = cst;
                cb = __float_as_uint(__fadd_rn(cst, 0.0f));
            }
            const uint32_t cmin = wave_min_u32(cb);
            const uint64_t win = __ballot(lane < W && cb == cmin);
            if (lane == 0 && am_out) am_out[i] = __ffsll((unsigned long long)win) - 1;
        }
    }
}

__global__ __launch_bounds__(256) void index_clear_kernel(IndexSlot* __restrict__ t, uint64_t n)
{
    const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (uint64_t)gridDim.x * blockDim.x)
        *reinterpret_cast<uint4*>(t + i) = zero;
}

__global__ __launch_bounds__(256) void index_insert_kernel(const uint64_t* __restrict__ keys, int64_t n, int32_t j,
                                                           IndexSlot* __restrict__ t, uint64_t smask, int32_t* status)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const uint64_t key = keys[i];
        if (key == kEmpty) {
            atomicOr(status, RK_DEV_ZERO_KEY);
            continue;
        }
        uint64_t s = key & smask;
        bool done = false;
        for (uint64_t probe = 0; probe <= smask; ++probe) {
            const unsigned long long prev = atomicCAS((unsigned long long*)&t[s].key, (unsigned long long)kEmpty,
                                                      (unsigned long long)key);
            if (prev == kEmpty || prev == key) {
                atomicOr((unsigned long long*)&t[s].mask, 1ull << j);
                done = true;
                break;
            }
            s = (s + 1) & smask;
        }
        if (!done) atomicOr(status, RK_DEV_TABLE_FULL);
    }
}

}  // namespace rk

using namespace rk;

extern "C" int rk_index_build(int32_t W, const uint64_t* keys, const int64_t* key_off, void* index,
                              int32_t log2_slots, void* stream)
{
    if (W < 1 || W > 64) return fail(RK_EUNSUPPORTED, "rk_index_build: W outside 1..64");
    if (log2_slots < 4 || log2_slots > 31) return fail(RK_EINVAL, "rk_index_build: log2_slots outside 4..31");
    if (!key_off || !index) return fail(RK_EINVAL, "rk_index_build: NULL array");
    const uint64_t slots = 1ull << log2_slots;
    for (int32_t j = 0; j < W; ++j)
        if (key_off[j + 1] < key_off[j]) return fail(RK_EINVAL, "rk_index_build: key_off not monotone at %d", j);
    const int64_t total = key_off[W] - key_off[0];
    if ((uint64_t)total > slots / 2)
        return fail(RK_ETABLEFULL, "rk_index_build: %lld keys for %llu slots (load above 0.5)", (long long)total,
                    (unsigned long long)slots);
    if (total > 0 && !keys) return fail(RK_EINVAL, "rk_index_build: keys is NULL");
    int32_t* st = status_word();
    if (!st) return fail(RK_EHIP, "rk_index_build: no status word");
    hipStream_t s = (hipStream_t)stream;
    IndexSlot* t = (IndexSlot*)index;
    uint64_t blocks = (slots + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(index_clear_kernel, dim3((unsigned)blocks), dim3(256), 0, s, t, slots);
    int rc = hip_check(hipGetLastError(), "rk_index_build clear launch");
    if (rc) return rc;
    for (int32_t j = 0; j < W; ++j) {
        const int64_t n = key_off[j + 1] - key_off[j];
        if (n == 0) continue;
        int64_t b = (n + 255) / 256;
        if (b > 65536) b = 65536;
        hipLaunchKernelGGL(index_insert_kernel, dim3((unsigned)b), dim3(256), 0, s, keys + key_off[j], n, j, t,
                           slots - 1, st);
        rc = hip_check(hipGetLastError(), "rk_index_build insert launch");
        if (rc) return rc;
    }
    return RK_OK;
}

extern "C" int rk_route_score_index(int32_t B, int32_t W, const uint64_t* chains, const int64_t* chain_off,
                                    const void* index, int32_t log2_slots, const int32_t* active_blocks,
                                    rk_cost_params params, int32_t probe_mode, int32_t* overlap_out, float* cost_out,
                                    int32_t* argmin_out, void* stream)
{
    if (B < 0) return fail(RK_EINVAL, "rk_route_score_index: B < 0");
    if (W < 1 || W > 64) return fail(RK_EUNSUPPORTED, "rk_route_score_index: W outside 1..64");
    if (log2_slots < 4 || log2_slots > 31) return fail(RK_EINVAL, "rk_route_score_index: log2_slots outside 4..31");
    if (!(params.w_ov >= 0.0f) || !(params.w_act >= 0.0f) || !(params.w_sat >= 0.0f))
        return fail(RK_EINVAL, "rk_route_score_index: weights must be >= 0");
    if (params.cap_blocks < 1) return fail(RK_EINVAL, "rk_route_score_index: cap_blocks < 1");
    if (probe_mode != RK_PROBE_PREFIX && probe_mode != RK_PROBE_SCAN)
        return fail(RK_EINVAL, "rk_route_score_index: unknown probe_mode");
    if (B == 0) return RK_OK;
    if (!chain_off || !index || !active_blocks) return fail(RK_EINVAL, "rk_route_score_index: NULL array");
    int32_t* st = status_word();
    if (!st) return fail(RK_EHIP, "rk_route_score_index: no status word");
    hipStream_t s = (hipStream_t)stream;
    int64_t blocks = ((int64_t)B + kRPW - 1) / kRPW;
    if (blocks > 1 << 20) blocks = 1 << 20;
    blocks = (blocks + 7) / 8 * 8;
    const IndexSlot* t = (const IndexSlot*)index;
    if (probe_mode == RK_PROBE_SCAN)
        hipLaunchKernelGGL(score_index_kernel<RK_PROBE_SCAN>, dim3((unsigned)blocks), dim3(64), 0, s, B, W,
                           chains, chain_off, t, log2_slots, active_blocks, params, overlap_out, cost_out, argmin_out,
                           st);
    else
        hipLaunchKernelGGL(score_index_kernel<RK_PROBE_PREFIX>, dim3((unsigned)blocks), dim3(64), 0, s, B,
                           W, chains, chain_off, t, log2_slots, active_blocks, params, overlap_out, cost_out,
                           argmin_out, st);
    return hip_check(hipGetLastError(), "rk_route_score_index launch");
}
