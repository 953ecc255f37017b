// rk_internal.h -- shared device helpers and host plumbing of the routing library.
// Internal to the library (not part of the C ABI in include/rkroute.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "rkroute.h"

namespace rk {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;  // splitmix64 increment; also the zero remap
constexpr uint64_t kEmpty = 0;                       // empty table slot
constexpr uint32_t kTomb = 0xFFFFFFFFu;              // stamp of an evicted (tombstoned) slot

// ------------------------------------------------------------------ hashing

// One splitmix64 generator step applied to state x (Vigna, splitmix64.c).
__device__ __forceinline__ uint64_t mix64(uint64_t x)
{
    uint64_t z = x + kGolden;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// FNV-1a 64 over the four little-endian bytes of one int32 token.
__device__ __forceinline__ uint64_t fnv_word(uint64_t h, uint32_t v)
{
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        h ^= (uint64_t)((v >> (8 * b)) & 0xffu);
        h *= 0x100000001b3ull;
    }
    return h;
}

__device__ __forceinline__ uint64_t chain_next(uint64_t prev, uint64_t f)
{
    uint64_t h = mix64(prev ^ f);
    return h == 0 ? kGolden : h;
}

// -------------------------------------------------------------------- cost

// Router cost in fp32 with the fixed operation order of the ABI; explicit
// round-to-nearest intrinsics keep every product and sum separately rounded.
__device__ __forceinline__ float route_cost(float w_ov, float w_act, float w_sat, int32_t cap,
                                            int32_t P, int32_t o, int32_t A)
{
    float t1 = __fmul_rn(w_ov, (float)(P - o));
    float t2 = __fmul_rn(w_act, (float)A);
    float r = __fdiv_rn((float)((int64_t)A + (int64_t)P), (float)cap);
    float x = fmaxf(__fsub_rn(r, 1.0f), 0.0f);
    float t3 = __fmul_rn(w_sat, __fmul_rn(x, x));
    return __fadd_rn(__fadd_rn(t1, t2), t3);
}

// The cost when the cached prefix spans memory tiers (Section 4.2, Eq.
// kv-cost): o1 leading blocks in G1, o12 in G1 or G2, the rest of the o cached
// ones in G3; a block served from a tier counts tw of a recomputed block in the
// prefill term, summed in tier order.
__device__ __forceinline__ float route_cost_tiers(float w_ov, float w_act, float w_sat, int32_t cap, int32_t P,
                                                  int32_t o, int32_t o1, int32_t o12, const float* tw, int32_t A)
{
    float pf = (float)(P - o);
    pf = __fadd_rn(pf, __fmul_rn(tw[0], (float)o1));
    pf = __fadd_rn(pf, __fmul_rn(tw[1], (float)(o12 - o1)));
    pf = __fadd_rn(pf, __fmul_rn(tw[2], (float)(o - o12)));
    float t1 = __fmul_rn(w_ov, pf);
    float t2 = __fmul_rn(w_act, (float)A);
    float r = __fdiv_rn((float)((int64_t)A + (int64_t)P), (float)cap);
    float x = fmaxf(__fsub_rn(r, 1.0f), 0.0f);
    float t3 = __fmul_rn(w_sat, __fmul_rn(x, x));
    return __fadd_rn(__fadd_rn(t1, t2), t3);
}

// exp(x) for x <= 0 in float, Cody and Waite's method: x = n ln2 + r with
// n = floor(x log2(e) + 1/2) and ln2 split into a part exact in float and a
// correction, |r| <= ln2/2; exp(r) by its Taylor series to degree 7 (Horner);
// times 2^n through the exponent field.  Every operation is rounded on its
// own.  Below -87 the result is 0; x > 0 or NaN gives 1.
__device__ __forceinline__ float exp_neg_f32(float x)
{
    if (!(x <= 0.0f)) return 1.0f;
    if (x < -87.0f) return 0.0f;
    const float n = floorf(__fadd_rn(__fmul_rn(x, 1.44269504088896341f), 0.5f));
    const float r = __fsub_rn(__fsub_rn(x, __fmul_rn(n, 0.693145751953125f)),
                              __fmul_rn(n, 1.42860682030941723212e-6f));
    float p = 1.98412698412698412698e-4f;                      // 1/7!
    p = __fadd_rn(__fmul_rn(p, r), 1.38888888888888888889e-3f);   // 1/6!
    p = __fadd_rn(__fmul_rn(p, r), 8.33333333333333333333e-3f);   // 1/5!
    p = __fadd_rn(__fmul_rn(p, r), 4.16666666666666666667e-2f);   // 1/4!
    p = __fadd_rn(__fmul_rn(p, r), 1.66666666666666666667e-1f);   // 1/3!
    p = __fadd_rn(__fmul_rn(p, r), 0.5f);
    p = __fadd_rn(__fmul_rn(p, r), 1.0f);
    p = __fadd_rn(__fmul_rn(p, r), 1.0f);
    return __fmul_rn(p, __uint_as_float((uint32_t)((int32_t)n + 127) << 23));
}

// Key whose unsigned order is (cost, worker) lexicographic for cost >= 0.
__device__ __forceinline__ uint64_t argmin_key(float c, int32_t j)
{
    return ((uint64_t)__float_as_uint(__fadd_rn(c, 0.0f)) << 32) | (uint32_t)j;
}

// ------------------------------------------------- wavefront primitives (DPP)
// Cross-lane steps as DPP operand modifiers of ordinary VALU instructions
// (GFX9-family controls), so a scan or reduction over the 64 lanes costs a few
// dependent VALU operations instead of round trips through the LDS crossbar.
constexpr int kDppQuadSwap1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kDppQuadSwap2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;
constexpr int kDppRowMirror = 0x140, kDppRowHalfMirror = 0x141;
constexpr int kDppRowBcast15 = 0x142;     // lane 15 of each row to the whole next row
constexpr int kDppRowBcast31 = 0x143;     // lane 31 to rows 2 and 3

// v moved by the DPP control CTRL into the rows of ROWS; lanes without a
// source, and rows outside ROWS, receive old.
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ uint32_t dpp32(uint32_t old, uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROWS, 0xF, false);
}

template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ uint64_t dpp64(uint64_t old, uint64_t v)
{
    const uint32_t lo = dpp32<CTRL, ROWS>((uint32_t)old, (uint32_t)v);
    const uint32_t hi = dpp32<CTRL, ROWS>((uint32_t)(old >> 32), (uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// Lane l's value of v (l uniform across the wavefront).
__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}

// Inclusive prefix AND over the lanes (lane order): shifts within each row of
// 16 lanes, then each row's total carried into the rows after it.  All lanes
// must be active.
__device__ __forceinline__ uint64_t wave_scan_and_u64(uint64_t v)
{
    const uint64_t id = ~0ull;
    v &= dpp64<kDppRowShr1>(id, v);
    v &= dpp64<kDppRowShr2>(id, v);
    v &= dpp64<kDppRowShr4>(id, v);
    v &= dpp64<kDppRowShr8>(id, v);
    v &= dpp64<kDppRowBcast15, 0xA>(id, v);
    v &= dpp64<kDppRowBcast31, 0xC>(id, v);
    return v;
}

// Exclusive prefix sum over the lanes; total receives the sum of all lanes.
// All lanes must be active.
__device__ __forceinline__ int32_t wave_excl_sum_dpp(int32_t v, int32_t& total)
{
    uint32_t x = (uint32_t)v;
    x += dpp32<kDppRowShr1>(0u, x);
    x += dpp32<kDppRowShr2>(0u, x);
    x += dpp32<kDppRowShr4>(0u, x);
    x += dpp32<kDppRowShr8>(0u, x);
    x += dpp32<kDppRowBcast15, 0xA>(0u, x);
    x += dpp32<kDppRowBcast31, 0xC>(0u, x);
    total = __builtin_amdgcn_readlane((int)x, 63);
    return (int32_t)x - v;
}

// Minimum / OR of v over the lanes, the same value in every lane: a butterfly
// within each row of 16 (pair swap, quad swap, half-row mirror, row mirror),
// then the four row results.  All lanes must be active.
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v)
{
    auto mn = [](uint64_t a, uint64_t b) { return b < a ? b : a; };
    v = mn(v, dpp64<kDppQuadSwap1>(v, v));
    v = mn(v, dpp64<kDppQuadSwap2>(v, v));
    v = mn(v, dpp64<kDppRowHalfMirror>(v, v));
    v = mn(v, dpp64<kDppRowMirror>(v, v));
    return mn(mn(readlane64(v, 0), readlane64(v, 16)), mn(readlane64(v, 32), readlane64(v, 48)));
}

__device__ __forceinline__ uint64_t wave_or_u64(uint64_t v)
{
    v |= dpp64<kDppQuadSwap1>(v, v);
    v |= dpp64<kDppQuadSwap2>(v, v);
    v |= dpp64<kDppRowHalfMirror>(v, v);
    v |= dpp64<kDppRowMirror>(v, v);
    return (readlane64(v, 0) | readlane64(v, 16)) | (readlane64(v, 32) | readlane64(v, 48));
}

// route_cost for the episodes, where A + P stays far below 2^31 (blocks in
// flight), so the sum converts from 32 bits; a power-of-two cap divides by the
// exact multiplication with its reciprocal inv_cap (the same correctly
// rounded quotient), and inv_cap = 0 selects the division.
__device__ __forceinline__ float route_cost_ep(float w_ov, float w_act, float w_sat, int32_t cap, float inv_cap,
                                               int32_t P, int32_t o, int32_t A)
{
    float t1 = __fmul_rn(w_ov, (float)(P - o));
    float t2 = __fmul_rn(w_act, (float)A);
    const float L = (float)(A + P);
    float r = inv_cap != 0.0f ? __fmul_rn(L, inv_cap) : __fdiv_rn(L, (float)cap);
    float x = fmaxf(__fsub_rn(r, 1.0f), 0.0f);
    float t3 = __fmul_rn(w_sat, __fmul_rn(x, x));
    return __fadd_rn(__fadd_rn(t1, t2), t3);
}

// Sum of v over the lanes, the same value in every lane (DPP butterfly within
// each row of 16, then the four row sums).  All lanes must be active.
__device__ __forceinline__ int32_t wave_sum_i32(int32_t v)
{
    uint32_t x = (uint32_t)v;
    x += dpp32<kDppQuadSwap1>(x, x);
    x += dpp32<kDppQuadSwap2>(x, x);
    x += dpp32<kDppRowHalfMirror>(x, x);
    x += dpp32<kDppRowMirror>(x, x);
    return (int32_t)(((uint32_t)__builtin_amdgcn_readlane((int)x, 0) + (uint32_t)__builtin_amdgcn_readlane((int)x, 16)) +
                     ((uint32_t)__builtin_amdgcn_readlane((int)x, 32) + (uint32_t)__builtin_amdgcn_readlane((int)x, 48)));
}

// ------------------------------------------------- read-only table probes
// Open addressing, home slot key & mask, linear probing; 0 is empty.
__device__ __forceinline__ bool table_has(const uint64_t* __restrict__ t, uint64_t mask, uint64_t key)
{
    uint64_t s = key & mask;
    for (uint64_t n = 0; n <= mask; ++n) {
        uint64_t k = t[s];
        if (k == key) return true;
        if (k == kEmpty) return false;
        s = (s + 1) & mask;
    }
    return false;
}

// ------------------------------------------------------------ host plumbing
int fail(int status, const char* fmt, ...);                  // records rk_last_error
int hip_check(hipError_t e, const char* what);
int32_t* status_word();                                      // device address for the current device
inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline uint64_t next_pow2(uint64_t x)
{
    uint64_t p = 1;
    while (p < x) p <<= 1;
    return p;
}

// One cached block of an episode's worker table: the chained hash, the log
// position of its latest touch (kTomb once evicted) and, under frequency
// eviction, the block's frequency key (frequency plus the decay epoch of its
// last update).  They travel in one 16-byte load.
struct __align__(16) Slot {
    uint64_t key;
    uint32_t stamp;
    uint32_t fkey;
};

// An entry of an episode's run index: a route added the blocks [o, end) of
// its chain to a worker that held the blocks before o; the run is entered
// under the hash of block o and of every block of it at a position that is a
// multiple of 2^kCkptLog.  val packs the chain's base index (bits 63..24), the
// worker (23..16) and end (15..0).  Key 0 marks an empty slot.
struct __align__(16) RunSlot {
    uint64_t key;
    uint64_t val;
};
constexpr int kCkptLog = 4;

constexpr int kEpisodeThreads = 256;   // threads of an episode's workgroup

// Episode workspace layout (bytes), shared by the size query and the launch.
struct EpisodeLayout {
    uint64_t slots;        // table slots per worker (power of two)
    uint64_t ring;         // LRU log records per worker (power of two)
    uint64_t runs;         // run slots of the episode's prefix index (power of two)
    size_t off_slots, off_log, off_scratch, off_scratch_f, off_queue, off_next, off_hist, off_replay, off_later,
        off_ctl, off_runs;
    size_t per_episode;
};
EpisodeLayout episode_layout(int32_t W, int32_t cache_blocks, int32_t max_blocks, int32_t max_conv,
                             int32_t max_routes);

}  // namespace rk
