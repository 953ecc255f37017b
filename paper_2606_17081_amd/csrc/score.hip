// score.hip -- batched (request x worker) routing-cost evaluation and argmin.
//
// One wavefront scores one request at a time; lane j owns worker j (and
// j + 64, ... when W > 64).  Each lane finds the longest cached prefix of the
// request's block-hash chain in its worker's table, turns it into the fp32
// routing cost, and a wavefront min-reduction over packed (cost, worker) keys
// yields the argmin (lowest worker on ties).
#include <hip/hip_runtime.h>

#include "rk_internal.h"

namespace rk {

constexpr int kWinSlots = 4;      // slots one lookup loads together
constexpr int kStageS = 512;      // leading chain hashes staged in LDS
constexpr int kHintFan = 16;      // positions per round of the shared search on worker 0's table

// Membership of key in a table probed linearly from key & mask: the slots of
// a window starting at the home slot are loaded together, so one round trip
// settles a lookup unless every slot of the window holds another key.
__device__ __forceinline__ bool table_has_win(const uint64_t* __restrict__ t, uint64_t mask, uint64_t key)
{
    uint64_t s = key & mask;
    for (uint64_t n = 0; n <= mask; n += kWinSlots) {
        uint64_t k[kWinSlots];
#pragma unroll
        for (int x = 0; x < kWinSlots; ++x) k[x] = t[(s + x) & mask];
#pragma unroll
        for (int x = 0; x < kWinSlots; ++x) {
            if (k[x] == key) return true;
            if (k[x] == kEmpty) return false;
        }
        s = (s + kWinSlots) & mask;
    }
    return false;
}

// LDS writes of one wavefront made visible to the other lanes of that wavefront.
__device__ __forceinline__ void score_wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One wavefront per request; lane j owns worker j (and j + 64, ... when W > 64).
// PREFIX mode with W <= 64: workers often hold a request's chain to the same
// depth (a shared prefix cached everywhere), so the lanes first find worker 0's
// overlap o0 together, in rounds of kHintFan probes of its table, and every
// lane then checks o0 on its own table with two probes (block o0 - 1 cached,
// block o0 missing); only a worker that fails the check searches further, by
// binary lifting on the side of o0 that holds its first miss.
// PREFIX mode otherwise: the first miss by binary lifting -- with lo blocks known
// cached, test block lo + step - 1 for step = 2^k, ..., 2, 1 and advance lo by
// step on a hit.  Exact when membership along the chain is monotone (a block
// is cached only with its parent).  The positions tested depend only on the
// outcomes, not on the chain's length, so requests of one prefix group that
// stop at the same block test the same table slots and share cache lines.
// SCAN mode: blocks from 0 until the first miss (any tables).
template <int MODE>
__global__ __launch_bounds__(64) void score_kernel(int32_t B, int32_t W, const uint64_t* __restrict__ chains,
                                                   const int64_t* __restrict__ chain_off,
                                                   const uint64_t* __restrict__ tables, int32_t log2_slots,
                                                   const int32_t* __restrict__ active, rk_cost_params p,
                                                   int32_t* __restrict__ ov_out, float* __restrict__ cost_out,
                                                   int32_t* __restrict__ am_out, int32_t* status)
{
    __shared__ uint64_t s_ch[kStageS];
    const int lane = threadIdx.x & 63;
    const uint64_t mask = (1ull << log2_slots) - 1;
    // Workgroups are handed to the 8 XCDs round-robin; renumber them so each
    // XCD walks one contiguous range of requests (gridDim.x is a multiple of 8).
    const uint32_t nb8 = gridDim.x >> 3;
    const uint32_t lb = (blockIdx.x & 7u) * nb8 + (blockIdx.x >> 3);
    for (int64_t i = lb; i < B; i += gridDim.x) {
        const int64_t c0 = chain_off[i], c1 = chain_off[i + 1];
        int32_t P = 0;
        if (c1 < c0 || c1 - c0 > 0x7fffffff) {
            if (lane == 0) atomicOr(status, RK_DEV_BAD_OFFSETS);
        } else {
            P = (int32_t)(c1 - c0);
        }
        const uint64_t* __restrict__ hg = chains + c0;
        score_wave_sync();   // the previous request's reads of s_ch are done
        {
            const int32_t n = min(P, kStageS);
            uint64_t v[kStageS / 64];
#pragma unroll
            for (int k = 0; k < kStageS / 64; ++k) v[k] = lane + 64 * k < n ? hg[lane + 64 * k] : 0ull;
#pragma unroll
            for (int k = 0; k < kStageS / 64; ++k) s_ch[lane + 64 * k] = v[k];
        }
        score_wave_sync();
        auto h = [&](int32_t x) -> uint64_t { return x < kStageS ? s_ch[x] : hg[x]; };
        const int32_t top = P > 0 ? (int32_t)(1u << (31 - __clz(P))) : 0;
        uint64_t best = ~0ull;
        if (MODE == RK_PROBE_PREFIX && W <= 64) {
            // Phase A: the lanes search worker 0's table together.  [lo, hi) holds its
            // first miss, with block lo - 1 cached (or lo == 0) and block hi missing (or
            // hi == P); each round tests up to kHintFan positions spread over the interval.
            int32_t lo = 0, hi = P;
            while (hi > lo) {
                const int32_t span = hi - lo;
                const int32_t n = min(span, kHintFan);
                // sample k (k < n) at the end of the k-th of n near-equal parts of [lo, hi)
                const int32_t q = lo + (int32_t)(((int64_t)(lane + 1) * span) / n) - 1;
                const bool hit = lane < n && table_has_win(tables, mask, h(q));
                const uint64_t miss = __ballot(lane < n && !hit);
                if (miss == 0ull) {
                    lo = hi;
                    break;
                }
                const int k = __ffsll((unsigned long long)miss) - 1;
                const int32_t qk = __builtin_amdgcn_readlane(q, k);
                const int32_t qp = k == 0 ? lo - 1 : __builtin_amdgcn_readlane(q, k - 1);
                lo = qp + 1;
                hi = qk;
            }
            const int32_t o0 = lo;   // worker 0's overlap
            // Phase B: worker j's overlap is o0 when block o0 - 1 is in its table and
            // block o0 is not; otherwise binary lifting on the side of o0 that holds it.
            if (lane < W) {
                const uint64_t* __restrict__ t = tables + ((uint64_t)lane << log2_slots);
                const bool before = o0 == 0 || table_has_win(t, mask, h(o0 - 1));
                const bool at = o0 < P && table_has_win(t, mask, h(o0));
                int32_t o = o0;
                if (!before || at) {
                    // first miss in [b0, b1]: b0 blocks known cached, block b1 missing or b1 == P
                    const int32_t b0 = before ? o0 + 1 : 0, b1 = before ? P : o0 - 1;
                    o = b0;
                    const int32_t len = b1 - b0;
                    for (int32_t step = len > 0 ? (int32_t)(1u << (31 - __clz(len))) : 0; step > 0; step >>= 1) {
                        const int32_t pos = o + step - 1;
                        if (pos < b1 && table_has_win(t, mask, h(pos))) o += step;
                    }
                }
                const float c = route_cost(p.w_ov, p.w_act, p.w_sat, p.cap_blocks, P, o, active[lane]);
                if (ov_out) ov_out[i * W + lane] = o;
                if (cost_out) cost_out[i * W + lane] = c;
                best = argmin_key(c, lane);
            }
            best = wave_min_u64(best);
            if (lane == 0 && am_out) am_out[i] = (int32_t)(uint32_t)(best & 0xffffffffu);
            continue;
        }
        for (int32_t j = lane; j < W; j += 64) {
            const uint64_t* __restrict__ t = tables + ((uint64_t)j << log2_slots);
            int32_t o = 0;
            if (MODE == RK_PROBE_SCAN) {
                while (o < P && table_has_win(t, mask, h(o))) ++o;
            } else {
                for (int32_t step = top; step > 0; step >>= 1) {
                    const int32_t pos = o + step - 1;
                    if (pos < P && table_has_win(t, mask, h(pos))) o += step;
                }
            }
            const float c = route_cost(p.w_ov, p.w_act, p.w_sat, p.cap_blocks, P, o, active[j]);
            if (ov_out) ov_out[i * W + j] = o;
            if (cost_out) cost_out[i * W + j] = c;
            const uint64_t k = argmin_key(c, j);
            best = k < best ? k : best;
        }
        best = wave_min_u64(best);
        if (lane == 0 && am_out) am_out[i] = (int32_t)(uint32_t)(best & 0xffffffffu);
    }
}

}  // namespace rk

using namespace rk;

extern "C" int rk_route_score_batch(int32_t B, int32_t W, const uint64_t* chains, const int64_t* chain_off,
                                    const uint64_t* tables, int32_t log2_slots, const int32_t* active_blocks,
                                    rk_cost_params params, int32_t probe_mode, int32_t* overlap_out,
                                    float* cost_out, int32_t* argmin_out, void* stream)
{
    if (B < 0) return fail(RK_EINVAL, "rk_route_score_batch: B < 0");
    if (W < 1 || W > 1024) return fail(RK_EINVAL, "rk_route_score_batch: W outside 1..1024");
    if (log2_slots < 4 || log2_slots > 30) return fail(RK_EINVAL, "rk_route_score_batch: log2_slots outside 4..30");
    if (!(params.w_ov >= 0.0f) || !(params.w_act >= 0.0f) || !(params.w_sat >= 0.0f))
        return fail(RK_EINVAL, "rk_route_score_batch: weights must be >= 0");
    if (params.cap_blocks < 1) return fail(RK_EINVAL, "rk_route_score_batch: cap_blocks < 1");
    if (probe_mode != RK_PROBE_PREFIX && probe_mode != RK_PROBE_SCAN)
        return fail(RK_EINVAL, "rk_route_score_batch: unknown probe_mode");
    if (B == 0) return RK_OK;
    if (!chain_off || !tables || !active_blocks) return fail(RK_EINVAL, "rk_route_score_batch: NULL array");
    int32_t* st = status_word();
    if (!st) return fail(RK_EHIP, "rk_route_score_batch: no status word");
    hipStream_t s = (hipStream_t)stream;
    int64_t blocks = B;
    if (blocks > 1 << 20) blocks = 1 << 20;
    blocks = (blocks + 7) / 8 * 8;
    if (probe_mode == RK_PROBE_SCAN)
        hipLaunchKernelGGL(score_kernel<RK_PROBE_SCAN>, dim3((unsigned)blocks), dim3(64), 0, s, B, W, chains,
                           chain_off, tables, log2_slots, active_blocks, params, overlap_out, cost_out,
                           argmin_out, st);
    else
        hipLaunchKernelGGL(score_kernel<RK_PROBE_PREFIX>, dim3((unsigned)blocks), dim3(64), 0, s, B, W, chains,
                           chain_off, tables, log2_slots, active_blocks, params, overlap_out, cost_out,
                           argmin_out, st);
    return hip_check(hipGetLastError(), "rk_route_score_batch launch");
}
