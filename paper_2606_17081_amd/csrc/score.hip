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

// First miss by a scan from block 0 (any table).
__device__ __forceinline__ int32_t overlap_scan(const uint64_t* __restrict__ h, int32_t P,
                                                const uint64_t* __restrict__ t, uint64_t mask)
{
    int32_t o = 0;
    while (o < P && table_has(t, mask, h[o])) ++o;
    return o;
}

// First miss by binary search; exact when membership along the chain is
// monotone (a block is cached only together with its parent).
__device__ __forceinline__ int32_t overlap_bsearch(const uint64_t* __restrict__ h, int32_t P,
                                                   const uint64_t* __restrict__ t, uint64_t mask)
{
    int32_t lo = 0, hi = P;
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        if (table_has(t, mask, h[mid])) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

template <int MODE>
__global__ __launch_bounds__(256) void score_kernel(int32_t B, int32_t W, const uint64_t* __restrict__ chains,
                                                    const int64_t* __restrict__ chain_off,
                                                    const uint64_t* __restrict__ tables, int32_t log2_slots,
                                                    const int32_t* __restrict__ active, rk_cost_params p,
                                                    int32_t* __restrict__ ov_out, float* __restrict__ cost_out,
                                                    int32_t* __restrict__ am_out, int32_t* status)
{
    const int lane = threadIdx.x & 63;
    const int64_t nwaves = (int64_t)gridDim.x * (blockDim.x >> 6);
    const uint64_t mask = (1ull << log2_slots) - 1;
    for (int64_t i = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); i < B; i += nwaves) {
        const int64_t c0 = chain_off[i], c1 = chain_off[i + 1];
        int32_t P = 0;
        if (c1 < c0 || c1 - c0 > 0x7fffffff) {
            if (lane == 0) atomicOr(status, RK_DEV_BAD_OFFSETS);
        } else {
            P = (int32_t)(c1 - c0);
        }
        const uint64_t* h = chains + c0;
        uint64_t best = ~0ull;
        for (int32_t j = lane; j < W; j += 64) {
            const uint64_t* t = tables + ((uint64_t)j << log2_slots);
            const int32_t o = MODE == RK_PROBE_SCAN ? overlap_scan(h, P, t, mask) : overlap_bsearch(h, P, t, mask);
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
    int64_t blocks = ((int64_t)B + 3) / 4;
    if (blocks > 1 << 20) blocks = 1 << 20;
    if (probe_mode == RK_PROBE_SCAN)
        hipLaunchKernelGGL(score_kernel<RK_PROBE_SCAN>, dim3((unsigned)blocks), dim3(256), 0, s, B, W, chains,
                           chain_off, tables, log2_slots, active_blocks, params, overlap_out, cost_out,
                           argmin_out, st);
    else
        hipLaunchKernelGGL(score_kernel<RK_PROBE_PREFIX>, dim3((unsigned)blocks), dim3(256), 0, s, B, W, chains,
                           chain_off, tables, log2_slots, active_blocks, params, overlap_out, cost_out,
                           argmin_out, st);
    return hip_check(hipGetLastError(), "rk_route_score_batch launch");
}
