// poa.hip -- PoA-hat per window of routes (frozen cost matrix, selfish sum and
// the optimal capacity-constrained assignment) and per-episode ratios.
//
// OPT is computed by successive shortest paths: rows are added one at a time
// and each is placed along a cheapest augmenting path, which keeps the partial
// assignment optimal.  Because every replica of a worker column costs the
// same, the residual graph collapses onto the W workers: moving an assigned
// row r from worker a to worker b costs c[r][b] - c[r][a], so the edge a -> b
// weighs the minimum of that over rows on a.  A path starts with the new row
// on some worker and ends on a worker with spare capacity; Bellman-Ford over
// the W nodes finds it (no negative cycles, since the partial assignment is
// optimal).  Edge minima are kept across rows and recomputed only for workers
// whose rows changed on the last path.  One wavefront solves one window; the
// window's matrix lives in LDS when it fits, else in the workspace.  Lane y
// keeps worker y's distance, predecessor and row count in registers, values
// move between lanes by readlane and DPP, and the path is walked by the whole
// wavefront in lockstep.  With few workers the idle lanes share the work: for
// W <= 16 (W <= 32) the rows (halves) of the wavefront each relax from a part
// of the workers, and the edges that lost their argmin row are recomputed by
// groups of lanes side by side.  Windows are dispatched longest first (a
// bucket sort by size class), since the longest ones set the length of the
// launch.
#include <hip/hip_runtime.h>

#include <mutex>

#include "rk_internal.h"

namespace rk {

constexpr int PT = 64;   // threads per window

struct PoaArgs {
    int32_t n_windows, max_window, W, kmax;
    const int32_t* order;  // dispatch order of the windows, or NULL for 0..n_windows-1
    int64_t n_rows;
    const int64_t* win_off;
    const int32_t* route_worker;
    const int32_t* overlap;
    const int32_t* route_blocks;
    rk_poa_params p;
    double* selfish;
    double* coord;
    float* cm;            // workspace: frozen matrix, row-major by route row (when not in LDS)
    int32_t* status;
    uint32_t lds_int, lds_dbl, lds_mat;
};

__device__ __forceinline__ double dinf() { return __longlong_as_double(0x7ff0000000000000ll); }

// the double held by lane src (src uniform across the wavefront)
__device__ __forceinline__ double lane_f64(double v, int32_t src)
{
    const long long b = __double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, src);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), src);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

__device__ __forceinline__ void pick(double& v, int32_t& j, double ov, int32_t oj)
{
    if (ov < v || (ov == v && oj < j)) {
        v = ov;
        j = oj;
    }
}

template <int CTRL>
__device__ __forceinline__ void argmin_dpp_step(double& v, int32_t& j)
{
    const long long b = __double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)b, (int)(uint32_t)b, CTRL, 0xF, 0xF, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)(b >> 32), (int)(uint32_t)(b >> 32),
                                                              CTRL, 0xF, 0xF, false);
    const int32_t oj = __builtin_amdgcn_update_dpp(j, j, CTRL, 0xF, 0xF, false);
    pick(v, j, __longlong_as_double((long long)(((uint64_t)hi << 32) | lo)), oj);
}

// One candidate of the row-parallel relaxation: the distance at position P of the lane's row of
// 16, plus the edge weight e, against the best (bv, bx) so far.
template <int P>
__device__ __forceinline__ void relax_from_row(double rot, double e, int32_t x, double& bv, int32_t& bx)
{
    const double v = __builtin_amdgcn_update_dpp(rot, rot, 0x150 + P, 0xF, 0xF, false) + e;   // row_newbcast:P
    if (v < bv) {
        bv = v;
        bx = x;
    }
}

// Least (value, index) pair over the 64 lanes, by value and then by index;
// every lane receives it.  Swaps within quads, then the mirrored half row and
// row, leave each row of 16 lanes holding its minimum; the four rows are then
// combined in a fixed order.
// ROWS: the rows of 16 lanes that can hold a candidate (the others hold +inf).
template <int ROWS = 4>
__device__ __forceinline__ void wave_argmin_f64(double& v, int32_t& j)
{
    argmin_dpp_step<0xB1>(v, j);    // quad_perm [1,0,3,2]
    argmin_dpp_step<0x4E>(v, j);    // quad_perm [2,3,0,1]
    argmin_dpp_step<0x141>(v, j);   // row_half_mirror
    argmin_dpp_step<0x140>(v, j);   // row_mirror
    double bv = lane_f64(v, 0);
    int32_t bj = __builtin_amdgcn_readlane(j, 0);
#pragma unroll
    for (int32_t r = 16; r < 16 * ROWS; r += 16) pick(bv, bj, lane_f64(v, r), __builtin_amdgcn_readlane(j, r));
    v = bv;
    j = bj;
}

// Sum of term(i) over the m rows of a window, the same value in every lane:
// lane l adds rows l, l + 64, ... in order, then the 64 partial sums are added
// in lane order (fp64; a fixed order, so every launch gives the same bits).
template <class Term>
__device__ __forceinline__ double window_sum(int32_t m, const Term& term)
{
    const int lane = threadIdx.x & 63;
    double part = 0.0;
    for (int32_t i = lane; i < m; i += PT) part += term(i);
    double s = 0.0;
    for (int32_t l = 0; l < PT && l < m; ++l) s += lane_f64(part, l);
    return s;
}

// Dispatch order: windows by descending size class (bit length of m), so the
// longest windows start first.  Three small launches over the whole grid
// (one workgroup reading a million window offsets alone takes a millisecond):
// zero the 16 class counters and 16 class cursors; count the windows of each
// class (a wavefront adds its 64 windows per class with ballots, one atomic
// per class present); scatter each window to its class's range, the classes
// laid out from the longest down.  The order within a class is whatever the
// atomics give (it only affects scheduling).
__device__ __forceinline__ int32_t window_class(const int64_t* __restrict__ win_off, int32_t w)
{
    const int64_t m = win_off[w + 1] - win_off[w];
    return m <= 0 ? 0 : (m >= 4096 ? 13 : 64 - __clzll((unsigned long long)m));
}

__global__ void poa_order_zero_kernel(int32_t* __restrict__ cls_cnt)
{
    if (threadIdx.x < 32) cls_cnt[threadIdx.x] = 0;
}

__global__ __launch_bounds__(256) void poa_order_count_kernel(int32_t n_windows, const int64_t* __restrict__ win_off,
                                                               int32_t* __restrict__ cls_cnt)
{
    const int lane = threadIdx.x & 63;
    const int32_t stride = gridDim.x * blockDim.x;
    for (int32_t w0 = blockIdx.x * blockDim.x + threadIdx.x - lane; w0 < n_windows; w0 += stride) {
        const int32_t w = w0 + lane;
        const int32_t c = w < n_windows ? window_class(win_off, w) : -1;
        for (int32_t k = 0; k < 16; ++k) {
            const unsigned long long mb = __ballot(c == k);
            if (lane == 0 && mb) atomicAdd(&cls_cnt[k], (int32_t)__popcll(mb));
        }
    }
}

__global__ __launch_bounds__(256) void poa_order_scatter_kernel(int32_t n_windows, const int64_t* __restrict__ win_off,
                                                                 int32_t* __restrict__ cls_cnt,
                                                                 int32_t* __restrict__ order)
{
    // cls_cnt[0..15]: windows per class; cls_cnt[16..31]: windows of each class placed so far
    __shared__ int32_t base[16];
    if (threadIdx.x == 0) {
        int32_t o = 0;
        for (int32_t c = 15; c >= 0; --c) {
            base[c] = o;
            o += cls_cnt[c];
        }
    }
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int32_t stride = gridDim.x * blockDim.x;
    for (int32_t w0 = blockIdx.x * blockDim.x + threadIdx.x - lane; w0 < n_windows; w0 += stride) {
        const int32_t w = w0 + lane;
        const int32_t c = w < n_windows ? window_class(win_off, w) : -1;
        for (int32_t k = 0; k < 16; ++k) {
            const unsigned long long mb = __ballot(c == k);
            if (!mb) continue;
            int32_t b0 = 0;
            if (lane == 0) b0 = base[k] + atomicAdd(&cls_cnt[16 + k], (int32_t)__popcll(mb));
            b0 = __builtin_amdgcn_readfirstlane(b0);
            if (c == k) order[b0 + __popcll(mb & ((1ull << lane) - 1ull))] = w;
        }
    }
}

// For W <= 16 the kernel is held to 80 registers (six waves per SIMD, 24 windows per CU, about what
// the LDS allows) without spills: the saturation sweep's windows take 2% less time than at 85
// registers (five waves); at 64 registers (eight waves) the spills cost more than the waves gain.
template <bool LDSMAT, int WMAX>
__global__ __launch_bounds__(PT) __attribute__((amdgpu_waves_per_eu(WMAX <= 16 ? 6 : 1))) void poa_window_kernel(
    PoaArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ int32_t sh_bad;
    const int tid = threadIdx.x;
    const int32_t W = a.W;
    int32_t* s_n = (int32_t*)(smem + a.lds_int);   // [W] window counts of the greedy assignment
    float* s_base = (float*)(s_n + W);               // [W]
    // row indices and positions are below 4096: 16-bit, so that more windows fit a CU's LDS
    int16_t* s_mem = (int16_t*)(s_base + W);         // [W * kmax] rows held by each worker
    int16_t* s_pos = s_mem + W * a.kmax;             // [max_window] index of a row in its worker's list
    int16_t* s_er = s_pos + a.max_window;            // [W * W] row realising each edge weight (-1: none)
    double* s_e = (double*)(smem + a.lds_dbl);       // [W * W] edge weights a -> b

    for (int32_t wi = blockIdx.x; wi < a.n_windows; wi += gridDim.x) {
        const int32_t w = a.order ? a.order[wi] : wi;
        const int64_t r0 = a.win_off[w], r1 = a.win_off[w + 1];
        const int64_t m64 = r1 - r0;
        if (r0 < 0 || m64 < 0 || r1 > a.n_rows || m64 > a.max_window) {
            if (tid == 0) {
                atomicOr(a.status, RK_DEV_TOO_LARGE);
                if (a.selfish) a.selfish[w] = __longlong_as_double(0x7ff8000000000000ll);
                if (a.coord) a.coord[w] = __longlong_as_double(0x7ff8000000000000ll);
            }
            continue;
        }
        const int32_t m = (int32_t)m64;
        int32_t K = a.p.K_fixed > 0 ? a.p.K_fixed : (m + W - 1) / W;
        if (K > m) K = m;
        if ((int64_t)K * W < m || K > a.kmax) {
            if (tid == 0) {
                atomicOr(a.status, RK_DEV_TOO_LARGE);
                if (a.selfish) a.selfish[w] = __longlong_as_double(0x7ff8000000000000ll);
                if (a.coord) a.coord[w] = __longlong_as_double(0x7ff8000000000000ll);
            }
            continue;
        }
        if (m == 0) {
            if (tid == 0) {
                if (a.selfish) a.selfish[w] = 0.0;
                if (a.coord) a.coord[w] = 0.0;
            }
            continue;
        }
        float* cm = LDSMAT ? (float*)(smem + a.lds_mat) : a.cm + r0 * W;
        // ---- frozen matrix
        for (int32_t j = tid; j < W; j += PT) s_n[j] = 0;
        for (int32_t pq = tid; pq < W * W; pq += PT) s_e[pq] = dinf();
        if (tid == 0) sh_bad = 0;
        __syncthreads();
        for (int32_t i = tid; i < m; i += PT) {
            const int32_t sg = a.route_worker[r0 + i];
            if (sg >= 0 && sg < W) atomicAdd(&s_n[sg], 1);
            else sh_bad = 1;
        }
        __syncthreads();
        for (int32_t j = tid; j < W; j += PT) {
            const int32_t gap = a.p.C_cap - s_n[j];
            const float g = (float)(gap > 1 ? gap : 1);
            float gb = g;
            for (int32_t k = 1; k < a.p.beta; ++k) gb = __fmul_rn(gb, g);
            s_base[j] = __fadd_rn(__fadd_rn(__fmul_rn(a.p.a, (float)s_n[j]), a.p.b), __fdiv_rn(a.p.d, gb));
        }
        __syncthreads();
        for (int64_t idx = tid; idx < (int64_t)m * W; idx += PT) {
            const int64_t i = idx / W;
            const int32_t j = (int32_t)(idx - i * W);
            const int32_t P = a.route_blocks[r0 + i];
            const float oh = P > 0 ? __fdiv_rn((float)a.overlap[(r0 + i) * W + j], (float)P) : 0.0f;
            cm[idx] = __fsub_rn(s_base[j], __fmul_rn(a.p.w_c, oh));
        }
        __syncthreads();
        const bool bad_rows = sh_bad != 0;
        __syncthreads();
        if (bad_rows) {
            if (tid == 0) {
                atomicOr(a.status, RK_DEV_BAD_OFFSETS);
                if (a.selfish) a.selfish[w] = __longlong_as_double(0x7ff8000000000000ll);
                if (a.coord) a.coord[w] = __longlong_as_double(0x7ff8000000000000ll);
            }
            continue;
        }
        if (a.selfish) {
            const double s = window_sum(m, [&](int32_t i) { return (double)cm[(int64_t)i * W + a.route_worker[r0 + i]]; });
            if (tid == 0) a.selfish[w] = s;
        }
        // ---- successive shortest paths (lane y < W stands for worker y)
        for (int32_t pq = tid; pq < W * W; pq += PT) s_er[pq] = -1;
        __syncthreads();
        const bool wl = tid < W;
        // lanes that share the recomputation of one edge: a power of two up to a row of 16 lanes,
        // so that DPP moves within rows combine them
        int32_t G = 1;
        while (G < 16 && 2 * G * W <= PT) G *= 2;
        int32_t cnt = 0;   // lane y: rows on worker y in the partial optimum
        bool placed_all = true;
        for (int32_t i = 0; i < m; ++i) {
            double dist;
            int32_t pred = -1;
            float c_row;   // lane y < W (row 0): the new row's cost on worker y
            if constexpr (WMAX <= 16) {
                // Bellman-Ford over the workers (Jacobi rounds), the wavefront as four rows of 16
                // lanes (W <= 16): every row keeps dist[y] at position y, row g relaxes from
                // workers 4g .. 4g + 3 (lane (g, y) keeps the weights e[4g + p][y] in registers),
                // and the rows' least (distance, worker) pairs are merged; worker order breaks ties
                // as in a relaxation from every worker in turn
                const int32_t g = tid >> 4, y = tid & 15;
                const bool wy = y < W;
                double ec[4];
#pragma unroll
                for (int32_t p = 0; p < 4; ++p) {
                    const int32_t x = 4 * g + p;
                    ec[p] = (x < W && wy) ? s_e[x * W + y] : dinf();
                }
                c_row = wy ? cm[(int64_t)i * W + y] : 0.0f;
                dist = wy ? (double)c_row : dinf();
                const int32_t src = (tid & ~15) | (4 * g + (tid & 3));   // position p < 4 of row g: dist[4g + p]
                for (int32_t round = 0;; ++round) {
                    const long long db = __double_as_longlong(dist);
                    const uint32_t rlo = (uint32_t)__shfl((int)(uint32_t)db, src);
                    const uint32_t rhi = (uint32_t)__shfl((int)(uint32_t)(db >> 32), src);
                    const double rot = __longlong_as_double((long long)(((uint64_t)rhi << 32) | rlo));
                    double bv = dinf();
                    int32_t bx = 0x7fffffff;
                    relax_from_row<0>(rot, ec[0], 4 * g, bv, bx);
                    relax_from_row<1>(rot, ec[1], 4 * g + 1, bv, bx);
                    relax_from_row<2>(rot, ec[2], 4 * g + 2, bv, bx);
                    relax_from_row<3>(rot, ec[3], 4 * g + 3, bv, bx);
#pragma unroll
                    for (int32_t sft = 16; sft < 64; sft <<= 1) {
                        const long long bb = __double_as_longlong(bv);
                        const uint32_t olo = (uint32_t)__shfl_xor((int)(uint32_t)bb, sft);
                        const uint32_t ohi = (uint32_t)__shfl_xor((int)(uint32_t)(bb >> 32), sft);
                        const int32_t ox = __shfl_xor(bx, sft);
                        pick(bv, bx, __longlong_as_double((long long)(((uint64_t)ohi << 32) | olo)), ox);
                    }
                    double nd = dist;
                    int32_t pb = pred;
                    if (wy && bv < nd) {
                        nd = bv;
                        pb = bx;
                    }
                    const uint64_t fell = __ballot(nd != dist);
                    dist = nd;
                    pred = pb;
                    if (fell == 0ull) break;
                    if (round > W + 1) {
                        if (tid == 0) atomicOr(a.status, RK_DEV_NO_CONVERGE);
                        break;
                    }
                }
            } else if constexpr (WMAX == 32) {
                // the same with two halves of 32 lanes (16 < W <= 32): every half keeps dist[y] at
                // position y, half h relaxes from workers 16h .. 16h + 15, each row of the half
                // reading them through a copy that holds dist[16h + q] at position q
                const int32_t hh = tid >> 5, y = tid & 31;
                const bool wy = y < W;
                double ec[16];
#pragma unroll
                for (int32_t p = 0; p < 16; ++p) {
                    const int32_t x = 16 * hh + p;
                    ec[p] = (x < W && wy) ? s_e[x * W + y] : dinf();
                }
                c_row = wy ? cm[(int64_t)i * W + y] : 0.0f;
                dist = wy ? (double)c_row : dinf();
                const int32_t src = 48 * hh + (tid & 15);
                for (int32_t round = 0;; ++round) {
                    const long long db = __double_as_longlong(dist);
                    const uint32_t rlo = (uint32_t)__shfl((int)(uint32_t)db, src);
                    const uint32_t rhi = (uint32_t)__shfl((int)(uint32_t)(db >> 32), src);
                    const double rot = __longlong_as_double((long long)(((uint64_t)rhi << 32) | rlo));
                    double bv = dinf();
                    int32_t bx = 0x7fffffff;
                    const int32_t x0 = 16 * hh;
                    relax_from_row<0>(rot, ec[0], x0, bv, bx);
                    relax_from_row<1>(rot, ec[1], x0 + 1, bv, bx);
                    relax_from_row<2>(rot, ec[2], x0 + 2, bv, bx);
                    relax_from_row<3>(rot, ec[3], x0 + 3, bv, bx);
                    relax_from_row<4>(rot, ec[4], x0 + 4, bv, bx);
                    relax_from_row<5>(rot, ec[5], x0 + 5, bv, bx);
                    relax_from_row<6>(rot, ec[6], x0 + 6, bv, bx);
                    relax_from_row<7>(rot, ec[7], x0 + 7, bv, bx);
                    relax_from_row<8>(rot, ec[8], x0 + 8, bv, bx);
                    relax_from_row<9>(rot, ec[9], x0 + 9, bv, bx);
                    relax_from_row<10>(rot, ec[10], x0 + 10, bv, bx);
                    relax_from_row<11>(rot, ec[11], x0 + 11, bv, bx);
                    relax_from_row<12>(rot, ec[12], x0 + 12, bv, bx);
                    relax_from_row<13>(rot, ec[13], x0 + 13, bv, bx);
                    relax_from_row<14>(rot, ec[14], x0 + 14, bv, bx);
                    relax_from_row<15>(rot, ec[15], x0 + 15, bv, bx);
                    {
                        const long long bb = __double_as_longlong(bv);
                        const uint32_t olo = (uint32_t)__shfl_xor((int)(uint32_t)bb, 32);
                        const uint32_t ohi = (uint32_t)__shfl_xor((int)(uint32_t)(bb >> 32), 32);
                        const int32_t ox = __shfl_xor(bx, 32);
                        pick(bv, bx, __longlong_as_double((long long)(((uint64_t)ohi << 32) | olo)), ox);
                    }
                    double nd = dist;
                    int32_t pb = pred;
                    if (wy && bv < nd) {
                        nd = bv;
                        pb = bx;
                    }
                    const uint64_t fell = __ballot(nd != dist);
                    dist = nd;
                    pred = pb;
                    if (fell == 0ull) break;
                    if (round > W + 1) {
                        if (tid == 0) atomicOr(a.status, RK_DEV_NO_CONVERGE);
                        break;
                    }
                }
            } else {
                // Bellman-Ford over the workers (Jacobi rounds): lane y keeps dist[y]
                // and pred[y]; lane y's column of edge weights sits in registers
                double ecol[WMAX];
#pragma unroll
                for (int32_t x = 0; x < WMAX; ++x) ecol[x] = (x < W && wl) ? s_e[x * W + tid] : dinf();
                c_row = wl ? cm[(int64_t)i * W + tid] : 0.0f;
                dist = wl ? (double)c_row : dinf();
                // workers to relax from: all in the first round, then those whose distance fell in
                // the round before (from any other worker every candidate was tried already with
                // the same distance, and a tie never replaces a distance or a predecessor)
                uint64_t relax = ~0ull;
                for (int32_t round = 0;; ++round) {
                    double nd = dist;
                    int32_t pb = pred;
#pragma unroll
                    for (int32_t x = 0; x < WMAX; ++x) {
                        if (x < W && ((relax >> x) & 1ull)) {
                            const double v = lane_f64(dist, x) + ecol[x];
                            if (wl && v < nd) {
                                nd = v;
                                pb = x;
                            }
                        }
                    }
                    const uint64_t fell = __ballot(nd != dist);
                    dist = nd;
                    pred = pb;
                    if (fell == 0ull) break;
                    relax = fell;
                    if (round > W + 1) {
                        if (tid == 0) atomicOr(a.status, RK_DEV_NO_CONVERGE);
                        break;
                    }
                }
            }
            // target: least distance among workers with spare capacity (lowest index on ties)
            double bd = wl && cnt < K ? dist : dinf();
            int32_t t = wl && cnt < K ? tid : 0x7fffffff;
            wave_argmin_f64<WMAX <= 16 ? 1 : WMAX <= 32 ? 2 : 4>(bd, t);
            if (t < 0 || t >= W) {   // no worker with spare capacity: impossible when K * W >= m
                if (tid == 0) atomicOr(a.status, RK_DEV_NO_CONVERGE);
                placed_all = false;
                break;
            }
            // walk the path back from the target, moving one row per edge; lane h
            // records move h (losing worker, gaining worker, row)
            int32_t hx = -1, hy = -1, hr = -1;
            int32_t y = t, hops = 0;
            for (;;) {
                const int32_t x = __builtin_amdgcn_readlane(pred, y);
                if (x < 0) break;
                const int32_t cx = __builtin_amdgcn_readlane(cnt, x), cy = __builtin_amdgcn_readlane(cnt, y);
                const int32_t r = s_er[x * W + y];
                const int32_t kk = r >= 0 ? s_pos[r] : -1;
                if (hops >= W - 1 || kk < 0 || kk >= cx || s_mem[x * a.kmax + kk] != r || cy >= a.kmax) {
                    if (tid == 0) atomicOr(a.status, RK_DEV_NO_CONVERGE);
                    break;
                }
                const int32_t last = s_mem[x * a.kmax + cx - 1];
                if (tid == 0) {
                    s_mem[x * a.kmax + kk] = (int16_t)last;
                    s_pos[last] = (int16_t)kk;
                    s_mem[y * a.kmax + cy] = (int16_t)r;
                    s_pos[r] = (int16_t)cy;
                }
                cnt += (tid == y) - (tid == x);
                if (tid == hops) {
                    hx = x;        // x lost r ...
                    hy = y;        // ... and y gained it
                    hr = r;
                }
                y = x;
                ++hops;
            }
            {
                const int32_t cy = __builtin_amdgcn_readlane(cnt, y);
                if (cy < a.kmax) {
                    if (tid == 0) {
                        s_mem[y * a.kmax + cy] = (int16_t)i;
                        s_pos[i] = (int16_t)cy;
                    }
                    cnt += tid == y;
                } else if (tid == 0) {
                    atomicOr(a.status, RK_DEV_NO_CONVERGE);
                }
                if (tid == hops) {
                    hx = -1;       // no loss
                    hy = y;        // the new row's worker gained row i
                    hr = i;
                }
                ++hops;
            }
            __syncthreads();
            // ---- edge maintenance, e[x][z] = min over rows r on x of c[r][z] - c[r][x]:
            // the edges whose argmin row left x are recomputed over x's rows together
            // (lane G z + g scans x's rows g, g + G, ... for edge x -> z; the G lanes of
            // an edge then take the least (value, row) pair); a gained row is folded in.
            for (int32_t h = 0; h < hops; ++h) {
                const int32_t x = __builtin_amdgcn_readlane(hx, h), r = __builtin_amdgcn_readlane(hr, h);
                if (x < 0) continue;
                const bool lz = wl && tid != x && s_er[x * W + tid] == r;
                const uint64_t lost = __ballot(lz);
                if (lost == 0ull) continue;
                const int32_t cx = __builtin_amdgcn_readlane(cnt, x);
                if ((lost & (lost - 1)) == 0ull) {
                    // a single edge: every lane scans rows for it, then a wavefront argmin
                    const int32_t z1 = __ffsll((unsigned long long)lost) - 1;
                    double best = dinf();
                    int32_t brow = 0x7fffffff;
                    for (int32_t k = tid; k < cx; k += PT) {
                        const int32_t q = s_mem[x * a.kmax + k];
                        pick(best, brow, (double)cm[(int64_t)q * W + z1] - (double)cm[(int64_t)q * W + x], q);
                    }
                    wave_argmin_f64(best, brow);
                    if (tid == 0) {
                        s_e[x * W + z1] = best;
                        s_er[x * W + z1] = (int16_t)(brow == 0x7fffffff ? -1 : brow);
                    }
                    continue;
                }
                const int32_t z = tid / G, g = tid % G;
                const bool mine = z < W && z != x && s_er[x * W + z] == r;
                double best = dinf();
                int32_t brow = 0x7fffffff;
                if (mine) {
                    // four rows per lane at a time, their loads issued before any is used
                    for (int32_t k0 = g; k0 < cx; k0 += 4 * G) {
                        int32_t q[4];
                        float cz[4], cxv[4];
#pragma unroll
                        for (int u = 0; u < 4; ++u) {
                            const int32_t k = k0 + u * G;
                            q[u] = k < cx ? s_mem[x * a.kmax + k] : -1;
                        }
#pragma unroll
                        for (int u = 0; u < 4; ++u) {
                            const int64_t row = q[u] >= 0 ? (int64_t)q[u] * W : 0;
                            cz[u] = cm[row + z];
                            cxv[u] = cm[row + x];
                        }
#pragma unroll
                        for (int u = 0; u < 4; ++u)
                            if (q[u] >= 0) pick(best, brow, (double)cz[u] - (double)cxv[u], q[u]);
                    }
                }
                if (G >= 2) argmin_dpp_step<0xB1>(best, brow);    // quad_perm [1,0,3,2]
                if (G >= 4) argmin_dpp_step<0x4E>(best, brow);    // quad_perm [2,3,0,1]
                if (G >= 8) argmin_dpp_step<0x141>(best, brow);   // row_half_mirror
                if (G >= 16) argmin_dpp_step<0x140>(best, brow);  // row_mirror
                if (g == 0 && mine) {
                    s_e[x * W + z] = best;
                    s_er[x * W + z] = (int16_t)(brow == 0x7fffffff ? -1 : brow);
                }
            }
            for (int32_t h = 0; h < hops; ++h) {
                const int32_t yg = __builtin_amdgcn_readlane(hy, h), r = __builtin_amdgcn_readlane(hr, h);
                // the new row's costs are in registers already
                const float cg = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(c_row), yg));
                if (wl && tid != yg) {
                    const double v = r == i ? (double)c_row - (double)cg
                                            : (double)cm[(int64_t)r * W + tid] - (double)cm[(int64_t)r * W + yg];
                    if (v < s_e[yg * W + tid]) {
                        s_e[yg * W + tid] = v;
                        s_er[yg * W + tid] = (int16_t)r;
                    }
                }
            }
            __syncthreads();
        }
        if (tid == 0 && a.coord && !placed_all) a.coord[w] = __longlong_as_double(0x7ff8000000000000ll);
        if (a.coord && placed_all) {
            // lane y adds the rows of worker y in list order, then the W sums in worker order
            double part = 0.0;
            if (wl)
                for (int32_t k = 0; k < cnt; ++k) part += (double)cm[(int64_t)s_mem[tid * a.kmax + k] * W + tid];
            double sum = 0.0;
            for (int32_t y = 0; y < W; ++y) sum += lane_f64(part, y);
            if (tid == 0) a.coord[w] = sum;
        }
        __syncthreads();
    }
}

__global__ void poa_episode_kernel(int32_t n_episodes, const int64_t* __restrict__ ep_win_off,
                                   const double* __restrict__ selfish, const double* __restrict__ coord,
                                   double* __restrict__ poa)
{
    const int32_t e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n_episodes) return;
    double s = 0.0, c = 0.0;
    for (int64_t w = ep_win_off[e]; w < ep_win_off[e + 1]; ++w) {
        s += selfish[w];
        c += coord[w];
    }
    poa[e] = s / c;
}

}  // namespace rk

using namespace rk;

extern "C" size_t rk_poa_workspace_size(int64_t n_rows, int32_t W)
{
    if (n_rows < 0 || W < 1) return 0;
    return align_up((size_t)n_rows * (size_t)W * sizeof(float), 256) + 2 * 256 +
           2 * align_up(((size_t)n_rows + 1) * sizeof(double), 256) +
           align_up(((size_t)n_rows + 1) * sizeof(int32_t), 256) + 256;
}

template <bool LDSMAT>
static void launch_windows(int32_t W, unsigned grid, size_t lds, hipStream_t s, const PoaArgs& a)
{
    if (W <= 8) hipLaunchKernelGGL((poa_window_kernel<LDSMAT, 8>), dim3(grid), dim3(PT), lds, s, a);
    else if (W <= 16) hipLaunchKernelGGL((poa_window_kernel<LDSMAT, 16>), dim3(grid), dim3(PT), lds, s, a);
    else if (W <= 32) hipLaunchKernelGGL((poa_window_kernel<LDSMAT, 32>), dim3(grid), dim3(PT), lds, s, a);
    else hipLaunchKernelGGL((poa_window_kernel<LDSMAT, 64>), dim3(grid), dim3(PT), lds, s, a);
}

// Argument checks shared by rk_poa_estimate and rk_poa_estimate_noalloc;
// RK_OK with *nothing set when there is no work.
static int poa_check(const char* who, int32_t n_windows, const int64_t* win_off, int32_t n_episodes,
                     const int64_t* ep_win_off, int64_t n_rows, int32_t max_window, int32_t W,
                     const int32_t* route_worker, const int32_t* overlap, const int32_t* route_blocks,
                     const rk_poa_params& params, const double* poa_hat_out, bool* nothing)
{
    *nothing = false;
    if (n_windows < 0 || n_episodes < 0 || n_rows < 0) return fail(RK_EINVAL, "%s: negative count", who);
    if (W < 1 || W > 64) return fail(RK_EUNSUPPORTED, "%s: W outside 1..64", who);
    if (max_window < 1 || max_window > 4096) return fail(RK_EUNSUPPORTED, "%s: max_window outside 1..4096", who);
    if (params.beta < 1 || params.beta > 64) return fail(RK_EINVAL, "%s: beta outside 1..64", who);
    if (params.K_fixed < 0) return fail(RK_EINVAL, "%s: K_fixed < 0", who);
    if (n_windows == 0 && n_episodes == 0) {
        *nothing = true;
        return RK_OK;
    }
    if (n_episodes > 0 && (!ep_win_off || !poa_hat_out))
        return fail(RK_EINVAL, "%s: episodes need ep_win_off and poa_hat_out", who);
    if (n_windows > 0 && (!win_off || !route_worker || !overlap || !route_blocks))
        return fail(RK_EINVAL, "%s: NULL array", who);
    return RK_OK;
}

// The launches of one estimate on a checked workspace of at least
// rk_poa_workspace_size(n_rows, W) bytes.
static int poa_launch(int32_t n_windows, const int64_t* win_off, int32_t n_episodes, const int64_t* ep_win_off,
                      int64_t n_rows, int32_t max_window, int32_t W, const int32_t* route_worker,
                      const int32_t* overlap, const int32_t* route_blocks, rk_poa_params params,
                      double* selfish_out, double* coord_out, double* poa_hat_out, unsigned char* ws, void* stream)
{
    int32_t* st = status_word();
    if (!st) return fail(RK_EHIP, "rk_poa_estimate: no status word");

    const size_t cm_bytes = align_up((size_t)n_rows * (size_t)W * sizeof(float), 256);
    const size_t vec_bytes = align_up(((size_t)n_rows + 1) * sizeof(double), 256);
    double* selfish = selfish_out ? selfish_out : (double*)(ws + cm_bytes + 256);
    double* coord = coord_out ? coord_out : (double*)(ws + cm_bytes + 512 + vec_bytes);
    // the dispatch order has room for n_rows + 1 windows; beyond that (many
    // empty windows) the windows run in index order, and so do up to 256
    // windows (each starts at once on a CU of its own, so no order shortens
    // the launch, and the three ordering launches are saved)
    int32_t* order = (n_windows > 256 && (size_t)n_windows <= (size_t)n_rows + 1)
                         ? (int32_t*)(ws + cm_bytes + 512 + 2 * vec_bytes) : nullptr;
    if (n_episodes > 0 && (!selfish_out || !coord_out) && (size_t)n_windows > (size_t)n_rows + 1)
        return fail(RK_EINVAL, "rk_poa_estimate: pass selfish_out and coord_out when windows exceed rows");
    hipStream_t s = (hipStream_t)stream;

    if (n_windows > 0) {
        PoaArgs a;
        a.n_windows = n_windows;
        a.max_window = max_window;
        a.order = order;
        a.W = W;
        a.kmax = params.K_fixed > 0 ? (params.K_fixed < max_window ? params.K_fixed : max_window)
                                    : (max_window + W - 1) / W;
        a.n_rows = n_rows;
        a.win_off = win_off;
        a.route_worker = route_worker;
        a.overlap = overlap;
        a.route_blocks = route_blocks;
        a.p = params;
        a.selfish = selfish;
        a.coord = coord;
        a.cm = (float*)ws;
        a.status = st;
        size_t o = 0;
        a.lds_int = 0;
        o = align_up((size_t)W * 2 * 4 + ((size_t)W * a.kmax + (size_t)max_window + (size_t)W * W) * 2, 16);
        a.lds_dbl = (uint32_t)o;
        o = align_up(o + (size_t)W * W * 8, 16);
        const size_t limit = 60 * 1024;
        if (o > limit)
            return fail(RK_EUNSUPPORTED, "rk_poa_estimate: %zu bytes of LDS per window exceed 60 KiB", o);
        // the frozen matrix goes to LDS only while a window's whole LDS stays within 20 KiB, so that
        // at least eight windows share a CU; a larger matrix is read from the workspace instead
        // (the solver's steps are latency-bound and need the waves: multi-turn windows of 256
        // rows x 32 workers, 43 KiB with the matrix, take half the time from the workspace)
        const size_t mat = (size_t)max_window * (size_t)W * sizeof(float);
        const bool lds_mat = o + mat <= 20 * 1024;
        a.lds_mat = (uint32_t)o;
        if (lds_mat) o += mat;
        if (order) {
            int32_t* cls_cnt = (int32_t*)(ws + cm_bytes + 512 + 2 * vec_bytes +
                                          align_up(((size_t)n_rows + 1) * sizeof(int32_t), 256));
            const unsigned og = (unsigned)((n_windows + 255) / 256 < 1024 ? (n_windows + 255) / 256 : 1024);
            hipLaunchKernelGGL(poa_order_zero_kernel, dim3(1), dim3(64), 0, s, cls_cnt);
            hipLaunchKernelGGL(poa_order_count_kernel, dim3(og), dim3(256), 0, s, n_windows, win_off, cls_cnt);
            hipLaunchKernelGGL(poa_order_scatter_kernel, dim3(og), dim3(256), 0, s, n_windows, win_off, cls_cnt,
                               order);
            int rc = hip_check(hipGetLastError(), "rk_poa_estimate order launch");
            if (rc) return rc;
        }
        // up to 2^17 workgroups, each looping over the windows a grid-stride apart (2^16: 0.9% slower on
        // the saturation sweep's 652,800 windows; one workgroup per window: no faster)
        unsigned grid = (unsigned)(n_windows < 131072 ? n_windows : 131072);
        if (lds_mat) launch_windows<true>(W, grid, o, s, a);
        else launch_windows<false>(W, grid, o, s, a);
        int rc = hip_check(hipGetLastError(), "rk_poa_estimate window launch");
        if (rc) return rc;
    }
    if (n_episodes > 0) {
        hipLaunchKernelGGL(poa_episode_kernel, dim3((n_episodes + 255) / 256), dim3(256), 0, s, n_episodes,
                           ep_win_off, selfish, coord, poa_hat_out);
        return hip_check(hipGetLastError(), "rk_poa_estimate episode launch");
    }
    return RK_OK;
}

extern "C" int rk_poa_estimate(int32_t n_windows, const int64_t* win_off, int32_t n_episodes,
                               const int64_t* ep_win_off, int64_t n_rows, int32_t max_window, int32_t W,
                               const int32_t* route_worker, const int32_t* overlap, const int32_t* route_blocks,
                               rk_poa_params params, double* selfish_out, double* coord_out, double* poa_hat_out,
                               void* workspace, size_t ws_bytes, void* stream)
{
    bool nothing;
    int rc = poa_check("rk_poa_estimate", n_windows, win_off, n_episodes, ep_win_off, n_rows, max_window, W,
                       route_worker, overlap, route_blocks, params, poa_hat_out, &nothing);
    if (rc || nothing) return rc;
    if (n_windows > 0 && !workspace) return fail(RK_EINVAL, "rk_poa_estimate: NULL workspace");
    const size_t need = rk_poa_workspace_size(n_rows, W);
    if (ws_bytes < need) return fail(RK_ENOMEM, "rk_poa_estimate: workspace %zu bytes < %zu", ws_bytes, need);
    return poa_launch(n_windows, win_off, n_episodes, ep_win_off, n_rows, max_window, W, route_worker, overlap,
                      route_blocks, params, selfish_out, coord_out, poa_hat_out, (unsigned char*)workspace, stream);
}

// ---- the estimate without a caller workspace (for callers that cannot allocate)
//
// The workspace is a file-scope device array; each device holds its own copy
// until the process ends.  Host code never passes the array's name to a kernel
// (on the host it only stands for the symbol): the device address comes from
// hipGetSymbolAddress, taken once per device with that device current.

static __device__ __align__(256) unsigned char scratch[RK_POA_NOALLOC_BYTES];

static std::mutex g_scratch_mu;
static unsigned char* g_scratch_addr[64];

static unsigned char* scratch_address(int* err)
{
    int dev = 0;
    *err = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
        *err = 1;
        return nullptr;
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        unsigned char* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr) {
            *err = 2;
            return nullptr;
        }
        g_scratch_addr[dev] = ptr;
    }
    return g_scratch_addr[dev];
}

extern "C" int rk_poa_estimate_noalloc(int32_t n_windows, const int64_t* win_off, int32_t n_episodes,
                                       const int64_t* ep_win_off, int64_t n_rows, int32_t max_window, int32_t W,
                                       const int32_t* route_worker, const int32_t* overlap,
                                       const int32_t* route_blocks, rk_poa_params params, double* selfish_out,
                                       double* coord_out, double* poa_hat_out, void* stream)
{
    bool nothing;
    int rc = poa_check("rk_poa_estimate_noalloc", n_windows, win_off, n_episodes, ep_win_off, n_rows, max_window,
                       W, route_worker, overlap, route_blocks, params, poa_hat_out, &nothing);
    if (rc || nothing) return rc;
    const size_t need = rk_poa_workspace_size(n_rows, W);
    if (need > (size_t)RK_POA_NOALLOC_BYTES)
        return fail(RK_EUNSUPPORTED,
                    "rk_poa_estimate_noalloc: %lld rows x %d workers need %zu bytes of workspace, more than the "
                    "%zu of the static buffer (use rk_poa_estimate with a workspace)",
                    (long long)n_rows, W, need, (size_t)RK_POA_NOALLOC_BYTES);
    int err = 0;
    unsigned char* ws = scratch_address(&err);
    if (!ws)
        return fail(RK_EHIP, "rk_poa_estimate_noalloc: %s", err == 1 ? "no current device"
                                                                      : "hipGetSymbolAddress of the buffer failed");
    return poa_launch(n_windows, win_off, n_episodes, ep_win_off, n_rows, max_window, W, route_worker, overlap,
                      route_blocks, params, selfish_out, coord_out, poa_hat_out, ws, stream);
}
