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
// window's matrix lives in LDS when it fits, else in the workspace.
#include <hip/hip_runtime.h>

#include "rk_internal.h"

namespace rk {

constexpr int PT = 64;   // threads per window

struct PoaArgs {
    int32_t n_windows, max_window, W, kmax;
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

template <bool LDSMAT>
__global__ __launch_bounds__(PT) void poa_window_kernel(PoaArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ int32_t sh_bad;
    __shared__ int32_t sh_hops;
    const int tid = threadIdx.x;
    const int32_t W = a.W;
    int32_t* s_n = (int32_t*)(smem + a.lds_int);   // [W] window counts of the greedy assignment
    int32_t* s_cnt = s_n + W;                        // [W] rows per worker in the partial OPT
    int32_t* s_pred = s_cnt + W;                     // [W]
    int32_t* s_np = s_pred + W;                      // [W]
    float* s_base = (float*)(s_np + W);              // [W]
    int32_t* s_mem = (int32_t*)(s_base + W);         // [W * kmax] rows held by each worker
    int32_t* s_assign = s_mem + W * a.kmax;          // [max_window]
    int32_t* s_pos = s_assign + a.max_window;        // [max_window] index of a row in its worker's list
    int32_t* s_er = s_pos + a.max_window;            // [W * W] row realising each edge weight
    int32_t* s_hx = s_er + W * W;                    // [W + 2] path moves: losing worker
    int32_t* s_hy = s_hx + W + 2;                    // [W + 2]                gaining worker
    int32_t* s_hr = s_hy + W + 2;                    // [W + 2]                row
    double* s_e = (double*)(smem + a.lds_dbl);       // [W * W] edge weights a -> b

    for (int32_t w = blockIdx.x; w < a.n_windows; w += gridDim.x) {
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
        for (int32_t j = tid; j < W; j += PT) {
            s_n[j] = 0;
            s_cnt[j] = 0;
        }
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
        if (tid == 0 && a.selfish) {
            double s = 0.0;
            for (int32_t i = 0; i < m; ++i) s += (double)cm[(int64_t)i * W + a.route_worker[r0 + i]];
            a.selfish[w] = s;
        }
        // ---- successive shortest paths (lane y < W stands for worker y)
        for (int32_t pq = tid; pq < W * W; pq += PT) s_er[pq] = -1;
        __syncthreads();
        for (int32_t i = 0; i < m; ++i) {
            // Bellman-Ford over the workers, wavefront-synchronous: lane y keeps
            // dist[y] and pred[y] in registers and reads the others by shuffles
            double dist = tid < W ? (double)cm[(int64_t)i * W + tid] : dinf();
            int32_t pred = -1;
            for (int32_t round = 0;; ++round) {
                double nd = dist;
                int32_t pb = pred;
                for (int32_t x = 0; x < W; ++x) {
                    const double dx = __shfl(dist, x, 64);
                    if (tid < W) {
                        const double v = dx + s_e[x * W + tid];
                        if (v < nd) {
                            nd = v;
                            pb = x;
                        }
                    }
                }
                const bool changed = __ballot(nd != dist || pb != pred) != 0ull;
                dist = nd;
                pred = pb;
                if (!changed) break;
                if (round > W + 1) {
                    if (tid == 0) atomicOr(a.status, RK_DEV_NO_CONVERGE);
                    break;
                }
            }
            // target: least distance among workers with spare capacity (lowest index on ties)
            int32_t t = -1;
            {
                double bd = tid < W && s_cnt[tid] < K ? dist : dinf();
                int32_t bj = tid < W && s_cnt[tid] < K ? tid : 0x7fffffff;
                for (int off = 32; off > 0; off >>= 1) {
                    const double od = __shfl_xor(bd, off, 64);
                    const int32_t oj = __shfl_xor(bj, off, 64);
                    if (od < bd || (od == bd && oj < bj)) {
                        bd = od;
                        bj = oj;
                    }
                }
                t = bj;
            }
            if (tid < W) s_pred[tid] = pred;
            __syncthreads();
            if (tid == 0) {
                // walk the path back from the target, moving one row per edge
                int32_t y = t, hops = 0;
                while (s_pred[y] >= 0 && hops <= W) {
                    const int32_t x = s_pred[y];
                    const int32_t r = s_er[x * W + y];
                    int32_t kk = r >= 0 ? s_pos[r] : -1;
                    if (kk < 0 || kk >= s_cnt[x] || s_mem[x * a.kmax + kk] != r || s_cnt[y] >= a.kmax) {
                        atomicOr(a.status, RK_DEV_NO_CONVERGE);
                        break;
                    }
                    const int32_t last = s_mem[x * a.kmax + s_cnt[x] - 1];
                    s_mem[x * a.kmax + kk] = last;
                    s_pos[last] = kk;
                    s_cnt[x] -= 1;
                    s_mem[y * a.kmax + s_cnt[y]] = r;
                    s_pos[r] = s_cnt[y];
                    s_cnt[y] += 1;
                    s_assign[r] = y;
                    s_hx[hops] = x;        // x lost r ...
                    s_hy[hops] = y;        // ... and y gained it
                    s_hr[hops] = r;
                    y = x;
                    ++hops;
                }
                if (s_cnt[y] < a.kmax) {
                    s_mem[y * a.kmax + s_cnt[y]] = i;
                    s_pos[i] = s_cnt[y];
                    s_cnt[y] += 1;
                } else {
                    atomicOr(a.status, RK_DEV_NO_CONVERGE);
                }
                s_assign[i] = y;
                s_hx[hops] = -1;           // no loss
                s_hy[hops] = y;            // the new row's worker gained row i
                s_hr[hops] = i;
                sh_hops = hops + 1;
            }
            __syncthreads();
            // ---- edge maintenance, e[x][z] = min over rows r on x of c[r][z] - c[r][x]:
            // an edge whose argmin row left x is recomputed over x's rows (all
            // lanes scan, then a wavefront min); a gained row is folded in.
            const int32_t nev = sh_hops;
            for (int32_t h = 0; h < nev; ++h) {
                const int32_t x = s_hx[h], r = s_hr[h];
                if (x < 0) continue;
                for (int32_t z = 0; z < W; ++z) {
                    if (z == x || s_er[x * W + z] != r) continue;
                    double best = dinf();
                    int32_t brow = 0x7fffffff;
                    for (int32_t k = tid; k < s_cnt[x]; k += PT) {
                        const int32_t q = s_mem[x * a.kmax + k];
                        const double v = (double)cm[(int64_t)q * W + z] - (double)cm[(int64_t)q * W + x];
                        if (v < best || (v == best && q < brow)) {
                            best = v;
                            brow = q;
                        }
                    }
                    for (int off = 32; off > 0; off >>= 1) {
                        const double ob = __shfl_xor(best, off, 64);
                        const int32_t orow = __shfl_xor(brow, off, 64);
                        if (ob < best || (ob == best && orow < brow)) {
                            best = ob;
                            brow = orow;
                        }
                    }
                    if (tid == 0) {
                        s_e[x * W + z] = best;
                        s_er[x * W + z] = brow == 0x7fffffff ? -1 : brow;
                    }
                    __syncthreads();
                }
            }
            for (int32_t h = 0; h < nev; ++h) {
                const int32_t y = s_hy[h], r = s_hr[h];
                if (tid < W && tid != y) {
                    const double v = (double)cm[(int64_t)r * W + tid] - (double)cm[(int64_t)r * W + y];
                    if (v < s_e[y * W + tid]) {
                        s_e[y * W + tid] = v;
                        s_er[y * W + tid] = r;
                    }
                }
                __syncthreads();
            }
        }
        if (tid == 0 && a.coord) {
            double s = 0.0;
            for (int32_t i = 0; i < m; ++i) s += (double)cm[(int64_t)i * W + s_assign[i]];
            a.coord[w] = s;
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
           2 * align_up(((size_t)n_rows + 1) * sizeof(double), 256);
}

extern "C" int rk_poa_estimate(int32_t n_windows, const int64_t* win_off, int32_t n_episodes,
                               const int64_t* ep_win_off, int64_t n_rows, int32_t max_window, int32_t W,
                               const int32_t* route_worker, const int32_t* overlap, const int32_t* route_blocks,
                               rk_poa_params params, double* selfish_out, double* coord_out, double* poa_hat_out,
                               void* workspace, size_t ws_bytes, void* stream)
{
    if (n_windows < 0 || n_episodes < 0 || n_rows < 0) return fail(RK_EINVAL, "rk_poa_estimate: negative count");
    if (W < 1 || W > 64) return fail(RK_EUNSUPPORTED, "rk_poa_estimate: W outside 1..64");
    if (max_window < 1 || max_window > 4096) return fail(RK_EUNSUPPORTED, "rk_poa_estimate: max_window outside 1..4096");
    if (params.beta < 1 || params.beta > 64) return fail(RK_EINVAL, "rk_poa_estimate: beta outside 1..64");
    if (params.K_fixed < 0) return fail(RK_EINVAL, "rk_poa_estimate: K_fixed < 0");
    if (n_windows == 0 && n_episodes == 0) return RK_OK;
    if (n_episodes > 0 && (!ep_win_off || !poa_hat_out))
        return fail(RK_EINVAL, "rk_poa_estimate: episodes need ep_win_off and poa_hat_out");
    if (n_windows > 0 && (!win_off || !route_worker || !overlap || !route_blocks || !workspace))
        return fail(RK_EINVAL, "rk_poa_estimate: NULL array");
    const size_t need = rk_poa_workspace_size(n_rows, W);
    if (ws_bytes < need) return fail(RK_ENOMEM, "rk_poa_estimate: workspace %zu bytes < %zu", ws_bytes, need);
    int32_t* st = status_word();
    if (!st) return fail(RK_EHIP, "rk_poa_estimate: no status word");

    unsigned char* ws = (unsigned char*)workspace;
    const size_t cm_bytes = align_up((size_t)n_rows * (size_t)W * sizeof(float), 256);
    const size_t vec_bytes = align_up(((size_t)n_rows + 1) * sizeof(double), 256);
    double* selfish = selfish_out ? selfish_out : (double*)(ws + cm_bytes + 256);
    double* coord = coord_out ? coord_out : (double*)(ws + cm_bytes + 512 + vec_bytes);
    if (n_episodes > 0 && (!selfish_out || !coord_out) && (size_t)n_windows > (size_t)n_rows + 1)
        return fail(RK_EINVAL, "rk_poa_estimate: pass selfish_out and coord_out when windows exceed rows");
    hipStream_t s = (hipStream_t)stream;

    if (n_windows > 0) {
        PoaArgs a;
        a.n_windows = n_windows;
        a.max_window = max_window;
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
        o = align_up(((size_t)W * 5 + (size_t)W * a.kmax + 2 * (size_t)max_window + (size_t)W * W +
                      3 * ((size_t)W + 2)) * 4, 16);
        a.lds_dbl = (uint32_t)o;
        o = align_up(o + (size_t)W * W * 8, 16);
        const size_t limit = 60 * 1024;
        if (o > limit)
            return fail(RK_EUNSUPPORTED, "rk_poa_estimate: %zu bytes of LDS per window exceed 60 KiB", o);
        const size_t mat = (size_t)max_window * (size_t)W * sizeof(float);
        const bool lds_mat = o + mat <= limit;
        a.lds_mat = (uint32_t)o;
        if (lds_mat) o += mat;
        unsigned grid = (unsigned)(n_windows < 65536 ? n_windows : 65536);
        if (lds_mat) hipLaunchKernelGGL(poa_window_kernel<true>, dim3(grid), dim3(PT), o, s, a);
        else hipLaunchKernelGGL(poa_window_kernel<false>, dim3(grid), dim3(PT), o, s, a);
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
