// abi.hip -- status handling, block-hash chains and table construction.
#include <hip/hip_runtime.h>

#include <mutex>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "rk_internal.h"

namespace rk {

static thread_local char g_last_error[512] = "";

int fail(int status, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return status;
}

int hip_check(hipError_t e, const char* what)
{
    if (e == hipSuccess) return RK_OK;
    return fail(RK_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// One status word per device.  Kernels OR RK_DEV_* bits into it; the host
// finds its address per device once and reads it in rk_device_status.
static __device__ int32_t g_status;

static std::mutex g_status_mu;
static int32_t* g_status_addr[64];

int32_t* status_word()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
    std::lock_guard<std::mutex> lk(g_status_mu);
    if (!g_status_addr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(g_status)) != hipSuccess) return nullptr;
        g_status_addr[dev] = (int32_t*)p;
    }
    return g_status_addr[dev];
}

EpisodeLayout episode_layout(int32_t W, int32_t cache_blocks, int32_t max_blocks, int32_t max_conv,
                             int32_t max_routes)
{
    EpisodeLayout L;
    uint64_t live_max = (uint64_t)cache_blocks + (uint64_t)max_blocks;
    L.slots = next_pow2(2 * live_max);
    L.ring = next_pow2(2 * live_max);
    // run index entries: a run's first block and its checkpoints, at most 2 per route plus one per
    // 2^kCkptLog cached blocks of each worker, at load <= 1/2
    L.runs = next_pow2(2 * (2 * (uint64_t)(max_routes > 2 ? max_routes : 2) +
                            (uint64_t)W * ((live_max >> kCkptLog) + 1)));
    size_t o = 0;
    L.off_slots = o;   o = align_up(o + (size_t)W * L.slots * sizeof(Slot), 256);
    L.off_log = o;     o = align_up(o + (size_t)W * L.ring * sizeof(uint32_t), 256);
    L.off_scratch = o; o = align_up(o + live_max * sizeof(uint64_t), 256);
    L.off_scratch_f = o; o = align_up(o + live_max * sizeof(uint32_t), 256);
    L.off_queue = o;   o = align_up(o + ((size_t)max_conv + 1) * sizeof(int32_t), 256);
    L.off_next = o;    o = align_up(o + ((size_t)max_conv + 1) * sizeof(int32_t), 256);
    L.off_hist = o;    o = align_up(o + ((size_t)max_routes + 1) * 2 * sizeof(int32_t), 256);
    L.off_replay = o;  o = align_up(o + (size_t)kEpisodeThreads * 16, 256);
    L.off_later = o;   o = align_up(o + ((size_t)max_conv + 1) * sizeof(int32_t), 256);
    L.off_ctl = o;     o = align_up(o + 256, 256);     // launch control (episode queue counter)
    L.off_runs = o;    o = align_up(o + L.runs * sizeof(RunSlot), 256);
    L.per_episode = o;
    return L;
}

// ------------------------------------------------------------------ hashing

// FNV-1a of every block: one wavefront per sequence, lanes over blocks.  The
// per-block values are written in place of the chain and chained afterwards.
__global__ __launch_bounds__(256) void block_fnv_kernel(int64_t n_seq, const int32_t* __restrict__ tokens,
                                                        const int64_t* __restrict__ tok_off,
                                                        const int64_t* __restrict__ chain_off,
                                                        uint64_t* __restrict__ chains, int32_t* status)
{
    const int lane = threadIdx.x & 63;
    const int64_t nwaves = (int64_t)gridDim.x * (blockDim.x >> 6);
    for (int64_t s = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); s < n_seq; s += nwaves) {
        const int64_t t0 = tok_off[s], t1 = tok_off[s + 1];
        const int64_t c0 = chain_off[s], c1 = chain_off[s + 1];
        if (t1 < t0 || c1 < c0) {
            if (lane == 0) atomicOr(status, RK_DEV_BAD_OFFSETS);
            continue;
        }
        const int64_t nb = c1 - c0;
        const int64_t avail = (t1 - t0) / 16;
        if (nb > avail && lane == 0) atomicOr(status, RK_DEV_SHORT_INPUT);
        for (int64_t k = lane; k < nb; k += 64) {
            uint64_t h = 0;
            if (k < avail) {
                const int32_t* tk = tokens + t0 + 16 * k;
                h = 0xcbf29ce484222325ull;
#pragma unroll
                for (int q = 0; q < 16; ++q) h = fnv_word(h, (uint32_t)tk[q]);
            }
            chains[c0 + k] = h;
        }
    }
}

// Serial chaining of each sequence: one lane per sequence.  A wavefront runs
// as long as its longest sequence, so each 1024-thread workgroup first ranks
// its sequences by length (classes of 32 blocks, longest first) and hands
// them to lanes in that order: the sequences of one wavefront then have
// similar lengths.  The per-block values move through registers kChainChunk
// at a time, and the next chunk's reads are issued before the current chunk
// is chained, so a lane's memory latency overlaps its arithmetic.  Reads and
// writes past a sequence's end are clamped to its last block (a write there
// stores that block's final value), which keeps every memory instruction
// unconditional.
constexpr int kChainChunk = 16;
// two chained values, 8-byte aligned (a 16-byte access needs only the element alignment)
typedef uint64_t u64x2 __attribute__((ext_vector_type(2), aligned(8)));
constexpr int kChainWG = 1024;
constexpr int kChainClasses = 32;

__device__ __forceinline__ int64_t chain_length(int64_t s, const int64_t* __restrict__ tok_off,
                                                const int64_t* __restrict__ chain_off, int64_t& c0)
{
    c0 = chain_off[s];
    const int64_t c1 = chain_off[s + 1], t0 = tok_off[s], t1 = tok_off[s + 1];
    if (c1 < c0 || t1 < t0) return 0;
    return min(c1 - c0, (t1 - t0) / 16);
}

__global__ __launch_bounds__(kChainWG) void chain_kernel(int64_t n_seq, const int64_t* __restrict__ tok_off,
                                                         const int64_t* __restrict__ chain_off,
                                                         uint64_t* __restrict__ chains)
{
    __shared__ int32_t cnt[kChainClasses], base[kChainClasses];
    __shared__ int32_t order[kChainWG];
    const int tid = threadIdx.x;
    const int64_t s0 = (int64_t)blockIdx.x * kChainWG;
    const int32_t m = (int32_t)min((int64_t)kChainWG, n_seq - s0);
    if (tid < kChainClasses) cnt[tid] = 0;
    __syncthreads();
    int cls = 0;
    if (tid < m) {
        int64_t c0;
        const int64_t n = chain_length(s0 + tid, tok_off, chain_off, c0);
        cls = (int)min(n / 32, (int64_t)(kChainClasses - 1));
        atomicAdd(&cnt[cls], 1);
    }
    __syncthreads();
    if (tid == 0) {
        int32_t o = 0;
        for (int c = kChainClasses - 1; c >= 0; --c) {
            base[c] = o;
            o += cnt[c];
        }
    }
    __syncthreads();
    if (tid < m) order[atomicAdd(&base[cls], 1)] = tid;
    __syncthreads();
    if (tid >= m) return;
    const int64_t s = s0 + order[tid];
    int64_t c0;
    const int64_t n = chain_length(s, tok_off, chain_off, c0);
    if (n <= 0) return;
    const int64_t last = c0 + n - 1;
    uint64_t cur[kChainChunk], nxt[kChainChunk];
    // whole chunks move as pairs of values (16-byte accesses); a chunk that reaches past the
    // sequence's last block moves value by value, clamped to it
    auto load_chunk = [&](int64_t k, uint64_t* v) {
        if (k + kChainChunk - 1 <= last - c0) {
#pragma unroll
            for (int u = 0; u < kChainChunk; u += 2) {
                const u64x2 q = *reinterpret_cast<const u64x2*>(chains + c0 + k + u);
                v[u] = q.x;
                v[u + 1] = q.y;
            }
        } else {
#pragma unroll
            for (int u = 0; u < kChainChunk; ++u) v[u] = chains[min(c0 + k + u, last)];
        }
    };
    load_chunk(0, cur);
    uint64_t h = 0;
    for (int64_t k0 = 0; k0 < n; k0 += kChainChunk) {
        load_chunk(k0 + kChainChunk, nxt);
#pragma unroll
        for (int u = 0; u < kChainChunk; ++u) {
            const uint64_t hn = chain_next(h, cur[u]);
            h = k0 + u < n ? hn : h;
            cur[u] = h;
        }
        if (k0 + kChainChunk - 1 <= last - c0) {
#pragma unroll
            for (int u = 0; u < kChainChunk; u += 2) {
                u64x2 q;
                q.x = cur[u];
                q.y = cur[u + 1];
                *reinterpret_cast<u64x2*>(chains + c0 + k0 + u) = q;
            }
        } else {
#pragma unroll
            for (int u = 0; u < kChainChunk; ++u) chains[min(c0 + k0 + u, last)] = cur[u];
        }
#pragma unroll
        for (int u = 0; u < kChainChunk; ++u) cur[u] = nxt[u];
    }
}

// ------------------------------------------------------------------ tables

__global__ __launch_bounds__(256) void table_clear_kernel(uint64_t* __restrict__ t, uint64_t n)
{
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        t[i] = kEmpty;
}

__global__ __launch_bounds__(256) void table_insert_kernel(const uint64_t* __restrict__ keys, int64_t n,
                                                           uint64_t* __restrict__ t, uint64_t mask,
                                                           int32_t* status)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const uint64_t key = keys[i];
        if (key == kEmpty) {
            atomicOr(status, RK_DEV_ZERO_KEY);
            continue;
        }
        uint64_t s = key & mask;
        bool done = false;
        for (uint64_t probe = 0; probe <= mask; ++probe) {
            unsigned long long prev = atomicCAS((unsigned long long*)&t[s], (unsigned long long)kEmpty,
                                                (unsigned long long)key);
            if (prev == kEmpty || prev == key) { done = true; break; }
            s = (s + 1) & mask;
        }
        if (!done) atomicOr(status, RK_DEV_TABLE_FULL);
    }
}

}  // namespace rk

using namespace rk;

extern "C" {

const char* rk_status_string(int status)
{
    switch (status) {
    case RK_OK: return "ok";
    case RK_EINVAL: return "invalid argument";
    case RK_ENOMEM: return "workspace too small";
    case RK_EHIP: return "HIP runtime error";
    case RK_ETABLEFULL: return "table full";
    case RK_EUNSUPPORTED: return "unsupported size";
    default: return "unknown status";
    }
}

const char* rk_last_error(void) { return g_last_error; }

int rk_device_status(int reset, int32_t* bits, void* stream)
{
    if (!bits) return fail(RK_EINVAL, "rk_device_status: bits is NULL");
    int32_t* p = status_word();
    if (!p) return fail(RK_EHIP, "rk_device_status: no status word on this device");
    hipStream_t st = (hipStream_t)stream;
    int rc = hip_check(hipMemcpyAsync(bits, p, sizeof(int32_t), hipMemcpyDeviceToHost, st),
                       "rk_device_status copy");
    if (rc) return rc;
    rc = hip_check(hipStreamSynchronize(st), "rk_device_status sync");
    if (rc) return rc;
    if (reset) {
        rc = hip_check(hipMemsetAsync(p, 0, sizeof(int32_t), st), "rk_device_status reset");
        if (rc) return rc;
        rc = hip_check(hipStreamSynchronize(st), "rk_device_status sync");
    }
    return rc;
}

int rk_hash_chains(int64_t n_seq, const int32_t* tokens, const int64_t* tok_off,
                   const int64_t* chain_off, uint64_t* chains, void* stream)
{
    if (n_seq < 0) return fail(RK_EINVAL, "rk_hash_chains: n_seq < 0");
    if (n_seq == 0) return RK_OK;
    if (!tokens || !tok_off || !chain_off || !chains)
        return fail(RK_EINVAL, "rk_hash_chains: NULL array");
    int32_t* st = status_word();
    if (!st) return fail(RK_EHIP, "rk_hash_chains: no status word");
    hipStream_t s = (hipStream_t)stream;
    const int64_t waves_per_block = 4;
    int64_t blocks = (n_seq + waves_per_block - 1) / waves_per_block;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(block_fnv_kernel, dim3((unsigned)blocks), dim3(256), 0, s, n_seq, tokens, tok_off,
                       chain_off, chains, st);
    int rc = hip_check(hipGetLastError(), "rk_hash_chains fnv launch");
    if (rc) return rc;
    const int64_t cblocks = (n_seq + kChainWG - 1) / kChainWG;
    hipLaunchKernelGGL(chain_kernel, dim3((unsigned)cblocks), dim3(kChainWG), 0, s, n_seq, tok_off, chain_off,
                       chains);
    return hip_check(hipGetLastError(), "rk_hash_chains chain launch");
}

int rk_table_build(int32_t W, const uint64_t* keys, const int64_t* key_off, uint64_t* tables,
                   int32_t log2_slots, void* stream)
{
    if (W < 1) return fail(RK_EINVAL, "rk_table_build: W < 1");
    if (log2_slots < 4 || log2_slots > 30) return fail(RK_EINVAL, "rk_table_build: log2_slots out of 4..30");
    if (!key_off || !tables) return fail(RK_EINVAL, "rk_table_build: NULL array");
    const uint64_t slots = 1ull << log2_slots;
    for (int32_t j = 0; j < W; ++j) {
        const int64_t n = key_off[j + 1] - key_off[j];
        if (n < 0) return fail(RK_EINVAL, "rk_table_build: key_off not monotone at %d", j);
        if ((uint64_t)n > slots / 2)
            return fail(RK_ETABLEFULL, "rk_table_build: table %d gets %lld keys for %llu slots", j,
                        (long long)n, (unsigned long long)slots);
    }
    if (key_off[W] > 0 && !keys) return fail(RK_EINVAL, "rk_table_build: keys is NULL");
    int32_t* st = status_word();
    if (!st) return fail(RK_EHIP, "rk_table_build: no status word");
    hipStream_t s = (hipStream_t)stream;
    const uint64_t total = slots * (uint64_t)W;
    uint64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(table_clear_kernel, dim3((unsigned)blocks), dim3(256), 0, s, tables, total);
    int rc = hip_check(hipGetLastError(), "rk_table_build clear launch");
    if (rc) return rc;
    for (int32_t j = 0; j < W; ++j) {
        const int64_t n = key_off[j + 1] - key_off[j];
        if (n == 0) continue;
        int64_t b = (n + 255) / 256;
        if (b > 65536) b = 65536;
        hipLaunchKernelGGL(table_insert_kernel, dim3((unsigned)b), dim3(256), 0, s, keys + key_off[j], n,
                           tables + ((uint64_t)j << log2_slots), slots - 1, st);
        rc = hip_check(hipGetLastError(), "rk_table_build insert launch");
        if (rc) return rc;
    }
    return RK_OK;
}

}  // extern "C"
