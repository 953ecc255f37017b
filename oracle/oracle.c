/*
 * oracle.c -- plain, slow, CPU reference of KV-aware routing-cost evaluation,
 * routing episodes and the PoA-hat estimator.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The routing product
 * never calls it, and it shares no code, header, table or constant generator
 * with the HIP implementation.
 *
 * Every function follows the plain definition of what it computes:
 *
 *  - Block hash chain: the router identifies cached KV blocks by hashes of
 *    token blocks (Section 2.2, "The Smart Router": a radix tree of blocks per
 *    worker).  Block i of a prompt is tokens [16i, 16i+16); its hash is
 *    h_i = splitmix64(h_{i-1} XOR FNV-1a64(64 little-endian bytes of the 16
 *    int32 tokens)), with h_{-1} = 0.  A hash equal to 0 (the empty-slot
 *    sentinel) is replaced by 0x9E3779B97F4A7C15 both as the key and as the
 *    next chain input.
 *  - Overlap o_ij: the number of leading chain blocks of request i that are
 *    cached on worker j (first-miss scan; Section 2.2, Eq. router-cost, where
 *    the prefill blocks are the blocks not covered by the cached prefix).
 *  - Cost: Eq. router-cost (omega * prefill blocks + active blocks) with an
 *    overload term after Eq. latency-superlinear (Section 5.1), in fp32 with a
 *    fixed operation order and no fused multiply-add:
 *        t1 = w_ov * (float)(P - o)
 *        t2 = w_act * (float)A_j
 *        r  = (float)(A_j + P) / (float)cap
 *        x  = max(r - 1, 0)
 *        cost = (t1 + t2) + w_sat * (x * x)
 *  - Selection: argmin with temperature 0 (Section 2.2, Eq. router-softmax in
 *    the tau -> 0 limit; Section 4.3), lowest worker index on ties; or, per
 *    episode, a softmax sample at temperature tau > 0 (Eq. router-softmax), or
 *    one of the static counterfactual policies of the discussion section
 *    (round robin, uniform random, power of two choices under the same cost).
 *  - Sequential greedy routing = best-response dynamics (Section 4.3): each
 *    request is routed given the loads and caches left by earlier ones.  The
 *    chosen worker's LRU cache touches the prompt's blocks from last to first
 *    (block 0 becomes most recent), inserts the missing ones and evicts least
 *    recently used blocks until it holds at most cache_blocks.  Per episode
 *    the cache may instead follow the KV block manager's frequency policy
 *    (Section 2.2): evict the least frequent block first, frequencies start
 *    at 1, double on a hit and drop by 1 (not below 1) every decay_steps
 *    routing steps.  With memory tiers (LRU only), the k1 most recently
 *    used blocks of a worker form G1, the next k2 G2 and the rest G3
 *    (Section 4.2): the order an exclusive hierarchy keeps when eviction
 *    demotes a tier's least recent block and a hit promotes a block to G1.
 *    The cost then charges the cached prefix per tier (Eq. kv-cost).
 *  - Steps: a step routes up to C/H requests from the ready queue; a request
 *    stays active (its blocks count in A_j) for H steps, so C requests are in
 *    flight once the ramp is over (the semaphore-held concurrency of
 *    Section 7.4).  A conversation's next turn joins the queue when its
 *    previous turn is released.
 *  - Controller 1: a route uses min(w_ov, ctrl_w_ov) when the mean, over the
 *    last ctrl_window routes, of sum_j A_j / (W * cap) exceeds num/den
 *    (integer test), in the spirit of the regime switch of Section 6.3.
 *  - Controller 2, the regime controller of Sections 6.2-6.3: after every
 *    route the chosen worker's latency f(n) = a n + b + d / max(n_sat - n,
 *    1)^beta (Eq. latency-superlinear, n its requests in flight including the
 *    new one) stands in for TTFT; its EWMA (Eq. saturation-signal, weight
 *    alpha per route) sets the regime Below / Transition / Saturated
 *    (Eq. saturation-state) with k-sample hysteresis and margin eps, and the
 *    regime sets the next routes' temperature and overlap weight
 *    (Tab. regime-params).  fp64.
 *  - PoA-hat (Section 6.4, Eq. poa-estimate): per window of consecutive
 *    routes, a frozen cost matrix c_ij = a n_j + b + d / (C_j - n_j)^beta
 *    - w_c o_ij / P_i, where n_j is the window's request count on worker j;
 *    the selfish sum evaluates it at the greedy assignment, and OPT is the
 *    Hungarian optimum on the matrix whose worker columns are replicated
 *    K = ceil(m/W) times (padded to square with zero-cost dummy rows).
 *
 * Floating point: fp32 exactly as written above (build with
 * -ffp-contract=off and no fast-math); sums of costs in fp64, in row order.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

#define ORC_OK 0
#define ORC_EINVAL -1
#define ORC_ENOMEM -2

static const uint64_t ZERO_REMAP = 0x9E3779B97F4A7C15ULL;

/* ------------------------------------------------------------------ hash */

uint64_t orc_fnv1a64(const uint8_t* p, int64_t n)
{
    uint64_t h = 0xcbf29ce484222325ULL;           /* FNV-1a 64-bit offset basis */
    for (int64_t i = 0; i < n; ++i) {
        h ^= (uint64_t)p[i];
        h *= 0x100000001b3ULL;                     /* FNV 64-bit prime */
    }
    return h;
}

uint64_t orc_splitmix64(uint64_t x)
{
    /* Vigna's splitmix64 generator step applied to state x. */
    uint64_t z = x + 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

uint64_t orc_block_fnv(const int32_t* tok16)
{
    uint8_t bytes[64];
    for (int t = 0; t < 16; ++t) {
        uint32_t v = (uint32_t)tok16[t];
        bytes[4 * t + 0] = (uint8_t)(v & 0xffu);
        bytes[4 * t + 1] = (uint8_t)((v >> 8) & 0xffu);
        bytes[4 * t + 2] = (uint8_t)((v >> 16) & 0xffu);
        bytes[4 * t + 3] = (uint8_t)((v >> 24) & 0xffu);
    }
    return orc_fnv1a64(bytes, 64);
}

uint64_t orc_chain_step(uint64_t prev, uint64_t block_fnv)
{
    uint64_t h = orc_splitmix64(prev ^ block_fnv);
    return h == 0 ? ZERO_REMAP : h;
}

/* Hash n_seq token sequences.  Sequence s contributes nblocks[s] blocks read
 * from tokens[tok_off[s] ...]; its chain is written to chains[chain_off[s] ...]. */
int orc_hash_chains(int64_t n_seq, const int32_t* tokens, const int64_t* tok_off,
                    const int32_t* nblocks, const int64_t* chain_off, uint64_t* chains)
{
    for (int64_t s = 0; s < n_seq; ++s) {
        if (nblocks[s] < 0 || (int64_t)nblocks[s] * 16 > tok_off[s + 1] - tok_off[s])
            return ORC_EINVAL;
        if (chain_off[s + 1] - chain_off[s] != nblocks[s])
            return ORC_EINVAL;
        uint64_t h = 0;
        for (int32_t i = 0; i < nblocks[s]; ++i) {
            uint64_t f = orc_block_fnv(tokens + tok_off[s] + 16 * (int64_t)i);
            h = orc_chain_step(h, f);
            chains[chain_off[s] + i] = h;
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------ cost */

float orc_route_cost(float w_ov, float w_act, float w_sat, int32_t cap,
                     int32_t P, int32_t o, int64_t A)
{
    float t1 = w_ov * (float)(P - o);
    float t2 = w_act * (float)A;
    float r = (float)(A + (int64_t)P) / (float)cap;
    float x = fmaxf(r - 1.0f, 0.0f);
    float t3 = w_sat * (x * x);
    return (t1 + t2) + t3;
}

/* The same cost when the cached prefix spans memory tiers (Section 4.2,
 * Eq. kv-cost): of the o cached blocks, o1 lead in G1 and o12 in G1 or G2; a
 * block served from tier t counts tw[t] of a recomputed block, so the prefill
 * term is (P - o) + tw0 o1 + tw1 (o12 - o1) + tw2 (o - o12), summed in that
 * order. */
float orc_route_cost_tiers(float w_ov, float w_act, float w_sat, int32_t cap, int32_t P, int32_t o,
                           int32_t o1, int32_t o12, const float* tw, int64_t A)
{
    float pf = (float)(P - o);
    pf = pf + tw[0] * (float)o1;
    pf = pf + tw[1] * (float)(o12 - o1);
    pf = pf + tw[2] * (float)(o - o12);
    float t1 = w_ov * pf;
    float t2 = w_act * (float)A;
    float r = (float)(A + (int64_t)P) / (float)cap;
    float x = fmaxf(r - 1.0f, 0.0f);
    float t3 = w_sat * (x * x);
    return (t1 + t2) + t3;
}

/* ------------------------------------------------- worker selection policies
 * Random draws are inputs: two uniform 32-bit words (r0, r1) per route.
 */
#define ORC_POLICY_ARGMIN 0
#define ORC_POLICY_SOFTMAX 1
#define ORC_POLICY_ROUND_ROBIN 2
#define ORC_POLICY_RANDOM 3
#define ORC_POLICY_P2C 4

/* Eviction policies of a worker's block cache: least recently used, or the
 * KV block manager's frequency policy of Section 2.2 (frequency 1 on insert,
 * doubled on a hit, minus 1 per time-decay step and never below 1; the least
 * frequent block goes first, the least recently used among equals).  A
 * time-decay step happens every decay_steps routing steps; frequencies stop
 * doubling at ORC_FREQ_CAP. */
#define ORC_EVICT_LRU 0
#define ORC_EVICT_FREQ 1
#define ORC_FREQ_CAP (1 << 20)

/* exp(x) for x <= 0 in float arithmetic (Cody and Waite's argument
 * reduction): x = n ln2 + r with n = floor(x log2(e) + 1/2), ln2 split into a
 * part exact in float times n and a small correction, so |r| <= ln2 / 2;
 * exp(r) by its Taylor series to degree 7 in Horner form (truncation error
 * below 3e-9 relative); times 2^n built in the exponent field.  Below -87 the
 * result is 0; x > 0 or NaN gives 1 (not used by the router). */
float orc_exp_neg(float x)
{
    if (!(x <= 0.0f)) return 1.0f;
    if (x < -87.0f) return 0.0f;
    const float log2e = 1.44269504088896341f;
    const float ln2_hi = 0.693145751953125f;          /* 0x3f317200: 9 low mantissa bits clear */
    const float ln2_lo = 1.42860682030941723212e-6f;  /* ln2 - ln2_hi */
    const float fn = floorf(x * log2e + 0.5f);
    const float r = (x - fn * ln2_hi) - fn * ln2_lo;
    float p = 1.98412698412698412698e-4f;             /* 1/7! */
    p = p * r + 1.38888888888888888889e-3f;           /* 1/6! */
    p = p * r + 8.33333333333333333333e-3f;           /* 1/5! */
    p = p * r + 4.16666666666666666667e-2f;           /* 1/4! */
    p = p * r + 1.66666666666666666667e-1f;           /* 1/3! */
    p = p * r + 0.5f;
    p = p * r + 1.0f;
    p = p * r + 1.0f;
    const int32_t n = (int32_t)fn;                    /* -125 .. 0 */
    union { uint32_t u; float f; } sc;
    sc.u = (uint32_t)(n + 127) << 23;
    return p * sc.f;
}

/* Worker chosen for route t (its index in the episode) from the costs of its
 * W workers:
 *   ARGMIN      least cost, lowest index on ties;
 *   SOFTMAX     with e_j = exp((min_k c_k - c_j) / tau) (Eq. router-softmax
 *               shifted by the minimum cost, the same distribution), the first
 *               j whose running sum e_0 + ... + e_j (float, in worker order)
 *               exceeds u * sum_k e_k, u = (r0 >> 8) / 2^24 in [0, 1); if
 *               rounding leaves none, the last j with e_j > 0;
 *   ROUND_ROBIN t mod W;
 *   RANDOM      floor(r0 * W / 2^32);
 *   P2C         a = floor(r0 * W / 2^32) and b = floor(r1 * (W-1) / 2^32),
 *               moved past a (b >= a: b + 1), two distinct uniform workers;
 *               the cheaper one, the lower index on equal cost.
 * Returns -1 for an unknown policy. */
int32_t orc_select(int32_t policy, float tau, int32_t W, const float* cost, int64_t t, uint32_t r0,
                   uint32_t r1)
{
    if (W < 1) return -1;
    if (policy == ORC_POLICY_ARGMIN) {
        int32_t s = 0;
        for (int32_t j = 1; j < W; ++j)
            if (cost[j] < cost[s]) s = j;
        return s;
    }
    if (policy == ORC_POLICY_SOFTMAX) {
        float cmin = cost[0];
        for (int32_t j = 1; j < W; ++j)
            if (cost[j] < cmin) cmin = cost[j];
        float total = 0.0f;
        for (int32_t j = 0; j < W; ++j) total = total + orc_exp_neg((cmin - cost[j]) / tau);
        const float u = (float)(r0 >> 8) * 5.9604644775390625e-8f;    /* 2^-24 */
        const float thr = u * total;
        float run = 0.0f;
        int32_t last = 0;
        for (int32_t j = 0; j < W; ++j) {
            const float e = orc_exp_neg((cmin - cost[j]) / tau);
            run = run + e;
            if (e > 0.0f) last = j;
            if (run > thr) return j;
        }
        return last;
    }
    if (policy == ORC_POLICY_ROUND_ROBIN) return (int32_t)(t % W);
    if (policy == ORC_POLICY_RANDOM) return (int32_t)(((uint64_t)r0 * (uint64_t)W) >> 32);
    if (policy == ORC_POLICY_P2C) {
        const int32_t a = (int32_t)(((uint64_t)r0 * (uint64_t)W) >> 32);
        if (W == 1) return 0;
        int32_t b = (int32_t)(((uint64_t)r1 * (uint64_t)(W - 1)) >> 32);
        if (b >= a) ++b;
        return (cost[b] < cost[a] || (cost[b] == cost[a] && b < a)) ? b : a;
    }
    return -1;
}

/* ------------------------------------------------- snapshot scoring (sets) */

static int cmp_u64(const void* a, const void* b)
{
    uint64_t x = *(const uint64_t*)a, y = *(const uint64_t*)b;
    return x < y ? -1 : (x > y ? 1 : 0);
}

static int sorted_has(const uint64_t* s, int64_t n, uint64_t key)
{
    int64_t lo = 0, hi = n;            /* binary search in a sorted key array */
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (s[mid] < key) lo = mid + 1; else hi = mid;
    }
    return lo < n && s[lo] == key;
}

/* Score B requests against W fixed key sets: overlap and cost per pair
 * (row-major, W contiguous) and the argmin worker per request. */
int orc_score_batch(int32_t B, int32_t W, const uint64_t* chains, const int64_t* chain_off,
                    const uint64_t* keys, const int64_t* key_off, const int32_t* active,
                    float w_ov, float w_act, float w_sat, int32_t cap,
                    int32_t* overlap, float* cost, int32_t* argmin)
{
    if (B < 0 || W < 1 || cap < 1) return ORC_EINVAL;
    uint64_t** sets = (uint64_t**)calloc((size_t)W, sizeof(uint64_t*));
    if (!sets) return ORC_ENOMEM;
    for (int32_t j = 0; j < W; ++j) {
        int64_t n = key_off[j + 1] - key_off[j];
        sets[j] = (uint64_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(uint64_t));
        if (!sets[j]) return ORC_ENOMEM;
        memcpy(sets[j], keys + key_off[j], (size_t)n * sizeof(uint64_t));
        qsort(sets[j], (size_t)n, sizeof(uint64_t), cmp_u64);
    }
    for (int32_t i = 0; i < B; ++i) {
        const uint64_t* h = chains + chain_off[i];
        int32_t P = (int32_t)(chain_off[i + 1] - chain_off[i]);
        float best = 0.0f;
        int32_t bj = -1;
        for (int32_t j = 0; j < W; ++j) {
            int64_t n = key_off[j + 1] - key_off[j];
            int32_t o = 0;
            while (o < P && sorted_has(sets[j], n, h[o])) ++o;
            float c = orc_route_cost(w_ov, w_act, w_sat, cap, P, o, active[j]);
            overlap[(int64_t)i * W + j] = o;
            cost[(int64_t)i * W + j] = c;
            if (bj < 0 || c < best) { best = c; bj = j; }
        }
        argmin[i] = bj;
    }
    for (int32_t j = 0; j < W; ++j) free(sets[j]);
    free(sets);
    return ORC_OK;
}

/* ------------------------------------------------ LRU cache of one worker
 * Textbook LRU: a chained hash map from key to node plus a doubly linked
 * recency list (oldest at the head, newest at the tail). */

typedef struct {
    uint64_t key;
    int64_t freq;         /* access frequency (frequency eviction only) */
    int64_t tmark;        /* route whose tier marking is in tier (memory tiers only) */
    int32_t tier;         /* 1 = G1, 2 = G2 at route tmark */
    int32_t prev, next;   /* recency list */
    int32_t hnext;        /* bucket chain */
} lru_node;

typedef struct {
    int32_t* bucket;
    uint64_t mask;
    lru_node* node;
    int32_t free_head;
    int32_t oldest, newest;
    int32_t size;
} lru_t;

static int lru_init(lru_t* c, int32_t max_nodes)
{
    uint64_t nb = 1;
    while (nb < (uint64_t)max_nodes * 2) nb <<= 1;
    c->bucket = (int32_t*)malloc(nb * sizeof(int32_t));
    c->node = (lru_node*)malloc((size_t)max_nodes * sizeof(lru_node));
    if (!c->bucket || !c->node) return ORC_ENOMEM;
    for (uint64_t b = 0; b < nb; ++b) c->bucket[b] = -1;
    c->mask = nb - 1;
    for (int32_t i = 0; i < max_nodes; ++i) c->node[i].hnext = i + 1 < max_nodes ? i + 1 : -1;
    c->free_head = max_nodes > 0 ? 0 : -1;
    c->oldest = c->newest = -1;
    c->size = 0;
    return ORC_OK;
}

static void lru_free(lru_t* c)
{
    free(c->bucket);
    free(c->node);
}

static int32_t lru_find(const lru_t* c, uint64_t key)
{
    int32_t i = c->bucket[key & c->mask];
    while (i >= 0 && c->node[i].key != key) i = c->node[i].hnext;
    return i;
}

static void list_unlink(lru_t* c, int32_t i)
{
    int32_t p = c->node[i].prev, n = c->node[i].next;
    if (p >= 0) c->node[p].next = n; else c->oldest = n;
    if (n >= 0) c->node[n].prev = p; else c->newest = p;
}

static void list_append(lru_t* c, int32_t i)
{
    c->node[i].prev = c->newest;
    c->node[i].next = -1;
    if (c->newest >= 0) c->node[c->newest].next = i; else c->oldest = i;
    c->newest = i;
}

/* Make key the most recently used entry; returns 1 if it was inserted.  An
 * inserted entry starts at frequency 1 and a hit doubles the frequency, up to
 * ORC_FREQ_CAP (Section 2.2, the KV block manager's frequency policy; the
 * frequencies only matter under frequency eviction). */
static int lru_touch(lru_t* c, uint64_t key, int* err)
{
    int32_t i = lru_find(c, key);
    if (i >= 0) {
        list_unlink(c, i);
        list_append(c, i);
        c->node[i].freq = 2 * c->node[i].freq < ORC_FREQ_CAP ? 2 * c->node[i].freq : ORC_FREQ_CAP;
        return 0;
    }
    if (c->free_head < 0) { *err = 1; return 0; }
    i = c->free_head;
    c->free_head = c->node[i].hnext;
    c->node[i].key = key;
    c->node[i].freq = 1;
    c->node[i].tmark = -1;
    c->node[i].hnext = c->bucket[key & c->mask];
    c->bucket[key & c->mask] = i;
    list_append(c, i);
    c->size += 1;
    return 1;
}

/* Remove entry i and return its key. */
static uint64_t lru_remove(lru_t* c, int32_t i)
{
    uint64_t key = c->node[i].key;
    list_unlink(c, i);
    int32_t* pp = &c->bucket[key & c->mask];
    while (*pp != i) pp = &c->node[*pp].hnext;
    *pp = c->node[i].hnext;
    c->node[i].hnext = c->free_head;
    c->free_head = i;
    c->size -= 1;
    return key;
}

/* Remove the least recently used entry and return its key. */
static uint64_t lru_evict_oldest(lru_t* c)
{
    return lru_remove(c, c->oldest);
}

/* Frequency eviction: remove the entry of least frequency, the least recently
 * used among equals, and return its key.  Frequencies never drop below 1, so
 * the oldest entry at frequency 1, if any, is that entry; otherwise the
 * minimum is found by a full pass. */
static uint64_t lfu_evict(lru_t* c)
{
    for (int32_t i = c->oldest; i >= 0; i = c->node[i].next)
        if (c->node[i].freq == 1) return lru_remove(c, i);
    int64_t fmin = INT64_MAX;
    for (int32_t i = c->oldest; i >= 0; i = c->node[i].next)
        if (c->node[i].freq < fmin) fmin = c->node[i].freq;
    int32_t i = c->oldest;
    while (c->node[i].freq != fmin) i = c->node[i].next;
    return lru_remove(c, i);
}

/* Memory tiers as consecutive runs of the recency order: the k1 most recently
 * used entries are in G1, the next k2 in G2, the rest in G3.  Marks them for
 * route t. */
static void lru_mark_tiers(lru_t* c, int64_t t, int32_t k1, int32_t k2)
{
    int32_t r = 0;
    for (int32_t i = c->newest; i >= 0 && r < k1 + k2; i = c->node[i].prev, ++r) {
        c->node[i].tmark = t;
        c->node[i].tier = r < k1 ? 1 : 2;
    }
}

/* Leading blocks of h held in tiers 1..max_tier as marked for route t. */
static int32_t lru_tier_overlap(const lru_t* c, const uint64_t* h, int32_t P, int64_t t, int32_t max_tier)
{
    int32_t o = 0;
    for (; o < P; ++o) {
        int32_t i = lru_find(c, h[o]);
        if (i < 0 || c->node[i].tmark != t || c->node[i].tier > max_tier) break;
    }
    return o;
}

/* One time-decay step: every cached entry's frequency drops by 1, to no less
 * than 1. */
static void lfu_decay(lru_t* c)
{
    for (int32_t i = c->oldest; i >= 0; i = c->node[i].next)
        if (c->node[i].freq > 1) c->node[i].freq -= 1;
}

static int32_t lru_overlap(const lru_t* c, const uint64_t* h, int32_t P)
{
    int32_t o = 0;
    while (o < P && lru_find(c, h[o]) >= 0) ++o;
    return o;
}

/* ------------------------------------------------------ routing episode
 * Turn indices and chain offsets are relative to this episode's arrays:
 * turn_off[0] == 0 and chain_off[0] == 0.  n_routes = turn_off[n_conv].
 *
 * totals[0] sum over routes of (P - o) on the chosen worker (recomputed blocks)
 * totals[1] evicted blocks
 * totals[2] sum of P
 * totals[3] routes that used the controller's overlap weight (controller 1), or
 *           that were routed outside the Below regime (controller 2)
 * totals[4] controller activations (inactive -> active transitions), or regime
 *           moves up (controller 2)
 * totals[5] routing steps (index of the last step that routed, plus one)
 * totals[6] sum over routes of o on the chosen worker
 * totals[7] final sum of cached blocks over workers
 *
 * Optional outputs (NULL to skip): final_keys [W * cache_blocks] holds each
 * worker's cached keys from least to most recently used, final_count [W] their
 * number; evicted_keys [evicted_cap] lists evicted keys in eviction order and
 * *n_evicted counts all evictions.
 */
/* Regime controller state after one sample of the latency signal (fp64):
 * ewma = lat for the first sample, else alpha * lat + (1 - alpha) * ewma;
 * Below -> Transition after k consecutive samples with ewma > theta1,
 * Transition -> Saturated after k with ewma >= theta2,
 * Transition -> Below after k with ewma < theta1 - eps,
 * Saturated -> Transition after k with ewma < theta2 - eps;
 * one regime step per sample, counters restart after a change.
 * Returns 1 when the regime moved up. */
int orc_regime_step(const double* rg_d, const int32_t* rg_i, double lat, int64_t sample, double* ewma,
                    int32_t* regime, int32_t* up, int32_t* down)
{
    const double alpha = rg_d[0], theta1 = rg_d[1], theta2 = rg_d[2], eps = rg_d[3];
    const int32_t k = rg_i[0];
    *ewma = sample == 0 ? lat : alpha * lat + (1.0 - alpha) * *ewma;
    const double e = *ewma;
    int moved_up = 0;
    if (*regime == 0) {
        *up = e > theta1 ? *up + 1 : 0;
        if (*up >= k) { *regime = 1; *up = 0; *down = 0; moved_up = 1; }
    } else if (*regime == 1) {
        *up = e >= theta2 ? *up + 1 : 0;
        *down = e < theta1 - eps ? *down + 1 : 0;
        if (*up >= k) { *regime = 2; *up = 0; *down = 0; moved_up = 1; }
        else if (*down >= k) { *regime = 0; *up = 0; *down = 0; }
    } else {
        *down = e < theta2 - eps ? *down + 1 : 0;
        if (*down >= k) { *regime = 1; *up = 0; *down = 0; }
    }
    return moved_up;
}

/* Latency model f(n) = a n + b + d / max(n_sat - n, 1)^beta in fp64. */
double orc_latency(const double* rg_d, const int32_t* rg_i, int64_t n)
{
    const double a = rg_d[4], b = rg_d[5], d = rg_d[6];
    const int32_t beta = rg_i[1], n_sat = rg_i[2];
    double gap = (double)(n_sat - n);
    if (gap < 1.0) gap = 1.0;
    double pw = gap;
    for (int32_t i = 1; i < beta; ++i) pw = pw * gap;
    return (a * (double)n + b) + d / pw;
}

int orc_simulate_episode(int32_t W, int32_t cache_blocks, int32_t H, int32_t routes_per_step,
                         float w_ov, float w_act, float w_sat, int32_t cap,
                         int32_t controller, float ctrl_w_ov, int32_t ctrl_window,
                         int32_t ctrl_num, int32_t ctrl_den,
                         int32_t policy, float tau, const uint32_t* rand,
                         const double* rg_d, const int32_t* rg_i, const float* rg_f, int32_t* route_regime,
                         int32_t evict_policy, int32_t decay_steps,
                         int32_t tier_g1, int32_t tier_g2, const float* tier_w, int32_t* tier_overlap,
                         int32_t n_conv, const int64_t* turn_off, const int32_t* turn_blocks,
                         const int64_t* chain_off, const uint64_t* chains,
                         int32_t* route_turn, int32_t* route_worker, int32_t* route_step,
                         int32_t* route_blocks, int32_t* overlap, float* cost,
                         int32_t* evict_count, uint64_t* evict_digest, uint64_t* last_hash,
                         int64_t* totals,
                         uint64_t* final_keys, int32_t* final_count,
                         uint64_t* evicted_keys, int64_t evicted_cap, int64_t* n_evicted)
{
    if (W < 1 || cache_blocks < 1 || H < 1 || routes_per_step < 1 || cap < 1 || n_conv < 0)
        return ORC_EINVAL;
    if (controller < 0 || controller > 2) return ORC_EINVAL;
    /* the weights of the cost are non-negative (NaN rejected as well) */
    if (!(w_ov >= 0.0f) || !(w_act >= 0.0f) || !(w_sat >= 0.0f) || !(ctrl_w_ov >= 0.0f)) return ORC_EINVAL;
    if (controller == 1 && (ctrl_window < 1 || ctrl_den < 1 || ctrl_num < 0)) return ORC_EINVAL;
    if (controller == 2) {
        if (!rg_d || !rg_i || !rg_f) return ORC_EINVAL;
        if (!(rg_d[0] > 0.0 && rg_d[0] <= 1.0) || !(rg_d[1] <= rg_d[2]) || !(rg_d[3] >= 0.0)) return ORC_EINVAL;
        if (rg_i[0] < 1 || rg_i[1] < 1 || rg_i[1] > 8 || rg_i[2] < 1) return ORC_EINVAL;
        for (int r = 0; r < 3; ++r) {
            if (!(rg_f[r] >= 0.0f) || !(rg_f[3 + r] >= 0.0f)) return ORC_EINVAL;
            if (rg_f[r] > 0.0f && !rand) return ORC_EINVAL;
        }
    }
    if (policy < ORC_POLICY_ARGMIN || policy > ORC_POLICY_P2C) return ORC_EINVAL;
    if (policy == ORC_POLICY_SOFTMAX && !(tau > 0.0f)) return ORC_EINVAL;
    if (evict_policy != ORC_EVICT_LRU && evict_policy != ORC_EVICT_FREQ) return ORC_EINVAL;
    if (evict_policy == ORC_EVICT_FREQ && decay_steps < 1) return ORC_EINVAL;
    const int tiers = tier_g1 > 0;
    if (tier_g1 < 0 || tier_g2 < 0 || (int64_t)tier_g1 + tier_g2 > cache_blocks) return ORC_EINVAL;
    if (tiers && (evict_policy != ORC_EVICT_LRU || !tier_w)) return ORC_EINVAL;
    if (tiers)
        for (int r = 0; r < 3; ++r)
            if (!(tier_w[r] >= 0.0f)) return ORC_EINVAL;
    if (!rand && (policy == ORC_POLICY_SOFTMAX || policy == ORC_POLICY_RANDOM || policy == ORC_POLICY_P2C))
        return ORC_EINVAL;
    const int64_t n_routes = turn_off[n_conv];
    int32_t max_P = 0;
    for (int32_t c = 0; c < n_conv; ++c) {
        int64_t len = chain_off[c + 1] - chain_off[c];
        for (int64_t t = turn_off[c]; t < turn_off[c + 1]; ++t) {
            if (turn_blocks[t] < 0 || turn_blocks[t] > len) return ORC_EINVAL;
            if (turn_blocks[t] > max_P) max_P = turn_blocks[t];
        }
    }

    int rc = ORC_OK;
    lru_t* lru = (lru_t*)calloc((size_t)W, sizeof(lru_t));
    int64_t* A = (int64_t*)calloc((size_t)W, sizeof(int64_t));
    int32_t* o_row = (int32_t*)malloc((size_t)W * sizeof(int32_t));
    int32_t* queue = (int32_t*)malloc((size_t)(n_conv + 1) * sizeof(int32_t));
    int64_t* next_turn = (int64_t*)malloc((size_t)(n_conv + 1) * sizeof(int64_t));
    int32_t* route_conv = (int32_t*)malloc((size_t)(n_routes + 1) * sizeof(int32_t));
    int64_t* step_first = (int64_t*)calloc((size_t)H, sizeof(int64_t));
    int64_t* step_count = (int64_t*)calloc((size_t)H, sizeof(int64_t));
    int64_t* u_ring = (int64_t*)calloc((size_t)(ctrl_window > 0 ? ctrl_window : 1), sizeof(int64_t));
    int64_t* inflight_n = (int64_t*)calloc((size_t)W, sizeof(int64_t));
    if (!lru || !A || !o_row || !queue || !next_turn || !route_conv || !step_first ||
        !step_count || !u_ring || !inflight_n) { rc = ORC_ENOMEM; goto done; }
    for (int32_t j = 0; j < W; ++j)
        if (lru_init(&lru[j], cache_blocks + max_P + 1) != ORC_OK) { rc = ORC_ENOMEM; goto done; }

    for (int k = 0; k < 8; ++k) totals[k] = 0;
    int64_t q_head = 0, q_size = 0;
    const int64_t q_cap = n_conv + 1;
    for (int32_t c = 0; c < n_conv; ++c) {
        next_turn[c] = turn_off[c];
        if (turn_off[c + 1] > turn_off[c]) { queue[(q_head + q_size) % q_cap] = c; ++q_size; }
    }
    int64_t t = 0;            /* routes done */
    int64_t u_sum = 0;        /* sum of the last ctrl_window load samples */
    int prev_active = 0;
    double rg_ewma = 0.0;     /* regime controller: smoothed latency, regime, hysteresis counters */
    int32_t rg_regime = 0, rg_up = 0, rg_down = 0;

    for (int64_t s = 0;; ++s) {
        const int64_t slot = s % H;
        if (s >= H) {                               /* release the routes of step s-H */
            for (int64_t r = step_first[slot]; r < step_first[slot] + step_count[slot]; ++r) {
                A[route_worker[r]] -= route_blocks[r];
                inflight_n[route_worker[r]] -= 1;
                int32_t c = route_conv[r];
                if (next_turn[c] < turn_off[c + 1]) { queue[(q_head + q_size) % q_cap] = c; ++q_size; }
            }
        }
        step_count[slot] = 0;
        if (evict_policy == ORC_EVICT_FREQ && s > 0 && s % decay_steps == 0)
            for (int32_t j = 0; j < W; ++j) lfu_decay(&lru[j]);   /* time-decay step */
        int64_t inflight = 0;
        for (int64_t k = 1; k < H && k <= s; ++k) inflight += step_count[(s - k) % H];
        if (q_size == 0 && inflight == 0) break;
        int64_t n = q_size < routes_per_step ? q_size : routes_per_step;
        step_first[slot] = t;
        step_count[slot] = n;
        if (n > 0) totals[5] = s + 1;

        for (int64_t k = 0; k < n; ++k, ++t) {
            int32_t c = queue[q_head];
            q_head = (q_head + 1) % q_cap;
            --q_size;
            int64_t turn = next_turn[c]++;
            int32_t P = turn_blocks[turn];
            const uint64_t* h = chains + chain_off[c];

            float w_eff = w_ov;
            int32_t pol = policy;
            float tau_eff = tau;
            int active = 0;
            if (controller == 2) {
                w_eff = rg_f[3 + rg_regime];
                tau_eff = rg_f[rg_regime];
                pol = tau_eff > 0.0f ? ORC_POLICY_SOFTMAX : ORC_POLICY_ARGMIN;
                if (rg_regime > 0) totals[3] += 1;
            }
            if (controller == 1 && t >= ctrl_window &&
                (int64_t)ctrl_den * u_sum > (int64_t)ctrl_num * ctrl_window * W * (int64_t)cap)
                active = 1;
            if (active) {
                w_eff = fminf(w_ov, ctrl_w_ov);
                totals[3] += 1;
                if (!prev_active) totals[4] += 1;
            }
            prev_active = active;

            for (int32_t j = 0; j < W; ++j) {
                int32_t o = lru_overlap(&lru[j], h, P);
                float cj;
                if (tiers) {
                    lru_mark_tiers(&lru[j], t, tier_g1, tier_g2);
                    int32_t o1 = lru_tier_overlap(&lru[j], h, P, t, 1);
                    int32_t o12 = lru_tier_overlap(&lru[j], h, P, t, 2);
                    if (tier_overlap) {
                        tier_overlap[(t * W + j) * 2] = o1;
                        tier_overlap[(t * W + j) * 2 + 1] = o12;
                    }
                    cj = orc_route_cost_tiers(w_eff, w_act, w_sat, cap, P, o, o1, o12, tier_w, A[j]);
                } else {
                    cj = orc_route_cost(w_eff, w_act, w_sat, cap, P, o, A[j]);
                }
                o_row[j] = o;
                overlap[t * W + j] = o;
                cost[t * W + j] = cj;
            }
            const int32_t sigma = orc_select(pol, tau_eff, W, cost + t * W, t, rand ? rand[2 * t] : 0u,
                                             rand ? rand[2 * t + 1] : 0u);
            if (route_regime) route_regime[t] = controller == 2 ? rg_regime : 0;

            int err = 0;
            for (int32_t k2 = P - 1; k2 >= 0; --k2) lru_touch(&lru[sigma], h[k2], &err);
            if (err) { rc = ORC_ENOMEM; goto done; }
            int32_t ev = 0;
            uint64_t dig = 0;
            while (lru[sigma].size > cache_blocks) {
                uint64_t key = evict_policy == ORC_EVICT_FREQ ? lfu_evict(&lru[sigma]) : lru_evict_oldest(&lru[sigma]);
                ev += 1;
                dig += orc_splitmix64(key);
                if (evicted_keys && totals[1] + ev - 1 < evicted_cap)
                    evicted_keys[totals[1] + ev - 1] = key;
            }
            A[sigma] += P;
            inflight_n[sigma] += 1;
            if (controller == 2)
                totals[4] += orc_regime_step(rg_d, rg_i, orc_latency(rg_d, rg_i, inflight_n[sigma]), t, &rg_ewma,
                                             &rg_regime, &rg_up, &rg_down);

            int64_t u = 0;
            for (int32_t j = 0; j < W; ++j) u += A[j];
            if (controller == 1) {
                int64_t pos = t % ctrl_window;
                if (t >= ctrl_window) u_sum -= u_ring[pos];
                u_ring[pos] = u;
                u_sum += u;
            }

            route_turn[t] = (int32_t)turn;
            route_worker[t] = sigma;
            route_step[t] = (int32_t)s;
            route_blocks[t] = P;
            route_conv[t] = c;
            evict_count[t] = ev;
            evict_digest[t] = dig;
            last_hash[t] = P > 0 ? h[P - 1] : 0;
            totals[0] += P - o_row[sigma];
            totals[1] += ev;
            totals[2] += P;
            totals[6] += o_row[sigma];
        }
    }
    for (int32_t j = 0; j < W; ++j) {
        totals[7] += lru[j].size;
        if (final_keys && final_count) {
            int32_t n = 0;
            for (int32_t i = lru[j].oldest; i >= 0; i = lru[j].node[i].next)
                final_keys[(int64_t)j * cache_blocks + n++] = lru[j].node[i].key;
            final_count[j] = n;
        }
    }
    if (n_evicted) *n_evicted = totals[1];

done:
    if (lru)
        for (int32_t j = 0; j < W; ++j) lru_free(&lru[j]);
    free(lru); free(A); free(o_row); free(queue); free(next_turn); free(route_conv); free(inflight_n);
    free(step_first); free(step_count); free(u_ring);
    return rc;
}

/* ----------------------------------------------------------------- PoA-hat */

/* Hungarian algorithm (Kuhn-Munkres with row/column potentials), minimising
 * the total cost of a one-to-one assignment of n rows to n columns.
 * cost(i, j) is supplied by the callback; rows and columns are 0-based.
 * On return col_of_row[i] is the column assigned to row i. */
typedef double (*cost_fn)(const void* ctx, int32_t i, int32_t j);

static int hungarian(int32_t n, cost_fn f, const void* ctx, int32_t* col_of_row)
{
    const double INF = 1e300;
    double* u = (double*)calloc((size_t)n + 1, sizeof(double));
    double* v = (double*)calloc((size_t)n + 1, sizeof(double));
    double* minv = (double*)malloc(((size_t)n + 1) * sizeof(double));
    int32_t* p = (int32_t*)calloc((size_t)n + 1, sizeof(int32_t));     /* p[col] = row (1-based) */
    int32_t* way = (int32_t*)calloc((size_t)n + 1, sizeof(int32_t));
    char* used = (char*)malloc((size_t)n + 1);
    if (!u || !v || !minv || !p || !way || !used) {
        free(u); free(v); free(minv); free(p); free(way); free(used);
        return ORC_ENOMEM;
    }
    for (int32_t i = 1; i <= n; ++i) {
        p[0] = i;
        int32_t j0 = 0;
        for (int32_t j = 0; j <= n; ++j) { minv[j] = INF; used[j] = 0; }
        do {
            used[j0] = 1;
            int32_t i0 = p[j0], j1 = 0;
            double delta = INF;
            for (int32_t j = 1; j <= n; ++j) {
                if (used[j]) continue;
                double cur = f(ctx, i0 - 1, j - 1) - u[i0] - v[j];
                if (cur < minv[j]) { minv[j] = cur; way[j] = j0; }
                if (minv[j] < delta) { delta = minv[j]; j1 = j; }
            }
            for (int32_t j = 0; j <= n; ++j) {
                if (used[j]) { u[p[j]] += delta; v[j] -= delta; }
                else minv[j] -= delta;
            }
            j0 = j1;
        } while (p[j0] != 0);
        do {
            int32_t j1 = way[j0];
            p[j0] = p[j1];
            j0 = j1;
        } while (j0 != 0);
    }
    for (int32_t j = 1; j <= n; ++j)
        if (p[j] > 0) col_of_row[p[j] - 1] = j - 1;
    free(u); free(v); free(minv); free(p); free(way); free(used);
    return ORC_OK;
}

typedef struct {
    const float* c;      /* m x W */
    int32_t m, W, K;
} rep_ctx;

static double rep_cost(const void* vctx, int32_t i, int32_t j)
{
    const rep_ctx* x = (const rep_ctx*)vctx;
    if (i >= x->m) return 0.0;                       /* dummy row */
    return (double)x->c[(int64_t)i * x->W + j / x->K];  /* column j is a replica of worker j/K */
}

/* Frozen cost matrix of one window (fp32, fixed op order). */
int orc_poa_matrix(int32_t m, int32_t W, const int32_t* worker, const int32_t* overlap,
                   const int32_t* blocks, float a, float b, float d, int32_t beta,
                   int32_t C_cap, float w_c, float* c_out, int32_t* n_out)
{
    if (m < 0 || W < 1 || beta < 1) return ORC_EINVAL;
    for (int32_t j = 0; j < W; ++j) n_out[j] = 0;
    for (int32_t i = 0; i < m; ++i) {
        if (worker[i] < 0 || worker[i] >= W) return ORC_EINVAL;
        n_out[worker[i]] += 1;
    }
    for (int32_t j = 0; j < W; ++j) {
        int32_t gap = C_cap - n_out[j];
        float g = (float)(gap > 1 ? gap : 1);
        float gb = g;
        for (int32_t k = 1; k < beta; ++k) gb = gb * g;
        float base = (a * (float)n_out[j] + b) + d / gb;
        for (int32_t i = 0; i < m; ++i) {
            float oh = blocks[i] > 0 ? (float)overlap[(int64_t)i * W + j] / (float)blocks[i] : 0.0f;
            c_out[(int64_t)i * W + j] = base - w_c * oh;
        }
    }
    return ORC_OK;
}

/* One window: selfish sum at the greedy assignment and the Hungarian OPT with
 * every worker column replicated K times (K <= 0 means ceil(m/W)). */
int orc_poa_window(int32_t m, int32_t W, const int32_t* worker, const int32_t* overlap,
                   const int32_t* blocks, float a, float b, float d, int32_t beta,
                   int32_t C_cap, float w_c, int32_t K, double* selfish, double* coordinated,
                   int32_t* opt_worker)
{
    if (m < 0 || W < 1) return ORC_EINVAL;
    if (K <= 0) K = (m + W - 1) / W;
    if ((int64_t)K * W < m) return ORC_EINVAL;
    *selfish = 0.0;
    *coordinated = 0.0;
    if (m == 0) return ORC_OK;
    float* c = (float*)malloc((size_t)m * (size_t)W * sizeof(float));
    int32_t* n = (int32_t*)malloc((size_t)W * sizeof(int32_t));
    int32_t N = K * W;
    int32_t* col = (int32_t*)malloc((size_t)N * sizeof(int32_t));
    if (!c || !n || !col) { free(c); free(n); free(col); return ORC_ENOMEM; }
    int rc = orc_poa_matrix(m, W, worker, overlap, blocks, a, b, d, beta, C_cap, w_c, c, n);
    if (rc == ORC_OK) {
        double s = 0.0;
        for (int32_t i = 0; i < m; ++i) s += (double)c[(int64_t)i * W + worker[i]];
        *selfish = s;
        rep_ctx ctx = { c, m, W, K };
        rc = hungarian(N, rep_cost, &ctx, col);
        if (rc == ORC_OK) {
            double o = 0.0;
            for (int32_t i = 0; i < m; ++i) {
                int32_t j = col[i] / K;
                if (opt_worker) opt_worker[i] = j;
                o += (double)c[(int64_t)i * W + j];
            }
            *coordinated = o;
        }
    }
    free(c); free(n); free(col);
    return rc;
}

/* Windows of `window` consecutive routes (the last one may be shorter). */
int orc_poa_windows(int64_t n_routes, int32_t W, int32_t window, const int32_t* worker,
                    const int32_t* overlap, const int32_t* blocks, float a, float b, float d,
                    int32_t beta, int32_t C_cap, float w_c, int32_t K,
                    double* selfish_out, double* coord_out)
{
    if (window < 1) return ORC_EINVAL;
    int64_t nw = (n_routes + window - 1) / window;
    for (int64_t w = 0; w < nw; ++w) {
        int64_t r0 = w * window;
        int32_t m = (int32_t)(n_routes - r0 < window ? n_routes - r0 : window);
        int rc = orc_poa_window(m, W, worker + r0, overlap + r0 * W, blocks + r0, a, b, d, beta,
                                C_cap, w_c, K, &selfish_out[w], &coord_out[w], NULL);
        if (rc != ORC_OK) return rc;
    }
    return ORC_OK;
}
