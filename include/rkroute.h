/*
 * rkroute.h -- C ABI of the MI355X (gfx950) KV-aware routing library.
 *
 * The library evaluates the per-(request, worker) routing cost of a KV-aware
 * router, routes requests by argmin, runs many independent sequential routing
 * episodes, and estimates the selfish-versus-coordinated cost ratio (PoA-hat).
 * The operations follow "The Price of Anarchy in Disaggregated Inference":
 *
 *   - routing cost c_j = omega * prefill_blocks_j + active_blocks_j
 *     (Section 2.2, Eq. router-cost), where prefill_blocks_j are the prompt
 *     blocks not covered by the longest prefix cached on worker j, found in a
 *     per-worker index of cached blocks (the router's radix tree of blocks);
 *   - deterministic selection at temperature 0: the argmin of the cost
 *     (Section 2.2 after Eq. router-softmax; Section 4.3);
 *   - routing as a congestion game whose players are requests and whose
 *     resources are workers, played by sequential best response
 *     (Section 4.3, Def. routing-game, Eq. routing-cost);
 *   - a superlinear congestion term near capacity (Section 5.1,
 *     Eq. latency-superlinear), here the overload term
 *     w_sat * max(0, (A_j + P)/cap - 1)^2;
 *   - PoA-hat = sum of selfish costs / OPT over a window of requests, OPT the
 *     optimal assignment on a frozen cost matrix whose worker columns are
 *     replicated up to a capacity (Section 6.4, Eq. poa-estimate).
 *
 * Conventions shared by every entry point:
 *   - Array arguments are DEVICE pointers unless a comment says "host".
 *     The caller owns every buffer; the library keeps no pointer after a call
 *     returns.
 *   - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL is the
 *     default stream).  Argument checks happen before any launch; a failed
 *     check launches nothing.
 *   - Calls return an rk_status.  rk_last_error() gives a message for the
 *     last failure on the calling thread.  No exception or abort crosses the
 *     ABI.
 *   - Conditions that only the device can see (an offset array that is not
 *     monotone, a prompt longer than its chain, a full hash table) are
 *     recorded in a per-device status word: kernels stay in bounds, skip or
 *     clamp the offending item, and rk_device_status() reports the bits.
 *   - Block hashes are nonzero uint64 values; 0 marks an empty table slot.
 *   - Counts are int32, offsets int64.
 */
#ifndef RKROUTE_H
#define RKROUTE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    RK_OK = 0,
    RK_EINVAL = -1,        /* invalid argument (checked on the host)          */
    RK_ENOMEM = -2,        /* workspace too small                             */
    RK_EHIP = -3,          /* a HIP runtime call or launch failed             */
    RK_ETABLEFULL = -4,    /* more keys than a table can hold                 */
    RK_EUNSUPPORTED = -5   /* outside the sizes the library supports          */
} rk_status;

/* Device status bits (rk_device_status). */
#define RK_DEV_BAD_OFFSETS   0x1   /* an offset range was negative or out of order      */
#define RK_DEV_SHORT_INPUT   0x2   /* fewer tokens / chain blocks than requested         */
#define RK_DEV_ZERO_KEY      0x4   /* a key equal to the empty marker was skipped        */
#define RK_DEV_TABLE_FULL    0x8   /* an insert found no empty slot                      */
#define RK_DEV_TOO_LARGE     0x10  /* a window or prompt exceeded the launch's maximum   */
#define RK_DEV_NO_CONVERGE   0x20  /* the assignment solver hit its iteration bound      */
#define RK_DEV_BAD_PARAMS    0x40  /* an episode's policy parameters were invalid       */

/* Static message for a status code. */
const char* rk_status_string(int status);
/* Detail of the last failing call on this thread ("" if none). */
const char* rk_last_error(void);
/* Reads (and, if reset != 0, clears) the device status word of the current
 * device after synchronising `stream`.  Returns the bits through *bits. */
int rk_device_status(int reset, int32_t* bits /* host */, void* stream);

/* ------------------------------------------------------------------ hashing
 * rk_hash_chains -- block-hash chains of token sequences.
 * Block i of sequence s is its tokens [16i, 16i+16), hashed as 64 little-endian
 * bytes with FNV-1a 64; the chain is h_i = splitmix64(h_{i-1} XOR fnv_i) with
 * h_{-1} = 0, and a chain value of 0 is replaced by 0x9E3779B97F4A7C15 (both as
 * the key and as the next chain input).  A chained hash identifies the whole
 * prefix up to its block, which is what lets a hash set answer prefix
 * queries of the router's block index (Section 2.2, "The Smart Router").
 *
 *   n_seq      number of sequences (>= 0)
 *   tokens     int32 [tok_off[n_seq]]   token ids
 *   tok_off    int64 [n_seq+1]          sequence s owns tokens[tok_off[s] .. tok_off[s+1])
 *   chain_off  int64 [n_seq+1]          sequence s writes chain_off[s+1]-chain_off[s]
 *                                       hashes to chains[chain_off[s] ..]; it must own at
 *                                       least 16 tokens per hash (a trailing partial
 *                                       block is ignored)
 *   chains     uint64 [chain_off[n_seq]] output
 * Short token ranges set RK_DEV_SHORT_INPUT and leave the missing hashes 0.
 */
int rk_hash_chains(int64_t n_seq, const int32_t* tokens, const int64_t* tok_off,
                   const int64_t* chain_off, uint64_t* chains, void* stream);

/* ----------------------------------------------------------- cached-block tables
 * rk_table_build -- fill W open-addressing tables of cached block hashes.
 * Table j occupies tables[j << log2_slots ..], 2^log2_slots uint64 slots; 0 is
 * an empty slot; a key's home slot is (key & (2^log2_slots - 1)) and collisions
 * probe linearly upward with wrap-around.  Each table is cleared, then the keys
 * keys[key_off[j] .. key_off[j+1]) are inserted (duplicates once, zero keys
 * skipped with RK_DEV_ZERO_KEY).
 *
 *   W          number of tables (>= 1)
 *   keys       uint64 [key_off[W]]
 *   key_off    int64 [W+1], HOST pointer
 *   log2_slots 4..30
 * Returns RK_ETABLEFULL when a table would receive more than half its slots.
 */
int rk_table_build(int32_t W, const uint64_t* keys, const int64_t* key_off /* host */,
                   uint64_t* tables, int32_t log2_slots, void* stream);

/* ------------------------------------------------------------ snapshot scoring */
typedef struct {
    float w_ov;        /* weight of prefill blocks (omega in Eq. router-cost)   >= 0 */
    float w_act;       /* weight of the worker's active blocks                   >= 0 */
    float w_sat;       /* weight of the squared overload above cap               >= 0 */
    int32_t cap_blocks;/* active blocks at which the overload term starts        >= 1 */
} rk_cost_params;

/* Overlap search modes for rk_route_score_batch. */
#define RK_PROBE_PREFIX 0  /* tables are prefix-closed along every chain (a block is cached
                              only with its parent, as in a radix tree of blocks):
                              membership along a chain is monotone and the first
                              miss is found by searching positions out of order
                              (results are unspecified for tables that are not)   */
#define RK_PROBE_SCAN   1  /* any tables: first miss by a scan from block 0         */

/*
 * rk_route_score_batch -- score B requests against W workers' fixed tables.
 * For request i with chain h_0..h_{P-1} and worker j:
 *   o_ij    = number of leading chain blocks present in table j (first miss);
 *   cost_ij = fp32, in this order and without fused multiply-add:
 *             t1 = w_ov * (float)(P - o); t2 = w_act * (float)A_j;
 *             r = (float)(A_j + P) / (float)cap; x = max(r - 1, 0);
 *             cost = (t1 + t2) + w_sat * (x * x)
 *   argmin_i = the j of least cost, lowest j among equal costs.
 * The tables are read-only and no state is kept (Section 2.2, Eq. router-cost;
 * Section 4.3).
 *
 *   B, W          requests (>= 0) and workers (1..1024)
 *   chains        uint64, request i's chain is chains[chain_off[i] .. chain_off[i+1])
 *   chain_off     int64 [B+1]
 *   tables        uint64 [W << log2_slots] in rk_table_build's layout
 *   active_blocks int32 [W]   A_j
 *   overlap_out   int32 [B*W] row-major (W contiguous), or NULL
 *   cost_out      float [B*W] row-major, or NULL
 *   argmin_out    int32 [B], or NULL
 *   probe_mode    RK_PROBE_PREFIX or RK_PROBE_SCAN
 */
int rk_route_score_batch(int32_t B, int32_t W, const uint64_t* chains, const int64_t* chain_off,
                         const uint64_t* tables, int32_t log2_slots,
                         const int32_t* active_blocks, rk_cost_params params, int32_t probe_mode,
                         int32_t* overlap_out, float* cost_out, int32_t* argmin_out,
                         void* stream);

/* ------------------------------------------------------------ global block index
 * The router's index over all workers (the global radix tree of the Smart
 * Router, background section on the Dynamo architecture; best_worker in
 * Alg. adaptive-router).  A chained hash names a whole prefix, so the tree is
 * held as one open-addressing table of 2^log2_slots 16-byte slots
 *   struct { uint64_t key; uint64_t mask; }   (key 0 = empty slot)
 * where bit j of mask is set when worker j caches the block.  A key's home
 * slot is (key & (2^log2_slots - 1)); collisions probe linearly upward one
 * slot at a time with wrap-around.  Worker count is limited to 64 by the mask.
 *
 * rk_index_build -- clear the index and insert worker j's keys
 * keys[key_off[j] .. key_off[j+1]) for j < W (the same key sets as
 * rk_table_build; duplicates once, zero keys skipped with RK_DEV_ZERO_KEY).
 *   W          1..64 (else RK_EUNSUPPORTED)
 *   keys       uint64 [key_off[W]], device
 *   key_off    int64 [W+1], HOST pointer, non-decreasing
 *   index      device buffer of 16 << log2_slots bytes, 16-byte aligned, owned by the caller
 *   log2_slots 4..31
 * Returns RK_ETABLEFULL when key_off[W] - key_off[0] exceeds half the slots.
 */
int rk_index_build(int32_t W, const uint64_t* keys, const int64_t* key_off /* host */,
                   void* index, int32_t log2_slots, void* stream);

/*
 * rk_route_score_index -- rk_route_score_batch against the global index
 * instead of per-worker tables: same o_ij, cost_ij and argmin_i definitions,
 * same output layouts, same probe modes (RK_PROBE_PREFIX requires every
 * worker's set to be prefix-closed along every chain; RK_PROBE_SCAN takes
 * any sets).  The index is read-only.
 *   B, W          requests (>= 0) and workers (1..64, else RK_EUNSUPPORTED)
 *   chains, chain_off, active_blocks, params, outputs as in rk_route_score_batch
 *   index         rk_index_build's layout, 2^log2_slots slots
 */
int rk_route_score_index(int32_t B, int32_t W, const uint64_t* chains, const int64_t* chain_off,
                         const void* index, int32_t log2_slots, const int32_t* active_blocks,
                         rk_cost_params params, int32_t probe_mode,
                         int32_t* overlap_out, float* cost_out, int32_t* argmin_out, void* stream);

/* ------------------------------------------------------------ routing episodes
 * One episode is a sequential greedy routing run (best-response dynamics,
 * Section 4.3) over the conversations conv_begin .. conv_begin+n_conv-1 of the
 * trace arrays:
 *   - a step first releases the requests routed H steps earlier (their blocks
 *     leave A_j; a released conversation turn lets the conversation's next turn
 *     join the ready queue), then routes up to routes_per_step requests from
 *     the head of the queue, one at a time; the queue starts with every
 *     conversation's first turn in conversation order; the episode ends when
 *     the queue is empty and nothing is in flight.  With routes_per_step = C/H
 *     the in-flight count ramps to C and stays there, as a closed-loop client
 *     holding C requests would (Section 7.4);
 *   - a route scores every worker as in rk_route_score_batch against the
 *     worker's LRU cache of blocks, with weight w_ov replaced by
 *     min(w_ov, ctrl_w_ov) when the controller is on and
 *     ctrl_den * (sum of the last ctrl_window samples of sum_j A_j)
 *       > ctrl_num * ctrl_window * W * cap_blocks
 *     (a sample is taken after every route; at least ctrl_window samples are
 *     needed), a load-triggered switch of the overlap weight in the spirit of
 *     Section 6.3;
 *   - with controller = 2 (the regime controller of Sections 6.2-6.3), the
 *     route's temperature and overlap weight come from the current regime r
 *     (regime.tau[r], regime.w_ov[r]; Tab. regime-params): tau = 0 routes by
 *     argmin, tau > 0 by the softmax below, and the episode's policy, tau
 *     and w_ov are not used.  After every route the chosen worker's latency
 *     f(n) = a n + b + d / max(n_sat - n, 1)^beta (Eq. latency-superlinear,
 *     n = its requests in flight including the new one) stands in for TTFT:
 *     ewma = f for the first route, else alpha f + (1 - alpha) ewma
 *     (Eq. saturation-signal); the regime (Eq. saturation-state) moves
 *     Below -> Transition after k consecutive samples with ewma > theta1,
 *     Transition -> Saturated after k with ewma >= theta2, and back down
 *     after k with ewma < theta1 - eps (resp. theta2 - eps), one regime per
 *     sample, counters restarting after a change; all in fp64;
 *   - the worker sigma is chosen by the episode's policy from the W costs of
 *     route t (its index in the episode) and the two random words r0, r1 of
 *     its output row (route_rand[2 * row], route_rand[2 * row + 1]):
 *       RK_POLICY_ARGMIN      least cost, lowest index on ties (temperature 0,
 *                             Section 2.2 and Section 4.3);
 *       RK_POLICY_SOFTMAX     a sample of Eq. router-softmax at temperature
 *                             tau > 0 (cost units): with e_j = exp((min_k c_k
 *                             - c_j) / tau) in float (exp by Cody-Waite
 *                             reduction and a degree-7 Taylor series, each
 *                             operation rounded), the first j whose running
 *                             sum e_0 + ... + e_j exceeds u * sum_k e_k,
 *                             u = (r0 >> 8) / 2^24, else the last j with
 *                             e_j > 0;
 *       RK_POLICY_ROUND_ROBIN t mod W;
 *       RK_POLICY_RANDOM      floor(r0 * W / 2^32);
 *       RK_POLICY_P2C         the cheaper of a = floor(r0 * W / 2^32) and
 *                             b = floor(r1 * (W-1) / 2^32) (+1 when b >= a),
 *                             lower index on equal cost;
 *     the last three are the static counterfactual policies of the
 *     discussion section, under the same cost;
 *   - the chosen worker sigma touches the prompt's blocks from last to first
 *     (block 0 ends most recent), inserting those it lacks, then evicts blocks
 *     until it holds at most cache_blocks; A_sigma += P.  Caches start empty;
 *     blocks stay cached after a request is released.  Eviction order:
 *       RK_EVICT_LRU   least recently used first;
 *       RK_EVICT_FREQ  the KV block manager's frequency policy (Section 2.2):
 *                      a block's frequency is 1 when inserted, doubles on a
 *                      hit (at most RK_FREQ_CAP) and drops by 1, never below
 *                      1, at every time-decay step (the start of each routing
 *                      step s > 0 with s a multiple of decay_steps); the least
 *                      frequent block goes first, the least recently used
 *                      among equals.
 *   - memory tiers (tier_g1 > 0, Section 4.2 and Eq. kv-cost): a worker's
 *     tier_g1 most recently used blocks are in G1, the next tier_g2 in G2 and
 *     the rest in G3 (the order of an exclusive hierarchy that demotes a
 *     tier's least recent block and promotes a hit block to G1).  With o1 and
 *     o12 the leading blocks of the prompt held in G1 and in G1 or G2, the
 *     cost's prefill term becomes, in fp32 and this order,
 *       ((((float)(P - o) + tier_w[0] * o1) + tier_w[1] * (o12 - o1))
 *        + tier_w[2] * (o - o12));
 *     every route then stops the batch (as in RK_PROBE_SCAN) so that later
 *     requests see the new tier boundaries.
 * The queue order, the touch order and the tie rule make every result unique.
 */
typedef struct {
    int64_t conv_begin;      /* first conversation of the episode (index into turn_off) */
    int32_t n_conv;          /* conversations in the episode, >= 0                     */
    int32_t hold_steps;      /* H >= 1                                                 */
    int32_t routes_per_step; /* >= 1                                                   */
    int32_t controller;      /* 0 off, 1 load switch, 2 regime controller (see below)  */
    int32_t ctrl_window;     /* >= 1 when the controller is on                         */
    int32_t ctrl_num;        /* >= 0                                                   */
    int32_t ctrl_den;        /* >= 1                                                   */
    int32_t cap_blocks;      /* >= 1                                                   */
    float   w_ov, w_act, w_sat;   /* >= 0                                              */
    float   ctrl_w_ov;       /* weight used while the controller is active, >= 0       */
    int64_t out_base;        /* first output row of this episode                       */
    int32_t policy;          /* RK_POLICY_*                                            */
    float   tau;             /* softmax temperature, > 0 with RK_POLICY_SOFTMAX        */
    int32_t evict_policy;    /* RK_EVICT_*                                             */
    int32_t decay_steps;     /* routing steps per time-decay step, >= 1 with RK_EVICT_FREQ */
    int32_t tier_g1;         /* memory tiers: blocks in G1 (0 = no tiers), needs
                                RK_EVICT_LRU and a batch with tiers != 0            */
    int32_t tier_g2;         /* blocks in G2, >= 0, tier_g1 + tier_g2 <= cache_blocks;
                                G3 holds the rest of the cache                      */
    float   tier_w[3];       /* prefill weight of a cached block in G1, G2, G3, >= 0 */
    int32_t tier_pad;        /* 0                                                    */
} rk_episode_params;         /* 104 bytes; invalid policy, eviction or tier fields, or a
                                negative or NaN weight (w_ov, w_act, w_sat, ctrl_w_ov),
                                set RK_DEV_BAD_PARAMS and leave the episode's outputs
                                unwritten                                             */

#define RK_EVICT_LRU          0
#define RK_EVICT_FREQ         1
#define RK_FREQ_CAP           (1 << 20)

#define RK_POLICY_ARGMIN      0
#define RK_POLICY_SOFTMAX     1
#define RK_POLICY_ROUND_ROBIN 2
#define RK_POLICY_RANDOM      3
#define RK_POLICY_P2C         4

typedef struct {
    double  alpha;           /* EWMA weight of the newest sample, (0, 1]               */
    double  theta1, theta2;  /* regime thresholds (seconds), theta1 <= theta2           */
    double  eps;             /* hysteresis margin (seconds), >= 0                       */
    int32_t k;               /* consecutive samples for a regime change, >= 1           */
    int32_t beta;            /* exponent of the saturation term, 1..8                   */
    double  a, b, d;         /* latency model (seconds)                                 */
    int32_t n_sat;           /* requests at which the saturation term peaks, >= 1       */
    float   tau[3];          /* temperature per regime (Below, Transition, Saturated)   */
    float   w_ov[3];         /* overlap weight per regime, >= 0                         */
} rk_regime_params;          /* 96 bytes; invalid values set RK_DEV_BAD_PARAMS for the
                                episodes with controller = 2                          */

typedef struct {
    int32_t E;                       /* episodes (>= 0)                                 */
    int32_t W;                       /* workers per episode, 1..64                      */
    int32_t cache_blocks;            /* LRU capacity per worker, >= 1                   */
    int32_t max_blocks;              /* upper bound on any prompt's blocks, 1..8192     */
    int32_t max_conv;                /* upper bound on n_conv of any episode            */
    int32_t max_inflight;            /* upper bound on H * routes_per_step, <= 8192     */
    int32_t max_routes_per_step;     /* upper bound on routes_per_step                  */
    int32_t max_ctrl_window;         /* upper bound on ctrl_window (1 if unused), <= 4096 */
    int32_t probe_mode;              /* RK_PROBE_PREFIX: caches are prefix-closed along
                                        every chain, which holds for chained hashes (a
                                        block is touched and evicted after its children):
                                        the first miss is found by binary search;
                                        RK_PROBE_SCAN: scan from block 0 in 64-block steps */
    int32_t tiers;                   /* nonzero when some episode has tier_g1 > 0: the
                                        launch then keeps tier overlaps in LDS          */
    int32_t max_routes;              /* upper bound on any episode's routes (turns), >= 0 */
    int32_t flags;                   /* 0 (no flags are defined)                        */
    int32_t ws_slots;                /* episode workspaces the workspace holds: 0 (or >= E)
                                        means one per episode; 1 <= ws_slots < E runs the
                                        batch on ws_slots workgroups, each taking the next
                                        episode in index order when it finishes one and
                                        reusing its workspace, so that a batch larger than
                                        device memory runs in one call                   */
    int32_t ws_pad;                  /* 0                                               */
    const rk_episode_params* params; /* [E], device                                     */
    const int64_t* turn_off;         /* turns of conversation c: turn_off[c] .. turn_off[c+1]-1 */
    const int32_t* turn_blocks;      /* prompt blocks P of each turn; a turn's prompt is the
                                        first P blocks of its conversation's chain       */
    const int64_t* chain_off;        /* chain of conversation c: chains[chain_off[c] .. chain_off[c+1]) */
    const uint64_t* chains;          /* block-hash chains (rk_hash_chains)              */
    const uint32_t* route_rand;      /* 2 uniform 32-bit words per output row, read by the
                                        SOFTMAX, RANDOM and P2C policies; may be NULL when
                                        no episode uses them                             */
    rk_regime_params regime;         /* for the episodes with controller = 2            */
} rk_episode_batch;

/* Outputs, one row per route in routing order, written at out_base + t of the
 * episode (any pointer may be NULL). */
typedef struct {
    int32_t* route_turn;      /* [rows]   global turn index routed at t                 */
    int32_t* route_worker;    /* [rows]   sigma                                         */
    int32_t* route_step;      /* [rows]   step index                                    */
    int32_t* route_blocks;    /* [rows]   P                                             */
    int32_t* overlap;         /* [rows*W] o_ij for every worker at routing time         */
    float*   cost;            /* [rows*W] cost_ij                                       */
    int32_t* evict_count;     /* [rows]   blocks evicted by the route                   */
    uint64_t* evict_digest;   /* [rows]   sum of splitmix64(key) over evicted keys      */
    uint64_t* last_hash;      /* [rows]   h_{P-1} of the routed prompt (0 if P == 0)    */
    int64_t* totals;          /* [E*8]    per episode: sum(P - o_sigma), evictions,
                                 sum(P), controller routes, controller activations,
                                 steps, sum(o_sigma), blocks cached at the end; with
                                 controller = 2 the 4th and 5th count routes outside
                                 Below and regime moves up                           */
    int32_t* route_regime;    /* [rows]   regime the route was made in (0 without the
                                 regime controller)                                  */
    int32_t* tier_overlap;    /* [rows*W*2] (o1, o12) per worker with memory tiers (not
                                 written without them)                               */
} rk_episode_outputs;

/* Workspace bytes needed by rk_simulate_episodes for this batch shape, with E
 * episode workspaces (pass min(E, ws_slots) when the batch sets ws_slots). */
size_t rk_simulate_workspace_size(int32_t E, int32_t W, int32_t cache_blocks,
                                  int32_t max_blocks, int32_t max_conv, int32_t max_routes);

/* Run E independent episodes, one workgroup each (Section 4.3: sequential
 * greedy routing; Section 2.2: the router cost and the KV cache it reads).
 * `batch` and `out` are HOST structs holding device pointers; `workspace` is
 * device memory of at least rk_simulate_workspace_size(min(E, ws_slots or E),
 * ...) bytes whose contents need not be initialised: an episode clears the
 * parts of its workspace it uses.  Results do not depend on ws_slots.  Calls
 * that share a workspace must not overlap.  Nonzero flags, ws_slots < 0 or
 * ws_pad != 0: RK_EINVAL.
 * While a worker has not evicted yet (under LRU, in prefix mode), its cached
 * set is kept as runs, one per route that added blocks (the route's blocks
 * past its overlap, found again by a walk over the runs); at its first
 * eviction, and from the start for frequency eviction, memory tiers and
 * RK_PROBE_SCAN, it is kept block by block with its recency.  The results are
 * the same either way. */
int rk_simulate_episodes(const rk_episode_batch* batch /* host */,
                         const rk_episode_outputs* out /* host */,
                         void* workspace, size_t ws_bytes, void* stream);

/* ----------------------------------------------------------------- PoA-hat
 * For each window w of consecutive routes rows win_off[w] .. win_off[w+1]-1
 * (m rows), with n_j the number of the window's routes on worker j:
 *   c_ij = (a * (float)n_j + b) + d / g^beta - w_c * ((float)o_ij / (float)P_i),
 *   g = (float)max(C_cap - n_j, 1), g^beta by repeated fp32 multiplication,
 *   o/P taken as 0 when P = 0  (fp32, fixed order, no fused multiply-add);
 *   selfish_w     = sum_i c_{i,sigma(i)}                               (fp64)
 *   coordinated_w = min over assignments pi with |pi^-1(j)| <= K of
 *                   sum_i c_{i,pi(i)}                                  (fp64)
 * with K = ceil(m / W) (K_fixed = 0) or K_fixed, i.e. the optimum of the
 * frozen matrix with each worker column replicated K times (Section 6.4,
 * Eq. poa-estimate).  Per episode e (windows ep_win_off[e] .. ep_win_off[e+1]-1):
 *   poa_hat_e = sum_w selfish_w / sum_w coordinated_w.
 */
typedef struct {
    float a, b, d;      /* latency model a*n + b + d/(C_cap - n)^beta       */
    int32_t beta;       /* >= 1                                             */
    int32_t C_cap;      /* per-worker capacity of the latency model         */
    float w_c;          /* cache weight                                     */
    int32_t K_fixed;    /* replicas per worker column; 0 = ceil(m/W)        */
} rk_poa_params;

size_t rk_poa_workspace_size(int64_t n_rows, int32_t W);

/*   n_windows    windows (>= 0);  n_episodes  groups of windows (>= 0)
 *   win_off      int64 [n_windows+1], rows of each window (nondecreasing)
 *   ep_win_off   int64 [n_episodes+1], windows of each episode, or NULL
 *   n_rows       rows addressed by win_off (= win_off[n_windows]), host value
 *   max_window   upper bound on any window's m, 1..4096
 *   W            workers, 1..64
 *   route_worker int32 [n_rows]     sigma
 *   overlap      int32 [n_rows*W]   o_ij (row-major)
 *   route_blocks int32 [n_rows]     P_i
 *   selfish_out, coord_out  double [n_windows] (may be NULL)
 *   poa_hat_out  double [n_episodes] (may be NULL)
 */
int rk_poa_estimate(int32_t n_windows, const int64_t* win_off, int32_t n_episodes,
                    const int64_t* ep_win_off, int64_t n_rows, int32_t max_window, int32_t W,
                    const int32_t* route_worker, const int32_t* overlap,
                    const int32_t* route_blocks, rk_poa_params params,
                    double* selfish_out, double* coord_out, double* poa_hat_out,
                    void* workspace, size_t ws_bytes, void* stream);

/* rk_poa_estimate without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, outputs and results as
 * rk_poa_estimate minus workspace and ws_bytes: its scratch (the frozen
 * matrices, the dispatch order and its class counters and, when selfish_out
 * or coord_out is NULL, the window sums) lives in a static device buffer of
 * RK_POA_NOALLOC_BYTES that the library holds on each device it runs on
 * until the process ends.  The
 * call allocates nothing.  A shape whose rk_poa_workspace_size(n_rows, W)
 * exceeds RK_POA_NOALLOC_BYTES returns RK_EUNSUPPORTED before any launch.
 * Every call on one device shares that device's buffer and leaves its
 * contents behind: calls that overlap on one GPU (e.g. on two streams) race,
 * so the caller orders them. */
#define RK_POA_NOALLOC_BYTES (64u << 20)
int rk_poa_estimate_noalloc(int32_t n_windows, const int64_t* win_off, int32_t n_episodes,
                            const int64_t* ep_win_off, int64_t n_rows, int32_t max_window, int32_t W,
                            const int32_t* route_worker, const int32_t* overlap,
                            const int32_t* route_blocks, rk_poa_params params,
                            double* selfish_out, double* coord_out, double* poa_hat_out, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* RKROUTE_H */
