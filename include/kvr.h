/*
 * kvr.h - C ABI of the batched KV-cache routing / eviction simulator.
 *
 * The library simulates R independent replicas of the online problem of
 * Sec. 3.1 (Eqs. 1-3, Table 1): M = W workers, each with a prefix-sharing
 * token cache of B tokens, receive an ordered stream of queries q_j.  For
 * every query and every replica the library
 *   1. applies completions and load decay (Algorithm 2, update and decay
 *      threads; Sec. 4.2 "Queue Load Estimation"),
 *   2. computes h_ij, the longest prefix of q_j present in worker i's cache
 *      (Sec. 3.2 "Cache Matching"), for every worker,
 *   3. routes q_j to argmin_i of the LBGR score (Algorithm 2, routing
 *      thread; Eq. LBGR-score), lowest index on ties, and adds the estimated
 *      service time to that worker's load (Eq. 2 with the estimate),
 *   4. inserts q_j into the routed worker's cache with RLT (Algorithm 1):
 *      mark every token of the path, reset the marking set when it would
 *      exceed B, and evict a uniformly random unmarked leaf token before
 *      loading a missing token into a full cache (Eq. 3: no other cache
 *      changes); or, with evict = KVR_EVICT_LRU, with L-LRU (Sec. 3.2):
 *      every access stamps the tokens of its path and the leaf token
 *      accessed least recently is evicted.
 * Replicas see the same stream and differ only in the random key of RLT.
 *
 * Conventions
 *   - Every pointer named d_* is a device pointer (e.g. a torch tensor's
 *     data_ptr()) on the device current when kvr_init_replicas was called.
 *     h_* pointers are host memory.  The caller owns every buffer it passes,
 *     including the workspace; the library owns only the small host context.
 *   - kvr_route_batch is asynchronous on the context's stream (a hipStream_t
 *     given at init; NULL = the default stream).  Its outputs are valid after
 *     that stream has been synchronised; kvr_stats and kvr_check synchronise.
 *   - A batch is a transport unit only: query k of a batch has global index
 *     j0 + k, where j0 is the number of queries already routed, so splitting
 *     a stream into batches differently gives identical results.
 *   - Errors are status codes; nothing is thrown across the ABI.  Errors the
 *     host can see (bad configuration, bad arguments, NULL pointers) return
 *     before any device work.  Errors only the device can see (a query of
 *     length 0 or above max_query_tokens, with cache_responses a path no
 *     longer than its response, a negative token, decreasing
 *     arrival times, a full completion ring, a full node table or arena) set
 *     a sticky status word in the workspace: an invalid batch is rejected
 *     as a whole before any state changes (KVR_EINVAL), a capacity overflow
 *     stops the replica where it happened (KVR_ECAPACITY; re-initialise).
 *     kvr_check / kvr_stats report it, and later kvr_route_batch calls
 *     return KVR_ESTATE once the host has seen it.
 */
#ifndef KVR_H
#define KVR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVR_ABI_VERSION 8u

typedef enum kvr_status {
  KVR_OK = 0,
  KVR_EINVAL = -1,    /* invalid configuration, argument or batch content */
  KVR_ENOMEM = -2,    /* workspace too small */
  KVR_EDEVICE = -3,   /* HIP runtime error (no device, launch failure) */
  KVR_ECAPACITY = -4, /* a device-side capacity was exceeded */
  KVR_ESTATE = -5     /* the context is in an error state */
} kvr_status;

enum { KVR_EVICT_RLT = 0, KVR_EVICT_LRU = 1 }; /* L-LRU: Sec. 3.2; at most 2^32 - 1 queries per context */
/* Routers: LBGR (Algorithm 2) and the baselines of Sec. 5: uniformly random
 * (word 0 of Philox4x64-10, key (seed, replica), counter (query index, 0, 0,
 * 1), times W, high 64 bits), round robin over the global query index, and
 * cache-aware: the least loaded worker (fewest queries in flight) when the
 * loads are imbalanced, else the highest hit when its share of the query
 * exceeds a threshold, else the worker with the fewest cached tokens; ties
 * go to the lowest index. */
enum { KVR_ROUTE_LBGR = 0, KVR_ROUTE_RANDOM = 1, KVR_ROUTE_ROUND_ROBIN = 2, KVR_ROUTE_CACHE_AWARE = 3 };
enum { KVR_UPD_NLMS = 0, KVR_UPD_RLS = 1, KVR_UPD_NONE = 2 };

/* Device status bits (kvr_check reports the first one as a kvr_status). */
enum {
  KVR_DEV_BAD_LENGTH = 1u,   /* a query of length 0 or > max_query_tokens, or a
                                path no longer than its cached response     */
  KVR_DEV_BAD_TOKEN = 2u,    /* a negative token id                        */
  KVR_DEV_BAD_ARRIVAL = 4u,  /* arrival times decrease                     */
  KVR_DEV_PENDING_FULL = 8u, /* completion ring of a worker is full        */
  KVR_DEV_NODES_FULL = 16u,  /* node table of a worker is full             */
  KVR_DEV_ARENA_FULL = 32u,  /* token/child arena of a worker is full      */
  KVR_DEV_INTERNAL = 64u     /* an internal consistency check failed       */
};

typedef struct kvr_config {
  uint32_t abi_version;      /* KVR_ABI_VERSION                                    */
  uint32_t struct_size;      /* sizeof(kvr_config)                                 */
  uint32_t num_replicas;     /* R >= 1                                             */
  uint32_t num_workers;      /* W = M of Sec. 3.1, 1..64                           */
  uint32_t cache_tokens;     /* B_i (same for all workers), >= 1                   */
  uint32_t max_query_tokens; /* bound on |q_j|: 1..min(cache_tokens, 16384)        */
  uint64_t seed;             /* Philox key word 0; key word 1 = replica index      */
  int32_t evict;             /* KVR_EVICT_*                                        */
  int32_t router;            /* KVR_ROUTE_*                                        */
  int32_t update;            /* KVR_UPD_*                                          */
  uint32_t pending_capacity; /* completion ring per (replica, worker), >= 1; 65536 by default */
  uint32_t node_capacity;    /* nodes per (replica, worker); 0 = cache_tokens + 3  */
  uint32_t arena_words;      /* words per semispace per (replica, worker), 0 = default
                                min(32*B + 2*max_query_tokens + 4096, 2^32 - 16);
                                else >= B + 2*max_q + 64                           */
  double alpha_cached;       /* s per 1k cached tokens (App. A: 0)                 */
  double alpha_miss;         /* s per 1k missed tokens (App. A: 1)                 */
  double rho;                /* load decay factor (App. A: 31/32), in (0, 1]       */
  int64_t decay_interval_us; /* decay interval (App. A: 20 ms), > 0                */
  double lr;                 /* NLMS step / RLS forgetting factor (App. A: 0.992)  */
  double nlms_eps;           /* NLMS regulariser (1e-9)                            */
  double rls_p0;             /* RLS initial inverse correlation scale (100)        */
  int64_t true_cached_us;    /* observed-latency model: us per cached token (0)    */
  int64_t true_miss_us;      /* us per missed token (1000)                         */
  int64_t true_out_us;       /* us per output token (10000)                        */
  int32_t ca_balance_abs;    /* cache-aware: imbalanced when max - min in flight > this (32) */
  int32_t pad0;
  double ca_balance_rel;     /* ... and max > this * min (1.0001)                  */
  double ca_cache_threshold; /* cache-aware: highest hit / |q| above this (0.5)    */
  /* 0 (default): a query is its prompt q_j and only the prompt is cached.
   * 1: a query is the complete token path Gamma_j = q_j || a_j of Sec. 3.2
   * ("Cache Matching and Arrival Model"): its last out_len[j] tokens are the
   * response a_j (out_len = 4 when d_out_len is NULL).  The match h_ij, the
   * routing features, the hit counts and the observed-latency cost use the
   * prompt, which is all the router sees; the insertion and its evictions
   * take the whole path.  Every path must then be longer than its response
   * (a prompt of >= 1 token), and max_query_tokens bounds the path. */
  int32_t cache_responses;
  /* Continuous batching with batch size beta (Sec. 3.2, Theorem 2): the
   * beta - 1 queries routed to a worker before the one being inserted form
   * its running batch, and no token on their paths is evicted; a path leaves
   * the running batch when beta - 1 later queries have been routed to that
   * worker.  1 (default) = single-query processing, where only the
   * insertion point is protected.  1..256, and batch_size *
   * max_query_tokens <= cache_tokens (the paper's assumption beta * L_max <=
   * B, so a full cache always has an evictable leaf).  Matching, routing and
   * the observed latency do not change. */
  int32_t batch_size;
  /* 0 (default): the router's hit estimate is the exact match h_ij on worker
   * i's cache.  1: the approximate router tree of App. E: the router keeps a
   * token tree of its own per worker, holding the prompts routed there
   * (inserted when routed; the router never sees a response) under L-LRU
   * eviction with a budget of router_tree_tokens tokens (0 = cache_tokens,
   * else max_query_tokens..2^30).  The scores, the routing decision, the
   * load estimate's features and d_all_hits use the estimate from that tree;
   * the observed latency, d_hits and the hit counters use the routed
   * worker's true match.  At most 2^32 - 1 queries per context (its access
   * stamps are 32-bit query indices). */
  int32_t router_tree;
  uint32_t router_tree_tokens;
  /* 1: the step kernel also accumulates, per replica, real-time counter
   * ticks (100 MHz) spent by its routing wave in each part of a step
   * (kvr_replica_stats.phase_ticks); only with evict = KVR_EVICT_RLT,
   * router_tree = 0 and batch_size = 1.  0 (default): no timing. */
  int32_t phase_timers;
  uint32_t pad1;
} kvr_config;

/* Final per-(replica, worker) state and counters (kvr_stats). */
typedef struct kvr_worker_stats {
  uint64_t routed, prompt_tokens, hit_tokens, matched_tokens;
  uint64_t loads, evictions, phase, cnt, forced_resets, resident;
  uint64_t digest_sum, digest_xor, marked_count, marked_sum;
  uint64_t completions, pending_depth, pending_max;
  uint64_t latency_sum_us, latency_max_us;
  int64_t backlog_us, last_decay_us;
  double load_est;
  double theta[4];
  uint64_t nodes, gc_runs; /* layout-dependent, informative only */
  /* the router's tree of this worker (router_tree = 1; else 0): tokens held,
   * path-hash digest (as for the cache), L-LRU evictions */
  uint64_t router_resident, router_digest_sum, router_digest_xor, router_evictions;
} kvr_worker_stats;

/* Parts of a step timed with phase_timers = 1 (kvr_replica_stats.phase_ticks):
 * ticks of the routing wave (0-8) and, when a separate evicting wave runs
 * the evictions of each insertion while the routing wave goes on to the
 * next query, of the evicting wave (9-11, 17) and of the helper waves,
 * summed over them (12-16). */
enum {
  KVR_PHASE_ROUTE = 0,        /* scores, argmin and commit (Algorithm 2 routing thread) */
  KVR_PHASE_STAGE_WAIT = 1,   /* waiting for the next query's staging                  */
  KVR_PHASE_MARK = 2,         /* RLT insertion: marking walk over the cached part      */
  KVR_PHASE_LOAD = 3,         /* split, new leaf's rank, edge copy, tree and list edits */
  KVR_PHASE_EVICT = 4,        /* evictions of the loaded tokens (Algorithm 1)          */
  KVR_PHASE_FINISH = 5,       /* marks of the loaded tokens, cache header              */
  KVR_PHASE_MATCH = 6,        /* h of the next query (routed worker), any left by helpers */
  KVR_PHASE_JOIN = 7,         /* waiting for the other workers' h of the next query    */
  KVR_PHASE_EVICTOR_WAIT = 8, /* waiting for the evicting wave                         */
  KVR_PHASE_E_EVICT = 9,      /* evicting wave: evictions                              */
  KVR_PHASE_E_FINISH = 10,    /* evicting wave: marks of the loaded tokens, header     */
  KVR_PHASE_E_IDLE = 11,      /* evicting wave: waiting for the next insertion         */
  KVR_PHASE_H_STAGE = 12,     /* helper waves (summed): staging the next query         */
  KVR_PHASE_H_WAIT = 13,      /* helper waves: waiting for the routing wave            */
  KVR_PHASE_H_DRAW = 14,      /* helper waves: draw words (Philox4x64-10)              */
  KVR_PHASE_H_OTHER = 15,     /* helper waves: completions, decay, new leaf's rank     */
  KVR_PHASE_H_MATCH = 16,     /* helper waves: h of the next query on the other workers */
  KVR_PHASE_E_MATCH = 17,     /* evicting wave: the routed worker's h of the next query */
  KVR_PHASES = 18
};

/* Per-replica state and counters (kvr_stats): the Sec. 5 metrics summed over
 * the replica's workers, and a digest of its routing decisions.
 * route_digest is the hash chain D_0 = 0,
 *   D_(j+1) = mix64(mix64(D_j + G*(j+1)) + ((route_j << 32) | hit_j)),
 * over the replica's queries j = 0, 1, ... in stream order, where route_j is
 * the routed worker, hit_j = h of the routed worker (as uint32), G =
 * 0x9E3779B97F4A7C15 and mix64 the SplitMix64 finaliser (z ^= z >> 30;
 * z *= 0xBF58476D1CE4E5B9; z ^= z >> 27; z *= 0x94D049BB133111EB;
 * z ^= z >> 31), all modulo 2^64: two runs route identically exactly when
 * the chains agree (up to hash collisions). */
typedef struct kvr_replica_stats {
  uint64_t queries;       /* queries routed for this replica                         */
  uint64_t route_digest;  /* D_queries                                               */
  uint64_t prompt_tokens, hit_tokens, matched_tokens; /* sums over the workers      */
  uint64_t loads, evictions, completions;
  uint64_t latency_sum_us, latency_max_us; /* observed-latency model (sum, maximum) */
  int64_t last_arrival_us;               /* arrival time of the last query routed   */
  uint64_t phase_ticks[KVR_PHASES];      /* phase_timers = 1: ticks per part, else 0 */
} kvr_replica_stats;

typedef struct kvr_ctx kvr_ctx;

/* Fill *cfg with the paper's constants (App. A) and the defaults above for
 * the given sizes.  Pure host function. */
void kvr_config_default(kvr_config* cfg, uint32_t num_replicas, uint32_t num_workers,
                        uint32_t cache_tokens, uint32_t max_query_tokens);

/* Bytes of device workspace kvr_init_replicas needs for *cfg.  Pure host
 * function, no device call.  KVR_EINVAL for an invalid configuration. */
kvr_status kvr_workspace_size(const kvr_config* cfg, size_t* bytes);

/* Lay the replicas out in d_workspace (>= kvr_workspace_size bytes, caller
 * owned, any content) and initialise them on hip_stream (a hipStream_t, or
 * NULL) in the initial state of Sec. 3.1 (Table 1): every cache S_i empty,
 * every load P_i = 0; for RLT the marking set of Algorithm 1 empty (T = {},
 * phase 1); for LBGR (Algorithm 2) the load estimate and residual model at
 * 0 and no pending completion.  On success *out is a new context (free with
 * kvr_destroy).  Asynchronous. */
kvr_status kvr_init_replicas(const kvr_config* cfg, void* d_workspace, size_t bytes,
                             void* hip_stream, kvr_ctx** out);

/* Route n queries for every replica (Algorithm 2 routing + Algorithm 1
 * insertion).  d_tokens: concatenated token ids (int32, >= 0); d_offsets:
 * n+1 uint64 offsets into d_tokens (d_offsets[0] may be non-zero);
 * d_arrival_us: n arrival times in us, non-decreasing, also across calls;
 * d_out_len: n output lengths, or NULL for 4 (the paper's default).
 * Outputs (each optional, NULL to skip): d_route[r*n + k] = routed worker
 * of query k for replica r; d_hits[r*n + k] = h of the routed worker;
 * d_all_hits[(r*n + k)*W + i] = h_ik for every worker.  n = 0 is a no-op.
 * Asynchronous on the context's stream. */
kvr_status kvr_route_batch(kvr_ctx* ctx, uint32_t n, const int32_t* d_tokens,
                           const uint64_t* d_offsets, const int64_t* d_arrival_us,
                           const uint16_t* d_out_len, int32_t* d_route, int32_t* d_hits,
                           int32_t* d_all_hits);

/* Synchronise the stream and report the metrics of Sec. 5 (hit tokens,
 * prompt tokens, observed latency, evictions, loads) with the state they
 * come from: h_replicas[r] (host memory, room for replica_count entries)
 * receives replica r's kvr_replica_stats, h_workers[r*W + i] (room for
 * worker_count entries) worker i's kvr_worker_stats, including the
 * path-hash digest of its cache.  Either pointer may be NULL (that part is
 * skipped).  KVR_EINVAL, with nothing written, when a non-NULL buffer holds
 * fewer than R (resp. R*W) entries.  Returns the device status as kvr_check
 * does (the entries are written also when it is an error). */
kvr_status kvr_stats(kvr_ctx* ctx, kvr_replica_stats* h_replicas, size_t replica_count,
                     kvr_worker_stats* h_workers, size_t worker_count);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * records as kvr_stats, computed without allocating anything and without the
 * workspace's statistics scratch.  The digest walks use a static device array
 * of the library (32 MiB per device, held until the process ends): workers
 * are processed in groups that fit it, and a configuration whose single
 * worker needs more (16 bytes per node of its tree, plus its record) is
 * refused with KVR_EINVAL.  h_workers is required (the replica sums come
 * from it); h_replicas may be NULL.  Every call on a device shares that
 * array: calls that overlap on one device (other threads, other contexts on
 * the same device) race and must be serialised by the caller.  Synchronous;
 * returns the device status as kvr_check does. */
kvr_status kvr_stats_noalloc(kvr_ctx* ctx, kvr_replica_stats* h_replicas, size_t replica_count,
                             kvr_worker_stats* h_workers, size_t worker_count);

/* Synchronise the stream and return the sticky device status as a
 * kvr_status; *h_bits (optional) receives the raw KVR_DEV_* bits. */
kvr_status kvr_check(kvr_ctx* ctx, uint32_t* h_bits);

/* Number of queries routed so far (the global index of the next query). */
uint64_t kvr_queries_done(const kvr_ctx* ctx);

/* Free the host context.  Does not free or touch the caller's workspace. */
void kvr_destroy(kvr_ctx* ctx);

/* Message for the last failure on this thread ("" if none). */
const char* kvr_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KVR_H */
