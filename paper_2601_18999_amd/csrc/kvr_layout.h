// kvr_layout.h - workspace layout of the HIP simulator (internal).
//
// One workspace holds every replica.  Per (replica r, worker i) there is a
// fixed-size block of each region below, addressed by (r * W + i) * stride,
// so the replicas stay independent and one workgroup owns one replica.
//
//   global header   status word, last arrival, queries routed
//   replica headers previous arrival time per replica
//   worker headers  cache counters, marking state, LBGR state, counters
//   node tables     compressed radix-tree nodes (32 B each), node 0 = root
//   arenas          two semispaces of int32 words holding edge tokens and
//                   child arrays; a copying collector compacts live data
//                   into the other semispace when the active one fills
//   leaf arrays     every leaf node, in lexicographic order of root paths
//   U arrays        the RLT candidates: leaves whose leaf token is not
//                   marked, in the same order
//   pending rings   completion records (FIFO per worker)
//   scratch         stack for the digest walk of kvr_stats
//   stats out       kvr_worker_stats staging for kvr_stats
//   stamps          (L-LRU only) last access of every edge token, laid out
//                   like the arenas
//   pins            (continuous batching only) per node, the number of
//                   paths of the worker's running batch through it
//   running rings   (continuous batching only) the end node of each path
//                   of the running batch, oldest first
//   router trees    (approximate router only) per worker a second token
//                   tree, the router's: header, node table, arenas, leaf
//                   list and access stamps, sized for its own budget
#ifndef KVR_LAYOUT_H
#define KVR_LAYOUT_H

#include <stddef.h>
#include <stdint.h>

#include "../../include/kvr.h"

namespace kvr {

constexpr uint32_t kMaxWorkers = 64;
constexpr uint32_t kWave = 64;
#ifndef KVR_MAX_WAVES
#define KVR_MAX_WAVES 8
#endif
constexpr uint32_t kMaxWavesPerBlock = KVR_MAX_WAVES;

// A compressed radix-tree node.  Its edge is `len` tokens at arena[off].
// Tokens of the edge are positions off..off+len-1; the last one is the
// node's leaf token when the node has no children.
// Marks: positions [0, ma) are marked when mphase equals the worker phase;
// one further interval per worker (WorkerHdr::rnode/rlo/rhi/rphase) holds
// the marks left by a phase reset in the middle of an edge.
struct NodeRec {
  int32_t parent;   // -1 for the root, -2 for a free slot
  uint32_t off;     // edge offset in the active arena; free slot: next free id
  int32_t len;      // edge length in tokens
  int32_t nchild;   // number of children
  uint32_t coff;    // child array offset in the active arena (even)
  int32_t ccap;     // child array capacity in entries (token, node) pairs
  uint32_t mphase;  // phase of the prefix marks
  int32_t ma;       // prefix marks [0, ma)
};
static_assert(sizeof(NodeRec) == 32, "node record is 32 bytes");

struct PendRec {      // completion record, 48 B
  int64_t t_route;    // arrival time of the query (us)
  int64_t t_done;     // completion time (us)
  double chat;        // estimated service time (s)
  double base;        // estimated service time + queue load at routing (s)
  double x3;          // queue load at routing (feature 3)
  int32_t h;          // hit tokens on this worker
  int32_t L;          // query length
};
static_assert(sizeof(PendRec) == 48, "pending record is 48 bytes");

struct WorkerHdr {
  // cache
  uint32_t phase, cnt, size, hwm;
  int32_t free_head;
  uint32_t nleaves, nU, U_valid;
  int32_t rnode, rlo, rhi;
  uint32_t rphase;
  uint32_t arena_sel, arena_top, nnodes, pad0;
  // LBGR
  double P;
  double theta[4];
  double Pm[16];
  int64_t tl, Wb;
  uint32_t pend_head, pend_count;
  // continuous batching: ring of the running batch's end nodes
  uint32_t run_head, run_count;
  // counters
  uint64_t routed, prompt_tokens, hit_tokens, matched_tokens;
  uint64_t loads, evictions, forced_resets, completions, pending_max;
  uint64_t lat_sum_us, lat_max_us, gc_runs;
  uint8_t pad[512 - 360];
};
static_assert(sizeof(WorkerHdr) == 512, "worker header is 512 bytes");

struct ReplicaHdr {
  int64_t tprev;          // arrival time of the replica's last query
  uint64_t queries;       // queries routed
  uint64_t route_digest;  // hash chain over (query index, route, hit), kvr_replica_stats
  uint64_t phase_ticks[KVR_PHASES];
  uint64_t pad[11];
};
static_assert(sizeof(ReplicaHdr) == 256, "replica header is 256 bytes");

struct GlobalHdr {
  uint32_t status;       // KVR_DEV_* bits, sticky
  uint32_t err_taken;    // 1 once the first error below was recorded
  int64_t last_arrival;  // arrival time of the last routed query
  // first device-side error: check id, replica, global query index, and
  // three values of the failing check
  uint32_t err_check, err_replica;
  uint64_t err_query;
  int64_t err_val[3];
  uint64_t pad[1];
};
static_assert(sizeof(GlobalHdr) == 64, "global header is 64 bytes");

struct Layout {
  uint32_t R, W, B, maxL, NC, A, PC;
  uint32_t beta;  // batch size of continuous batching (1: single-query processing)
  uint64_t off_global, off_rhdr, off_whdr, off_nodes, off_arena, off_leaf, off_U, off_pend,
      off_scratch, off_stats, off_stamp, off_pin, off_run, total;
  uint64_t node_stride, arena_stride, leaf_stride, pend_stride, scratch_stride, pin_stride, run_stride;
  uint32_t has_stamp;
  // the router's trees (approximate router): budget, node capacity, words per
  // semispace; offsets and strides of their regions
  uint32_t has_router;
  uint32_t RB, NCr, Ar, pad1;
  uint64_t off_rt_hdr, off_rt_nodes, off_rt_arena, off_rt_leaf, off_rt_stamp;
  uint64_t rt_node_stride, rt_arena_stride, rt_leaf_stride;
};

// Constants of one run, passed by value to the kernels.
struct Consts {
  uint64_t seed;
  double alpha_cached, alpha_miss, rho, lr, nlms_eps, rls_p0;
  int64_t dt_us, true_cached_us, true_miss_us, true_out_us;
  int32_t update;
  int32_t evict;
  int32_t router;
  int32_t ca_balance_abs;
  double ca_balance_rel, ca_cache_threshold;
  int32_t cache_responses;  // 1: a path is prompt || response (the last out_len tokens)
  int32_t phase_timers;     // 1: accumulate the routing wave's ticks per part of a step
};

// Arguments of one batch for the step kernel (device pointers).
struct StepArgs {
  char* ws;
  Layout L;
  Consts C;
  const int32_t* tokens;
  const uint64_t* offsets;
  const int64_t* arrival;
  const uint16_t* out_len;
  int32_t* route;
  int32_t* hits;
  int32_t* all_hits;
  uint32_t n;
  uint32_t ucap;  // candidate entries staged in LDS (0: U stays in global memory)
  uint32_t rcap;  // draw words precomputed in LDS per insertion
  uint64_t j0;
  uint32_t pipe;  // 1: the pipelined step kernel (a separate evicting wave)
  uint32_t pad2;
};

inline uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

// Compute the layout for a validated configuration.
inline Layout make_layout(const kvr_config& c) {
  Layout L{};
  L.R = c.num_replicas;
  L.W = c.num_workers;
  L.B = c.cache_tokens;
  L.maxL = c.max_query_tokens;
  // every non-root node holds >= 1 token, and an insertion adds at most a split
  // head and the new leaf before its evictions free space: B + 3 always fits
  L.NC = c.node_capacity ? c.node_capacity : c.cache_tokens + 3u;
  // 32 words per cache token: the live data takes about 1.2 B words, so the
  // collector (one wave copying the live data) runs once per about 31 B
  // words appended; HBM holds this easily (two semispaces of 128 B bytes
  // per worker), and each collection delays its step by tens of us
  uint64_t dflt_arena = 32ull * c.cache_tokens + 2ull * c.max_query_tokens + 4096ull;
  if (dflt_arena > 0xfffffff0ull) dflt_arena = 0xfffffff0ull;
  L.A = c.arena_words ? c.arena_words : (uint32_t)dflt_arena;
  L.A &= ~1u;  // even, so child arrays stay 8-byte aligned in both semispaces
  L.PC = c.pending_capacity;
  L.beta = c.batch_size;
  const uint64_t RW = (uint64_t)L.R * L.W;
  uint64_t o = 0;
  L.off_global = o;
  o = align_up(o + sizeof(GlobalHdr), 256);
  L.off_rhdr = o;
  o = align_up(o + (uint64_t)L.R * sizeof(ReplicaHdr), 256);
  L.off_whdr = o;
  o = align_up(o + RW * sizeof(WorkerHdr), 256);
  L.node_stride = align_up((uint64_t)L.NC * sizeof(NodeRec), 256);
  L.off_nodes = o;
  o += RW * L.node_stride;
  L.arena_stride = align_up(2ull * L.A * 4ull, 256);
  L.off_arena = o;
  o += RW * L.arena_stride;
  L.leaf_stride = align_up((uint64_t)L.NC * 4ull, 256);
  L.off_leaf = o;
  o += RW * L.leaf_stride;
  L.off_U = o;
  o += RW * L.leaf_stride;
  L.pend_stride = align_up((uint64_t)L.PC * sizeof(PendRec), 256);
  L.off_pend = o;
  o += RW * L.pend_stride;
  // the digest walk's stack serves the cache and the router's tree in turn
  const uint64_t ncr = c.router_tree ? (uint64_t)(c.router_tree_tokens ? c.router_tree_tokens : c.cache_tokens) + 3ull
                                     : 0ull;
  L.scratch_stride = align_up((ncr > L.NC ? ncr : (uint64_t)L.NC) * 16ull, 256);
  L.off_scratch = o;
  o += RW * L.scratch_stride;
  L.off_stats = o;
  o = align_up(o + RW * sizeof(kvr_worker_stats), 256);
  // L-LRU only: the last access (global query index) of every edge token,
  // at the same offsets as the tokens in both semispaces
  L.off_stamp = o;
  L.has_stamp = c.evict == KVR_EVICT_LRU;
  if (L.has_stamp) o += RW * L.arena_stride;
  // continuous batching only: in-progress counts per node, running rings
  L.pin_stride = L.beta > 1 ? align_up((uint64_t)L.NC * 4ull, 256) : 0;
  L.off_pin = o;
  o += RW * L.pin_stride;
  L.run_stride = L.beta > 1 ? align_up((uint64_t)(L.beta - 1) * 4ull, 256) : 0;
  L.off_run = o;
  o += RW * L.run_stride;
  // the router's trees: L-LRU token trees like the caches, with their own
  // budget (prompts only, so no query exceeds it)
  L.has_router = c.router_tree != 0;
  L.RB = c.router_tree_tokens ? c.router_tree_tokens : c.cache_tokens;
  L.NCr = L.RB + 3u;
  L.Ar = (uint32_t)((8ull * L.RB + 2ull * c.max_query_tokens + 4096ull) & ~1ull);
  L.pad1 = 0;
  const uint64_t RWr = L.has_router ? RW : 0;
  L.off_rt_hdr = o;
  o = align_up(o + RWr * sizeof(WorkerHdr), 256);
  L.rt_node_stride = align_up((uint64_t)L.NCr * sizeof(NodeRec), 256);
  L.off_rt_nodes = o;
  o += RWr * L.rt_node_stride;
  L.rt_arena_stride = align_up(2ull * L.Ar * 4ull, 256);
  L.off_rt_arena = o;
  o += RWr * L.rt_arena_stride;
  L.rt_leaf_stride = align_up((uint64_t)L.NCr * 4ull, 256);
  L.off_rt_leaf = o;
  o += RWr * L.rt_leaf_stride;
  L.off_rt_stamp = o;
  o += RWr * L.rt_arena_stride;
  L.total = o;
  return L;
}

}  // namespace kvr

#endif  // KVR_LAYOUT_H
