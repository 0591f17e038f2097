// kvr_api.cpp - host side of the C ABI declared in include/kvr.h.
//
// Validates configurations and arguments, computes the workspace layout,
// keeps the small host context (stream, layout, constants, number of
// queries routed) and launches the kernels of kvr_device.hip.  Every device
// buffer belongs to the caller.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstring>
#include <memory>
#include <new>
#include <string>

#include "kvr_layout.h"

namespace kvr {
hipError_t launch_init(char* ws, const Layout& L, double rls_p0, hipStream_t st);
hipError_t launch_step(const StepArgs& a, hipStream_t st);
hipError_t launch_stats(char* ws, const Layout& L, hipStream_t st);
hipError_t set_step_lds_limit(size_t bytes);
hipError_t step_static_lds(size_t* bytes);
size_t step_lds_bytes(uint32_t maxL, uint32_t W, uint32_t ucap, uint32_t rcap, uint32_t path_sets);
size_t step_lds_bytes_pipe(uint32_t maxL, uint32_t W, uint32_t ucap, uint32_t rcap);
hipError_t noalloc_scratch(int device, void** ptr, size_t* bytes);
hipError_t launch_stats_into(char* ws, const Layout& L, uint64_t w0, uint32_t n, uint64_t* fifo, uint64_t fifo_words,
                             kvr_worker_stats* out, hipStream_t st);
}  // namespace kvr

struct kvr_ctx {
  kvr::Layout L;
  kvr::Consts C;
  char* ws;
  hipStream_t stream;
  int device;
  uint64_t queries_done;
  uint32_t seen_bits;  // device status bits already reported to the host
  uint32_t ucap;       // candidate entries the step kernel stages in LDS
  uint32_t rcap;       // draw words the step kernel precomputes in LDS
  uint32_t pipe;       // 1: the pipelined step kernel (a separate evicting wave)
  uint32_t ucap_p;     // its staged candidates
  uint32_t rcap_p;     // its draw words per insertion (two insertions' worth)
  void* scratch;       // the device's static scratch of kvr_stats_noalloc
  size_t scratch_bytes;
};

namespace {

thread_local std::string g_err;

kvr_status fail(kvr_status st, const std::string& msg) {
  g_err = msg;
  return st;
}

kvr_status fail_hip(hipError_t e, const char* what) {
  g_err = std::string(what) + ": " + hipGetErrorString(e);
  return KVR_EDEVICE;
}

bool finite(double x) { return std::isfinite(x); }

kvr_status validate(const kvr_config* c) {
  if (!c) return fail(KVR_EINVAL, "config is NULL");
  if (c->abi_version != KVR_ABI_VERSION) return fail(KVR_EINVAL, "abi_version mismatch");
  if (c->struct_size != sizeof(kvr_config)) return fail(KVR_EINVAL, "struct_size mismatch");
  if (c->num_replicas < 1) return fail(KVR_EINVAL, "num_replicas must be >= 1");
  if (c->num_workers < 1 || c->num_workers > kvr::kMaxWorkers)
    return fail(KVR_EINVAL, "num_workers must be in 1..64");
  if (c->cache_tokens < 1 || c->cache_tokens > (1u << 30))
    return fail(KVR_EINVAL, "cache_tokens must be in 1..2^30");
  if (c->max_query_tokens < 1 || c->max_query_tokens > c->cache_tokens)
    return fail(KVR_EINVAL, "max_query_tokens must be in 1..cache_tokens");
  if (c->max_query_tokens > 16384)
    return fail(KVR_EINVAL, "max_query_tokens above 16384 does not fit the LDS query buffers");
  if (c->evict != KVR_EVICT_RLT && c->evict != KVR_EVICT_LRU) return fail(KVR_EINVAL, "unknown evict policy");
  if (c->router < KVR_ROUTE_LBGR || c->router > KVR_ROUTE_CACHE_AWARE) return fail(KVR_EINVAL, "unknown router");
  if (c->router == KVR_ROUTE_CACHE_AWARE &&
      (c->ca_balance_abs < 0 || !(c->ca_balance_rel >= 0.0) || !(c->ca_cache_threshold >= 0.0)))
    return fail(KVR_EINVAL, "cache-aware thresholds must be >= 0");
  if (c->cache_responses != 0 && c->cache_responses != 1) return fail(KVR_EINVAL, "cache_responses must be 0 or 1");
  if (c->batch_size < 1 || c->batch_size > 256) return fail(KVR_EINVAL, "batch_size must be in 1..256");
  if ((uint64_t)c->batch_size * c->max_query_tokens > c->cache_tokens)
    return fail(KVR_EINVAL, "batch_size * max_query_tokens must not exceed cache_tokens");
  if (c->router_tree != 0 && c->router_tree != 1) return fail(KVR_EINVAL, "router_tree must be 0 or 1");
  if (c->router_tree_tokens != 0 &&
      (c->router_tree_tokens < c->max_query_tokens || c->router_tree_tokens > (1u << 30)))
    return fail(KVR_EINVAL, "router_tree_tokens must be 0 or in max_query_tokens..2^30");
  if (c->router_tree && 8ull * (c->router_tree_tokens ? c->router_tree_tokens : c->cache_tokens) +
                                2ull * c->max_query_tokens + 4096ull >= (1ull << 32))
    return fail(KVR_EINVAL, "router tree too large for 32-bit arena offsets");
  if (c->update != KVR_UPD_NLMS && c->update != KVR_UPD_RLS && c->update != KVR_UPD_NONE)
    return fail(KVR_EINVAL, "unknown update rule");
  if (c->phase_timers != 0 && c->phase_timers != 1) return fail(KVR_EINVAL, "phase_timers must be 0 or 1");
  if (c->phase_timers && (c->evict != KVR_EVICT_RLT || c->router_tree || c->batch_size != 1))
    return fail(KVR_EINVAL, "phase_timers needs RLT eviction, no router tree and batch_size 1");
  if (c->pending_capacity < 1 || c->pending_capacity > (1u << 28))
    return fail(KVR_EINVAL, "pending_capacity must be in 1..2^28");
  if (c->node_capacity != 0 && (c->node_capacity < 2 || c->node_capacity > (1u << 30)))
    return fail(KVR_EINVAL, "node_capacity must be 0 or in 2..2^30");
  const uint64_t min_arena = (uint64_t)c->cache_tokens + 2ull * c->max_query_tokens + 64ull;
  if (c->arena_words != 0 && c->arena_words < min_arena)
    return fail(KVR_EINVAL, "arena_words must be 0 or >= cache_tokens + 2*max_query_tokens + 64");
  // (the default, 32*B + 2*max_q + 4096 capped at 2^32 - 16, is at least
  // min_arena for every cache_tokens <= 2^30)
  if (!finite(c->alpha_cached) || !finite(c->alpha_miss))
    return fail(KVR_EINVAL, "alpha_cached/alpha_miss must be finite");
  if (!finite(c->rho) || !(c->rho > 0.0) || c->rho > 1.0) return fail(KVR_EINVAL, "rho must be in (0, 1]");
  if (c->decay_interval_us <= 0) return fail(KVR_EINVAL, "decay_interval_us must be > 0");
  if (!finite(c->lr) || !(c->lr > 0.0)) return fail(KVR_EINVAL, "lr must be finite and > 0");
  if (!finite(c->nlms_eps) || c->nlms_eps < 0.0) return fail(KVR_EINVAL, "nlms_eps must be >= 0");
  if (!finite(c->rls_p0) || !(c->rls_p0 > 0.0)) return fail(KVR_EINVAL, "rls_p0 must be > 0");
  if (c->true_cached_us < 0 || c->true_miss_us < 0 || c->true_out_us < 0)
    return fail(KVR_EINVAL, "true_*_us must be >= 0");
  if (c->true_cached_us > (1ll << 32) || c->true_miss_us > (1ll << 32) || c->true_out_us > (1ll << 32))
    return fail(KVR_EINVAL, "true_*_us too large");
  return KVR_OK;
}

kvr_status status_from_bits(uint32_t bits) {
  if (bits & (KVR_DEV_BAD_LENGTH | KVR_DEV_BAD_TOKEN | KVR_DEV_BAD_ARRIVAL)) return KVR_EINVAL;
  if (bits & (KVR_DEV_PENDING_FULL | KVR_DEV_NODES_FULL | KVR_DEV_ARENA_FULL)) return KVR_ECAPACITY;
  if (bits) return KVR_ESTATE;
  return KVR_OK;
}

std::string describe_bits(uint32_t bits) {
  std::string s;
  const char* names[] = {"query length out of range", "negative token id", "arrival times decrease",
                         "completion ring full", "node table full", "arena full",
                         "internal consistency check failed"};
  for (int b = 0; b < 7; ++b)
    if (bits & (1u << b)) {
      if (!s.empty()) s += "; ";
      s += names[b];
    }
  return s;
}

}  // namespace

extern "C" {

void kvr_config_default(kvr_config* c, uint32_t R, uint32_t W, uint32_t B, uint32_t maxL) {
  if (!c) return;
  std::memset(c, 0, sizeof(*c));
  c->abi_version = KVR_ABI_VERSION;
  c->struct_size = sizeof(kvr_config);
  c->num_replicas = R;
  c->num_workers = W;
  c->cache_tokens = B;
  c->max_query_tokens = maxL;
  c->seed = 0;
  c->evict = KVR_EVICT_RLT;
  c->router = KVR_ROUTE_LBGR;
  c->ca_balance_abs = 32;
  c->pad0 = 0;
  c->ca_balance_rel = 1.0001;
  c->ca_cache_threshold = 0.5;
  c->cache_responses = 0;
  c->batch_size = 1;
  c->router_tree = 0;
  c->router_tree_tokens = 0;
  c->phase_timers = 0;
  c->pad1 = 0;
  c->update = KVR_UPD_NLMS;
  c->pending_capacity = 65536;
  c->node_capacity = 0;
  c->arena_words = 0;
  c->alpha_cached = 0.0;  // App. A: 0 ms per 1k cached tokens
  c->alpha_miss = 1.0;    // App. A: 1000 ms per 1k missed tokens
  c->rho = 31.0 / 32.0;   // App. A
  c->decay_interval_us = 20000;  // App. A: 20 ms
  c->lr = 0.992;                 // App. A
  c->nlms_eps = 1e-9;
  c->rls_p0 = 100.0;
  c->true_cached_us = 0;
  c->true_miss_us = 1000;
  c->true_out_us = 10000;
}

kvr_status kvr_workspace_size(const kvr_config* cfg, size_t* bytes) {
  kvr_status st = validate(cfg);
  if (st != KVR_OK) return st;
  if (!bytes) return fail(KVR_EINVAL, "bytes is NULL");
  *bytes = (size_t)kvr::make_layout(*cfg).total;
  return KVR_OK;
}

kvr_status kvr_init_replicas(const kvr_config* cfg, void* d_workspace, size_t bytes, void* hip_stream,
                             kvr_ctx** out) {
  kvr_status st = validate(cfg);
  if (st != KVR_OK) return st;
  if (!out) return fail(KVR_EINVAL, "out is NULL");
  *out = nullptr;
  if (!d_workspace) return fail(KVR_EINVAL, "workspace is NULL");
  if (((uintptr_t)d_workspace) % 256 != 0) return fail(KVR_EINVAL, "workspace must be 256-byte aligned");
  kvr::Layout L = kvr::make_layout(*cfg);
  if (bytes < L.total)
    return fail(KVR_ENOMEM, "workspace too small: need " + std::to_string(L.total) + " bytes");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
  // LDS per workgroup: the query buffer plus as much of the candidate list as
  // fits (16 B per entry, at most 8192 entries)
  int lds_max = 0;
  e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return fail_hip(e, "hipDeviceGetAttribute(max LDS per block)");
  size_t static_lds = 0;
  e = kvr::step_static_lds(&static_lds);
  if (e != hipSuccess) return fail_hip(e, "hipFuncGetAttributes(step kernel)");
  static_lds = (static_lds + 255u) & ~(size_t)255u;
  const uint32_t path_sets = L.has_router ? 2u : 1u;
  const size_t qbytes = kvr::step_lds_bytes(L.maxL, L.W, 0, 0, path_sets);
  if (qbytes + static_lds > (size_t)lds_max)
    return fail(KVR_EINVAL, "max_query_tokens does not fit in LDS (" + std::to_string(lds_max) + " bytes)");
  size_t room = (size_t)lds_max - static_lds - qbytes;
  // high halves of the draw words first (4 B each, as many as one query can
  // take, within 3/5 of the room), then candidates
  size_t rcap = room * 3u / 5u / 4u;
  if (rcap > L.maxL) rcap = L.maxL;
  room -= rcap * 4u;
  size_t ucap = room / 16u;
  if (ucap > 8192) ucap = 8192;
  if (ucap < 64) ucap = 0;
  // The dynamic-LDS limit is an attribute of the kernel functions, shared
  // by every context in the process: raise it to all the device allows, so
  // that a context with a smaller query buffer never lowers it under one
  // with a larger buffer.
  const size_t lds = kvr::step_lds_bytes(L.maxL, L.W, (uint32_t)ucap, (uint32_t)rcap, path_sets);
  if (lds > 65536) {
    e = kvr::set_step_lds_limit((size_t)lds_max - static_lds);
    if (e != hipSuccess) return fail_hip(e, "hipFuncSetAttribute(max dynamic LDS)");
  }
  // the pipelined kernel (RLT, prompts only, no router tree, single-query
  // processing): the draw words of two insertions take 2/5 of the room
  const bool pipe = cfg->evict == KVR_EVICT_RLT && !cfg->router_tree && cfg->batch_size == 1 && !cfg->cache_responses;
  size_t rcap_p = 0, ucap_p = 0;
  if (pipe) {
    const size_t qb = kvr::step_lds_bytes_pipe(L.maxL, L.W, 0, 0);
    if (qb + static_lds > (size_t)lds_max)
      return fail(KVR_EINVAL, "max_query_tokens does not fit in LDS (" + std::to_string(lds_max) + " bytes)");
    // (the candidate list is short on these workloads: 512 staged entries
    // first, then the draw words of two whole insertions, then the rest)
    size_t room_p = (size_t)lds_max - static_lds - qb;
    const size_t ufirst = room_p >= 512u * 16u ? 512u * 16u : 0u;
    rcap_p = (room_p - ufirst) / 8u;
    if (rcap_p > L.maxL) rcap_p = L.maxL;
    room_p -= rcap_p * 8u;
    ucap_p = room_p / 16u;
    if (ucap_p > 8192) ucap_p = 8192;
    if (ucap_p < 64) ucap_p = 0;
    if (kvr::step_lds_bytes_pipe(L.maxL, L.W, (uint32_t)ucap_p, (uint32_t)rcap_p) > 65536) {
      e = kvr::set_step_lds_limit((size_t)lds_max - static_lds);
      if (e != hipSuccess) return fail_hip(e, "hipFuncSetAttribute(max dynamic LDS)");
    }
  }
  // the static scratch of kvr_stats_noalloc on this device (its address,
  // looked up once per device, with the device current)
  void* scratch = nullptr;
  size_t scratch_bytes = 0;
  e = kvr::noalloc_scratch(dev, &scratch, &scratch_bytes);
  if (e != hipSuccess) return fail_hip(e, "hipGetSymbolAddress(scratch)");
  kvr_ctx* c = new (std::nothrow) kvr_ctx;
  if (!c) return fail(KVR_ENOMEM, "host allocation failed");
  c->scratch = scratch;
  c->scratch_bytes = scratch_bytes;
  c->pipe = pipe ? 1u : 0u;
  c->ucap_p = (uint32_t)ucap_p;
  c->rcap_p = (uint32_t)rcap_p;
  c->L = L;
  c->C.seed = cfg->seed;
  c->C.alpha_cached = cfg->alpha_cached;
  c->C.alpha_miss = cfg->alpha_miss;
  c->C.rho = cfg->rho;
  c->C.lr = cfg->lr;
  c->C.nlms_eps = cfg->nlms_eps;
  c->C.rls_p0 = cfg->rls_p0;
  c->C.dt_us = cfg->decay_interval_us;
  c->C.true_cached_us = cfg->true_cached_us;
  c->C.true_miss_us = cfg->true_miss_us;
  c->C.true_out_us = cfg->true_out_us;
  c->C.update = cfg->update;
  c->C.evict = cfg->evict;
  c->C.router = cfg->router;
  c->C.ca_balance_abs = cfg->ca_balance_abs;
  c->C.ca_balance_rel = cfg->ca_balance_rel;
  c->C.ca_cache_threshold = cfg->ca_cache_threshold;
  c->C.cache_responses = cfg->cache_responses;
  c->C.phase_timers = cfg->phase_timers;
  c->ws = static_cast<char*>(d_workspace);
  c->stream = static_cast<hipStream_t>(hip_stream);
  c->device = dev;
  c->queries_done = 0;
  c->seen_bits = 0;
  c->ucap = (uint32_t)ucap;
  c->rcap = (uint32_t)rcap;
  e = kvr::launch_init(c->ws, L, cfg->rls_p0, c->stream);
  if (e != hipSuccess) {
    delete c;
    return fail_hip(e, "init kernel launch");
  }
  *out = c;
  return KVR_OK;
}

kvr_status kvr_route_batch(kvr_ctx* ctx, uint32_t n, const int32_t* d_tokens, const uint64_t* d_offsets,
                           const int64_t* d_arrival_us, const uint16_t* d_out_len, int32_t* d_route,
                           int32_t* d_hits, int32_t* d_all_hits) {
  if (!ctx) return fail(KVR_EINVAL, "ctx is NULL");
  if (ctx->seen_bits) return fail(KVR_ESTATE, "context is in an error state: " + describe_bits(ctx->seen_bits));
  if (n == 0) return KVR_OK;
  if (!d_tokens || !d_offsets || !d_arrival_us) return fail(KVR_EINVAL, "tokens, offsets and arrival_us are required");
  if (n > (1u << 30)) return fail(KVR_EINVAL, "batch too large");
  if ((ctx->C.evict == KVR_EVICT_LRU || ctx->L.has_router) && ctx->queries_done + n > 0xffffffffull)
    return fail(KVR_EINVAL, "L-LRU access stamps hold 32-bit query indices: at most 2^32 - 1 queries per context");
  kvr::StepArgs a;
  a.ws = ctx->ws;
  a.L = ctx->L;
  a.C = ctx->C;
  a.tokens = d_tokens;
  a.offsets = d_offsets;
  a.arrival = d_arrival_us;
  a.out_len = d_out_len;
  a.route = d_route;
  a.hits = d_hits;
  a.all_hits = d_all_hits;
  a.n = n;
  a.pipe = ctx->pipe;
  a.pad2 = 0;
  a.ucap = ctx->pipe ? ctx->ucap_p : ctx->ucap;
  a.rcap = ctx->pipe ? ctx->rcap_p : ctx->rcap;
  a.j0 = ctx->queries_done;
  hipError_t e = kvr::launch_step(a, ctx->stream);
  if (e != hipSuccess) return fail_hip(e, "step kernel launch");
  ctx->queries_done += n;
  return KVR_OK;
}

kvr_status kvr_check(kvr_ctx* ctx, uint32_t* h_bits) {
  if (!ctx) return fail(KVR_EINVAL, "ctx is NULL");
  hipError_t e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
  kvr::GlobalHdr g;
  e = hipMemcpy(&g, ctx->ws + ctx->L.off_global, sizeof(g), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return fail_hip(e, "hipMemcpy(status)");
  const uint32_t bits = g.status;
  ctx->seen_bits |= bits;
  if (h_bits) *h_bits = bits;
  kvr_status st = status_from_bits(bits);
  if (st != KVR_OK) {
    std::string msg = describe_bits(bits);
    if (g.err_taken)
      msg += " (first: check " + std::to_string(g.err_check) + ", replica " + std::to_string(g.err_replica) +
             ", query " + std::to_string(g.err_query) + ", values " + std::to_string(g.err_val[0]) + " " +
             std::to_string(g.err_val[1]) + " " + std::to_string(g.err_val[2]) + ")";
    return fail(st, msg);
  }
  return KVR_OK;
}

kvr_status kvr_stats(kvr_ctx* ctx, kvr_replica_stats* h_replicas, size_t replica_count,
                     kvr_worker_stats* h_workers, size_t worker_count) {
  if (!ctx) return fail(KVR_EINVAL, "ctx is NULL");
  const size_t R = ctx->L.R, RW = (size_t)ctx->L.R * ctx->L.W;
  if (h_replicas && replica_count < R)
    return fail(KVR_EINVAL, "h_replicas holds " + std::to_string(replica_count) + " entries, the context has " +
                                std::to_string(R) + " replicas");
  if (h_workers && worker_count < RW)
    return fail(KVR_EINVAL, "h_workers holds " + std::to_string(worker_count) + " entries, the context has " +
                                std::to_string(RW));
  uint32_t bits = 0;
  kvr_status st = kvr_check(ctx, &bits);
  // the per-worker records are needed for the replica sums too
  hipError_t e = kvr::launch_stats(ctx->ws, ctx->L, ctx->stream);
  if (e != hipSuccess) return fail_hip(e, "stats kernel launch");
  e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
  kvr_worker_stats* ws = h_workers;
  std::unique_ptr<kvr_worker_stats[]> own;
  if (!ws) {
    own.reset(new (std::nothrow) kvr_worker_stats[RW]);
    if (!own) return fail(KVR_ENOMEM, "host allocation failed");
    ws = own.get();
  }
  e = hipMemcpy(ws, ctx->ws + ctx->L.off_stats, RW * sizeof(kvr_worker_stats), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return fail_hip(e, "hipMemcpy(stats)");
  if (h_replicas) {
    std::unique_ptr<kvr::ReplicaHdr[]> rh(new (std::nothrow) kvr::ReplicaHdr[R]);
    if (!rh) return fail(KVR_ENOMEM, "host allocation failed");
    e = hipMemcpy(rh.get(), ctx->ws + ctx->L.off_rhdr, R * sizeof(kvr::ReplicaHdr), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpy(replica headers)");
    for (size_t r = 0; r < R; ++r) {
      kvr_replica_stats o;
      std::memset(&o, 0, sizeof(o));
      o.queries = rh[r].queries;
      o.route_digest = rh[r].route_digest;
      o.last_arrival_us = rh[r].tprev;
      for (int k = 0; k < KVR_PHASES; ++k) o.phase_ticks[k] = rh[r].phase_ticks[k];
      for (size_t i = 0; i < ctx->L.W; ++i) {
        const kvr_worker_stats& w = ws[r * ctx->L.W + i];
        o.prompt_tokens += w.prompt_tokens;
        o.hit_tokens += w.hit_tokens;
        o.matched_tokens += w.matched_tokens;
        o.loads += w.loads;
        o.evictions += w.evictions;
        o.completions += w.completions;
        o.latency_sum_us += w.latency_sum_us;
        if (w.latency_max_us > o.latency_max_us) o.latency_max_us = w.latency_max_us;
      }
      h_replicas[r] = o;
    }
  }
  if (st != KVR_OK) return fail(st, describe_bits(bits));
  return KVR_OK;
}

kvr_status kvr_stats_noalloc(kvr_ctx* ctx, kvr_replica_stats* h_replicas, size_t replica_count,
                             kvr_worker_stats* h_workers, size_t worker_count) {
  if (!ctx) return fail(KVR_EINVAL, "ctx is NULL");
  const size_t R = ctx->L.R, RW = (size_t)ctx->L.R * ctx->L.W;
  if (!h_workers) return fail(KVR_EINVAL, "h_workers is NULL (kvr_stats_noalloc needs it)");
  if (worker_count < RW)
    return fail(KVR_EINVAL, "h_workers holds " + std::to_string(worker_count) + " entries, the context has " +
                                std::to_string(RW));
  if (h_replicas && replica_count < R)
    return fail(KVR_EINVAL, "h_replicas holds " + std::to_string(replica_count) + " entries, the context has " +
                                std::to_string(R) + " replicas");
  if (!ctx->scratch) return fail(KVR_EDEVICE, "no static scratch on this device");
  // per worker: the digest walk's FIFO (two words per node the tree can
  // hold, the router's tree included) and its record
  const uint64_t nodes = ctx->L.has_router && ctx->L.NCr > ctx->L.NC ? ctx->L.NCr : ctx->L.NC;
  const uint64_t fifo_words = 2ull * nodes;
  const uint64_t per = fifo_words * 8ull + sizeof(kvr_worker_stats);
  const uint64_t m = ctx->scratch_bytes / per;
  if (m == 0)
    return fail(KVR_EINVAL, "the digest walk of one worker needs " + std::to_string(per) +
                                " bytes of scratch; kvr_stats_noalloc has " + std::to_string(ctx->scratch_bytes) +
                                " (use kvr_stats)");
  uint32_t bits = 0;
  kvr_status st = kvr_check(ctx, &bits);
  uint64_t* fifo = static_cast<uint64_t*>(ctx->scratch);
  kvr_worker_stats* recs =
      reinterpret_cast<kvr_worker_stats*>(static_cast<char*>(ctx->scratch) + m * fifo_words * 8ull);
  for (uint64_t w0 = 0; w0 < RW; w0 += m) {
    const uint32_t n = (uint32_t)(RW - w0 < m ? RW - w0 : m);
    hipError_t e = kvr::launch_stats_into(ctx->ws, ctx->L, w0, n, fifo, fifo_words, recs, ctx->stream);
    if (e != hipSuccess) return fail_hip(e, "stats kernel launch");
    e = hipMemcpyAsync(h_workers + w0, recs, n * sizeof(kvr_worker_stats), hipMemcpyDeviceToHost, ctx->stream);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpyAsync(stats)");
    e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
  }
  if (h_replicas) {
    for (size_t r = 0; r < R; ++r) {
      kvr::ReplicaHdr rh;
      hipError_t e = hipMemcpy(&rh, ctx->ws + ctx->L.off_rhdr + r * sizeof(kvr::ReplicaHdr), sizeof(rh),
                               hipMemcpyDeviceToHost);
      if (e != hipSuccess) return fail_hip(e, "hipMemcpy(replica header)");
      kvr_replica_stats o;
      std::memset(&o, 0, sizeof(o));
      o.queries = rh.queries;
      o.route_digest = rh.route_digest;
      o.last_arrival_us = rh.tprev;
      for (int k = 0; k < KVR_PHASES; ++k) o.phase_ticks[k] = rh.phase_ticks[k];
      for (size_t i = 0; i < ctx->L.W; ++i) {
        const kvr_worker_stats& w = h_workers[r * ctx->L.W + i];
        o.prompt_tokens += w.prompt_tokens;
        o.hit_tokens += w.hit_tokens;
        o.matched_tokens += w.matched_tokens;
        o.loads += w.loads;
        o.evictions += w.evictions;
        o.completions += w.completions;
        o.latency_sum_us += w.latency_sum_us;
        if (w.latency_max_us > o.latency_max_us) o.latency_max_us = w.latency_max_us;
      }
      h_replicas[r] = o;
    }
  }
  // the walks' own consistency checks
  uint32_t bits2 = 0;
  const kvr_status st2 = kvr_check(ctx, &bits2);
  if (st != KVR_OK) return fail(st, describe_bits(bits));
  return st2;
}

uint64_t kvr_queries_done(const kvr_ctx* ctx) { return ctx ? ctx->queries_done : 0; }

void kvr_destroy(kvr_ctx* ctx) { delete ctx; }

const char* kvr_last_error(void) { return g_err.c_str(); }

}  // extern "C"
