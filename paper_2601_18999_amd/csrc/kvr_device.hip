// kvr_device.hip - gfx950 kernels of the batched KV-cache routing / eviction
// simulator.
//
// One workgroup owns one replica for a whole batch and walks the batch's
// queries in order (the simulation is sequential within a replica, Sec. 3.1:
// the state after query j-1 decides query j).  Per query, in two phases
// separated by workgroup barriers:
//   * phase A, wave 0: the LBGR score of every worker from its load,
//     residual model and h_ij, the longest cached prefix of the query (Sec.
//     3.2 "Cache Matching"); the argmin (lowest index on ties) and the commit
//     on the routed worker (Algorithm 2 routing thread, Eq. LBGR-score, Eq. 2
//     with the estimate), or a baseline router of Sec. 5.  The other waves
//     stage the next query in LDS.
//   * phase B, wave 0: the insertion into the routed worker's cache with RLT
//     (Algorithm 1: marks along the path, phase resets, a uniform draw over
//     the unmarked leaf tokens U for every token loaded into a full cache;
//     Eq. 3: no other cache changes) or L-LRU, then that worker's h for the
//     next query.  The other waves: the draw words of the insertion and the
//     new leaf's rank; completions and load decay at the next arrival, one
//     lane per worker (Algorithm 2, update and decay threads; Sec. 4.2); the
//     next query's h on every other worker, walking each compressed radix
//     tree from the point where the previous match on it can be resumed.

// The cache of a worker is a compressed radix tree: a node holds an edge of
// `len` tokens; its leaf token (when it has no children) is the last one.
// U is kept as an ordered list of candidate leaf nodes in lexicographic
// order of their root paths: rebuilt from the ordered list of all leaves
// when a phase starts, shortened when a candidate's leaf token is marked,
// and updated in place when an eviction exposes the parent as a new leaf
// (the parent inherits the rank of the leaf it replaces).  A draw takes
// index floor(r * |U| / 2^64), r = word 0 of Philox4x64-10 with key
// (seed, replica) and counter (query index, worker, draw index, 0).
//
// With cached responses a query is a complete token path q_j || a_j (Sec.
// 3.2 "Cache Matching and Arrival Model"): the match, the scores and the
// commit see the prompt q_j, the insertion takes the whole path.
//
// Floating point: double, left-to-right sums, built with -ffp-contract=off so
// no multiply-add is fused; the same expressions in the same order as the
// definition, so results are bit-identical to any IEEE implementation that
// evaluates them in that order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "kvr_core.h"

namespace kvr {

// ---------------------------------------------------------------- kernels

// Paths recorded in LDS: entries of worker i at [i * kPathMax, (i+1) * kPathMax)
// of the node, start and end arrays, then one count per worker.
struct PathArea {
  int32_t* base;
  uint32_t W;
  __device__ PathRef of(uint32_t i) const {
    PathRef p;
    p.node = base + (size_t)i * kPathMax;
    p.start = base + (size_t)(W + i) * kPathMax;
    p.end = base + (size_t)(2 * W + i) * kPathMax;
    p.cnt = base + (size_t)3 * W * kPathMax + i;
    return p;
  }
};

__device__ __forceinline__ void count_matched(const Ptrs& P, int32_t h, int32_t* hslot) {
  if (lane_id() == 0) {
    *hslot = h;
    P.hdr->matched_tokens += (uint64_t)h;
  }
}

// Stage q_next[0, Ln) (threads t0, t0 + stride, ...) and fold each thread's
// first position where it differs from q_cur into *ell (LDS minimum), so
// that after the next barrier *ell = LCP(q_cur, q_next).  The stream is read
// in aligned 16-byte blocks of four tokens, eight blocks per thread in flight;
// the first and last block may reach up to three tokens outside the query,
// inside the same aligned 16 bytes, and those are not staged.
template <int kUnroll = 8>  // blocks in flight per thread
__device__ __forceinline__ void stage_next(const int32_t* tokens, uint64_t n0, int32_t Ln, int32_t* qn,
                                           const int32_t* qc, int32_t Lc, uint32_t t0, uint32_t stride,
                                           int32_t* ell) {
  const uintptr_t sa = reinterpret_cast<uintptr_t>(tokens + n0);
  const int32_t lead = (int32_t)((sa & 15u) >> 2);
  const int4* base = reinterpret_cast<const int4*>(sa - (uintptr_t)lead * 4u);
  const uint32_t nb = (uint32_t)((lead + Ln + 3) >> 2);
  int32_t m = Lc < Ln ? Lc : Ln;
  for (uint32_t b = t0; b < nb; b += kUnroll * stride) {
    int4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t blk = b + (uint32_t)u * stride;
      v[u].x = v[u].y = v[u].z = v[u].w = 0;
      if (blk < nb) v[u] = base[blk];
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t blk = b + (uint32_t)u * stride;
      if (blk < nb) {
        const int32_t t4[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
        const int32_t x0 = (int32_t)blk * 4 - lead;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int32_t x = x0 + c;
          if (x >= 0 && x < Ln) {
            qn[x] = t4[c];
            if (x < m && qc[x] != t4[c]) m = x;
          }
        }
      }
    }
  }
  // minimum over the wave (m >= 0), then one LDS atomic per wave
  m = (int32_t)wave_min_u64((uint64_t)(uint32_t)m);
  if (lane_id() == 0) atomicMin(ell, m);
}

// Lowest index among the minimal scores (lanes >= W hold +inf): the same
// result as scanning i = 0..W-1 with a strict less-than.  -0.0 is folded
// into +0.0 (they compare equal); a NaN makes the scan itself decide.
__device__ __forceinline__ uint32_t wave_argmin(double eh, uint32_t W, const double* eh_sh) {
  if (__ballot(eh != eh)) {
    uint32_t best = 0;
    for (uint32_t i = 1; i < W; ++i)
      if (eh_sh[i] < eh_sh[best]) best = i;
    return best;
  }
  const double z = eh + 0.0;
  uint64_t b = (uint64_t)__double_as_longlong(z);
  b = (b >> 63) ? ~b : (b | 0x8000000000000000ull);  // order-preserving key
  const uint64_t mn = wave_min_u64(b);
  return (uint32_t)first_lane(__ballot(b == mn));
}

// Lowest lane among the minima of v (lanes >= W excluded).
__device__ __forceinline__ uint32_t wave_argmin_u32(uint32_t v, uint32_t W) {
  const uint64_t key = (uint32_t)lane_id() < W ? (((uint64_t)v << 32) | (uint32_t)lane_id()) : ~0ull;
  return (uint32_t)(wave_min_u64(key) & 0xffffffffull);
}

// The routed worker of query k (global index j0 + k): the LBGR argmin, or
// one of the baseline routers of Sec. 5.  Wave-uniform; one lane per worker.
__device__ __forceinline__ uint32_t route_choice(const StepArgs& a, uint32_t r, uint32_t k, uint32_t W, double eh,
                                                 const int32_t* hrow, int32_t Lq, const double* eh_sh,
                                                 const RouteView& v) {
  const uint64_t jg = a.j0 + k;
  if (a.C.router == KVR_ROUTE_RANDOM)
    return (uint32_t)__umul64hi(philox_word0(jg, 0ull, 0ull, 1ull, a.C.seed, r), (uint64_t)W);
  if (a.C.router == KVR_ROUTE_ROUND_ROBIN) return (uint32_t)(jg % W);
  if (a.C.router == KVR_ROUTE_CACHE_AWARE) {
    uint32_t load = 0, size = 0, h = 0;
    if ((uint32_t)lane_id() < W) {
      load = v.pend_count;
      size = v.size;
      h = (uint32_t)hrow[lane_id()];
    }
    const uint32_t lo = wave_argmin_u32(load, W);
    const uint32_t hi = wave_argmin_u32(~load, W);
    const uint32_t hmax = wave_argmin_u32(~h, W);
    const uint32_t small = wave_argmin_u32(size, W);
    const uint32_t lmin = (uint32_t)__builtin_amdgcn_readlane((int)load, (int)lo);
    const uint32_t lmax = (uint32_t)__builtin_amdgcn_readlane((int)load, (int)hi);
    const int32_t hbest = hrow[hmax];
    if (lmax - lmin > (uint32_t)a.C.ca_balance_abs && (double)lmax > a.C.ca_balance_rel * (double)lmin) return lo;
    if ((double)hbest > a.C.ca_cache_threshold * (double)Lq) return hmax;
    return small;
  }
  return wave_argmin(eh, W, eh_sh);
}

// Record a match length and count it in the workgroup's per-worker sums
// (LDS; added to the worker headers when the batch ends).
__device__ __forceinline__ void count_mtok(unsigned long long* mtok, uint32_t w, int32_t h, int32_t* hslot) {
  if (lane_id() == 0) {
    *hslot = h;
    atomicAdd(&mtok[w], (unsigned long long)(uint32_t)h);
  }
}

// Record a match length without counting it (the cache's own match when
// the router scores with its own tree).
__device__ __forceinline__ void store_h(int32_t h, int32_t* hslot) {
  if (lane_id() == 0) *hslot = h;
}

// The next query's h on the workers other than `best`, taken one item at a
// time from an LDS counter, so a wave that drew long matches takes fewer.
// Items 0..W-1 are the
// caches; with the approximate router, items W..2W-1 are the router's trees.
// The index is wave-uniform (lane 0's atomic, read back from lane 0) and the
// loop is bounded by the number of items.
__device__ __forceinline__ void take_matches(const StepArgs& a, uint32_t r, uint32_t W, uint32_t best,
                                             const int32_t* qn, int32_t Lnq, int32_t ell, const int32_t* h_cur,
                                             int32_t* h_next, const int32_t* g_cur, int32_t* g_next,
                                             const PathArea& paths, const PathArea& rpaths, bool rtree,
                                             uint32_t* next) {
  const uint32_t items = rtree ? 2u * W : W;
  for (uint32_t it = 0; it < items; ++it) {
    uint32_t got = 0;
    if (lane_id() == 0) got = atomicAdd(next, 1u);
    const uint32_t i = (uint32_t)__builtin_amdgcn_readlane((int)got, 0);
    if (i >= items) break;
    const uint32_t w = i < W ? i : i - W;
    if (w == best) continue;
    Ptrs Pw = worker_ptrs(a.ws, a.L, r, w);
    if (i < W) {
      const int32_t h = match_incremental(Pw, Pw.hdr->arena_sel, qn, Lnq, h_cur[w], ell, paths.of(w));
      if (rtree)
        store_h(h, &h_next[w]);
      else
        count_matched(Pw, h, &h_next[w]);
    } else {
      Ptrs Pr = router_ptrs(a.ws, a.L, r, w);
      count_matched(Pw, match_incremental(Pr, Pr.hdr->arena_sel, qn, Lnq, g_cur[w], ell, rpaths.of(w)), &g_next[w]);
    }
  }
}

// First device-side error of the run (check id and values for the message),
// then the sticky status bits; the workgroup stops after the next barrier.
__device__ __forceinline__ void report_error(GlobalHdr* g, uint32_t r, uint64_t jg, uint32_t err, const int64_t* dbg,
                                             uint32_t* abort_flag) {
  if (lane_id() != 0 || !err) return;
  if (atomicCAS(&g->err_taken, 0u, 1u) == 0u) {
    g->err_check = (uint32_t)dbg[0];
    g->err_replica = r;
    g->err_query = jg;
    g->err_val[0] = dbg[1];
    g->err_val[1] = dbg[2];
    g->err_val[2] = dbg[3];
  }
  atomicOr(&g->status, err);
  *abort_flag = 1;
}

// Approximate router: the router adds prompt q[0, Lq) to its tree of the
// routed worker (L-LRU; hr = the router's match of it), then matches the
// next prompt there, from the path just inserted.  Returns KVR_DEV_* bits.
__device__ __forceinline__ uint32_t router_admit(const StepArgs& a, uint32_t r, uint64_t jg, uint32_t best,
                                                 const int32_t* qs, int32_t Lq, int32_t hr, bool has_next,
                                                 const int32_t* qn, int32_t Lnq, int32_t ell, const PathArea& rpaths,
                                                 int32_t* g_next, int64_t* dbg) {
  Ptrs Pr = router_ptrs(a.ws, a.L, r, best);
  InsertArgs ia;
  ia.seed = a.C.seed;
  ia.jg = jg;
  ia.worker = best;
  ia.replica = r;
  ia.B = a.L.RB;
  ia.rn = 0;
  ia.rw = nullptr;
  ia.prog = nullptr;
  ia.nprog = 0;
  ia.round = 1;
  ia.rank = nullptr;
  ia.rank_ready = nullptr;
  const uint32_t err = lru_insert(Pr, ia, qs, Lq, hr, rpaths.of(best), dbg);
  if (!err && has_next)
    count_matched(worker_ptrs(a.ws, a.L, r, best),
                  match_incremental(Pr, Pr.hdr->arena_sel, qn, Lnq, Lq, ell, rpaths.of(best)), g_next);
  return err;
}

// One workgroup per replica walks the batch in order.  A worker's tree
// changes only when a query is routed to it, so while wave 0 inserts query k
// into the routed worker the other waves compute the draw words of that
// insertion, the completions and decay at the next arrival, and the next
// query's h on every other worker.  Matches are incremental: each worker
// keeps the path of its last match, and the next query follows it up to
// the longest common prefix of the two queries.  The routed worker's h for
// the next query is completed from the path of the inserted query.  With
// the approximate router every worker has two trees, the cache and the
// router's, each matched incrementally; the router's tree of the routed
// worker is updated by a helper wave.  The approximate router (RT) and
// continuous batching (BA) are template switches, so the kernel without
// them carries none of their registers.
template <bool RT, bool BA, bool PT>
__global__ void __launch_bounds__(512) step_kernel(StepArgs a) {
  // dynamic LDS: two query buffers (max_query_tokens entries each), the high
  // halves of the draw words, the match paths (the caches', then the router
  // trees'), then the staged candidate list
  extern __shared__ int32_t smem[];
  const uint32_t W = a.L.W;
  constexpr bool rtree = RT;
  const uint32_t qstride = (a.L.maxL + 3u) & ~3u;
  uint32_t* rw = reinterpret_cast<uint32_t*>(smem + 2 * qstride);
  PathArea paths, rpaths;
  paths.base = reinterpret_cast<int32_t*>(rw + a.rcap);
  paths.W = W;
  rpaths.base = paths.base + (size_t)W * (3 * kPathMax + 1);
  rpaths.W = W;
  UStage ustage;
  {
    int32_t* ub = paths.base + (size_t)(rtree ? 2 : 1) * W * (3 * kPathMax + 1);
    ustage.node = ub;
    ustage.len = ub + a.ucap;
    ustage.top = ub + 2 * a.ucap;
    ustage.par = ub + 3 * a.ucap;
    ustage.cap = a.ucap;
  }
  __shared__ int32_t h_sh[2][kMaxWorkers];  // h of the current and of the next query (the caches)
  __shared__ int32_t g_sh[2][kMaxWorkers];  // the same on the router's trees (approximate router)
  __shared__ double eh_sh[kMaxWorkers];
  __shared__ int32_t ell_sh[2];  // LCP(q_k, q_k+1) in slot k & 1
  __shared__ int32_t best_sh;
  __shared__ int32_t hins_sh;  // cached length of the inserted path (>= h of the prompt)
  __shared__ uint32_t abort_sh;
  __shared__ uint32_t nev_sh;
  __shared__ uint32_t prog_sh[16];  // rounds of draw words each drawing wave has written
  __shared__ uint32_t next_sh;    // next item for the helpers' matches
  __shared__ int32_t rank_sh;     // the new leaf's rank, from the last helper wave
  __shared__ uint32_t rank_ready_sh;
  // the hits the router scores with: the caches' own, or its trees'
  int32_t(*est)[kMaxWorkers] = rtree ? g_sh : h_sh;

  const uint32_t r = blockIdx.x;
  const bool resp = a.C.cache_responses != 0;
  const int lane = lane_id();
  const uint32_t wave = threadIdx.x / KVR_WAVE;
  const uint32_t nwaves = blockDim.x / KVR_WAVE;
  const uint32_t nh = nwaves - 1;  // helper waves
  GlobalHdr* g = reinterpret_cast<GlobalHdr*>(a.ws + a.L.off_global);
  ReplicaHdr* rh = reinterpret_cast<ReplicaHdr*>(a.ws + a.L.off_rhdr) + r;

  if (threadIdx.x == 0) {
    abort_sh = __atomic_load_n(&g->status, __ATOMIC_RELAXED);
    ell_sh[0] = 0x7fffffff;
  }
  __syncthreads();
  if (abort_sh) return;
  // the replica's route digest and query count, kept by the routing wave
  uint64_t chain = 0, routed = 0;
  if (wave == 0) {
    chain = rh->route_digest;
    routed = rh->queries;
  }
  PhaseClock clk;
  clock_start<PT>(&clk);

  // query 0: stage its path; completions and decay at its arrival; full
  // matches of its prompt
  {
    const uint64_t o0 = a.offsets[0];
    const int32_t L0 = (int32_t)(a.offsets[1] - o0);
    const int32_t L0q = resp ? L0 - query_out_len(a.out_len, 0) : L0;
    for (int32_t x = (int32_t)threadIdx.x; x < L0; x += (int32_t)blockDim.x) smem[x] = a.tokens[o0 + x];
    if (wave == 0 && (uint32_t)lane < W)
      complete_and_decay(a.C, worker_ptrs(a.ws, a.L, r, (uint32_t)lane), a.arrival[0], rh->tprev);
    __syncthreads();
    for (uint32_t i = wave; i < W; i += nwaves) {
      Ptrs P = worker_ptrs(a.ws, a.L, r, i);
      const int32_t h = match_lcp(P, P.hdr->arena_sel, smem, L0q, paths.of(i));
      if (rtree) {
        store_h(h, &h_sh[0][i]);
        Ptrs Pr = router_ptrs(a.ws, a.L, r, i);
        count_matched(P, match_lcp(Pr, Pr.hdr->arena_sel, smem, L0q, rpaths.of(i)), &g_sh[0][i]);
      } else {
        count_matched(P, h, &h_sh[0][i]);
      }
    }
  }
  for (uint32_t k = 0; k < a.n; ++k) {
    const uint64_t o0 = a.offsets[k];
    const int32_t Lp = (int32_t)(a.offsets[k + 1] - o0);  // the path inserted
    const int64_t t = a.arrival[k];
    const int32_t olen = query_out_len(a.out_len, k);
    const int32_t Lq = resp ? Lp - olen : Lp;  // the prompt
    const uint32_t cur = k & 1u;
    int32_t* qs = smem + cur * qstride;
    int32_t* qn = smem + (cur ^ 1u) * qstride;
    const bool has_next = k + 1 < a.n;
    int32_t Ln = 0, Lnq = 0;  // path and prompt of the next query
    uint64_t n0 = 0;
    if (has_next) {
      n0 = a.offsets[k + 1];
      Ln = (int32_t)(a.offsets[k + 2] - n0);
      Lnq = resp ? Ln - query_out_len(a.out_len, k + 1) : Ln;
    }
    __syncthreads();

    // ---- phase A.  Wave 0: scores, argmin, commit.  Helpers: stage the
    // next query.
    if (wave == 0) {
      double eh = __builtin_huge_val(), ch = 0.0;
      RouteView v{};
      if ((uint32_t)lane < W) {
        v = load_view(worker_ptrs(a.ws, a.L, r, (uint32_t)lane).hdr);
        eh = lbgr_score(a.C, v, est[cur][lane], Lq, &ch);
        eh_sh[lane] = eh;
      }
      __builtin_amdgcn_wave_barrier();
      const uint32_t best = route_choice(a, r, k, W, eh, est[cur], Lq, eh_sh, v);
      Ptrs P = worker_ptrs(a.ws, a.L, r, best);
      const int32_t hb = h_sh[cur][best];  // the worker's true hit
      // a cached prompt may continue into a cached response: the insertion
      // needs the cached length of the whole path, continued from the
      // prompt's recorded match
      int32_t hins = hb;
      if (resp && hb == Lq && Lp > Lq) hins = match_incremental(P, P.hdr->arena_sel, qs, Lp, Lq, Lq, paths.of(best));
      // the routed worker's lane commits from the header fields it holds
      uint32_t cerr = 0;
      if ((uint32_t)lane == best) cerr = commit_route(a.C, P, v, ch, hb, est[cur][best], Lq, t, olen);
      const uint32_t err = (uint32_t)__builtin_amdgcn_readlane((int)cerr, (int)best);
      const uint32_t size = (uint32_t)__builtin_amdgcn_readlane((int)v.size, (int)best);
      if ((uint32_t)lane < 16u) prog_sh[lane] = 0u;
      if (lane == 0) {
        best_sh = (int32_t)best;
        hins_sh = hins;
        next_sh = 0;
        rank_ready_sh = 0;
        const uint64_t orow = (uint64_t)r * a.n + k;
        if (a.route) a.route[orow] = (int32_t)best;
        if (a.hits) a.hits[orow] = hb;
        if (!err) {
          chain = route_chain(chain, a.j0 + k, best, hb);
          routed += 1;
        }
        // draws this insertion will take: one per token loaded into a full cache
        const uint32_t nload = (uint32_t)(Lp - hins);
        const uint32_t nfree = a.L.B - size;
        nev_sh = err ? 0u : (nload > nfree ? nload - nfree : 0u);
        if (err) {
          atomicOr(&g->status, err);
          abort_sh = 1;
        }
      }
      if (a.all_hits && (uint32_t)lane < W)
        a.all_hits[((uint64_t)r * a.n + k) * W + (uint32_t)lane] = est[cur][lane];
      if (nh == 0 && has_next) stage_next(a.tokens, n0, Ln, qn, qs, Lp, (uint32_t)lane, KVR_WAVE, &ell_sh[cur]);
    } else if (has_next) {
      stage_next(a.tokens, n0, Ln, qn, qs, Lp, threadIdx.x - KVR_WAVE, blockDim.x - KVR_WAVE, &ell_sh[cur]);
    }
    if (wave == 0) clock_mark<PT>(&clk, KVR_PHASE_ROUTE);
    __syncthreads();
    if (wave == 0) clock_mark<PT>(&clk, KVR_PHASE_STAGE_WAIT);
    if (abort_sh) break;
    const uint32_t best = (uint32_t)best_sh;
    const uint32_t nev = nev_sh;
    // draw words: RLT only
    const uint32_t rn = a.C.evict == KVR_EVICT_RLT ? (nev < a.rcap ? nev : a.rcap) : 0u;
    const int32_t hins = hins_sh;
    // LCP of the two paths, then of what the next match needs: the next
    // prompt against the inserted path (the routed cache) or against this
    // prompt (every other cache, whose recorded match is of this prompt, and
    // every router tree, which holds prompts only)
    const int32_t ellp = ell_sh[cur];
    const int32_t ell_r = ellp < Lnq ? ellp : Lnq;
    const int32_t ell = ell_r < Lq ? ell_r : Lq;
    const uint64_t jg = a.j0 + k;
    // with two or more helpers, the last one ranks the new leaf of an RLT
    // insertion while the others compute its draw words
    const bool ranker = nh >= 2 && a.C.evict == KVR_EVICT_RLT && hins < Lp;

    // ---- phase B.  Wave 0: the insertion, then the routed worker's h for
    // the next query.  Helpers: the insertion's draw words first, then
    // completions and decay at the next arrival (and the router's tree of
    // the routed worker), and the next query's h on the other workers.
    if (wave == 0) {
      if (nh == 0)
        for (uint32_t d = (uint32_t)lane; d < rn; d += KVR_WAVE)
          rw[d] = (uint32_t)(philox_word0(jg, best, d, 0ull, a.C.seed, r) >> 32);
      Ptrs P = worker_ptrs(a.ws, a.L, r, best);
      InsertArgs ia;
      ia.seed = a.C.seed;
      ia.jg = jg;
      ia.worker = best;
      ia.replica = r;
      ia.B = a.L.B;
      ia.rn = rn;
      ia.rw = rw;
      ia.prog = nh && rn ? prog_sh : nullptr;
      ia.nprog = ranker ? nh - 1u : nh;
      ia.round = 2u * (blockDim.x - (ranker ? 2u : 1u) * KVR_WAVE);
      ia.rank = ranker ? &rank_sh : nullptr;
      ia.rank_ready = &rank_ready_sh;
      int64_t dbg[4] = {0, 0, 0, 0};
      uint32_t err = a.C.evict == KVR_EVICT_RLT ? rlt_insert<PT>(P, ia, qs, Lp, hins, ustage, paths.of(best), dbg, &clk)
                                                : lru_insert(P, ia, qs, Lp, hins, paths.of(best), dbg);
      // continuous batching: the path joins the worker's running batch
      if (BA && !err && P.beta > 1) err = batch_admit(P, paths.of(best), qs, Lp, dbg);
      report_error(g, r, jg, err, dbg, &abort_sh);
      // the routed worker's h for the next query, from the path of the
      // query just inserted (all of it is cached now: the old h is Lp)
      if (has_next && !err) {
        Ptrs Pb = worker_ptrs(a.ws, a.L, r, best);
        const int32_t h = match_incremental(Pb, Pb.hdr->arena_sel, qn, Lnq, Lp, ell_r, paths.of(best));
        if (rtree)
          store_h(h, &h_sh[cur ^ 1u][best]);
        else
          count_matched(Pb, h, &h_sh[cur ^ 1u][best]);
      }
      clock_mark<PT>(&clk, KVR_PHASE_MATCH);
      if (nh == 0 && !err) {
        if (has_next) {
          if ((uint32_t)lane < W)
            complete_and_decay(a.C, worker_ptrs(a.ws, a.L, r, (uint32_t)lane), a.arrival[k + 1], t);
          if (lane == 0) ell_sh[cur ^ 1u] = 0x7fffffff;
        }
        if (rtree) {
          int64_t rdbg[4] = {0, 0, 0, 0};
          const uint32_t rerr = router_admit(a, r, jg, best, qs, Lq, g_sh[cur][best], has_next, qn, Lnq, ell, rpaths,
                                             &g_sh[cur ^ 1u][best], rdbg);
          report_error(g, r, jg, rerr, rdbg, &abort_sh);
        }
        if (has_next)
          take_matches(a, r, W, best, qn, Lnq, ell, h_sh[cur], h_sh[cur ^ 1u], g_sh[cur], g_sh[cur ^ 1u], paths,
                       rpaths, rtree, &next_sh);
      }
    } else {
      if (ranker && wave == nwaves - 1) {
        // the last helper ranks the insertion's new leaf
        rank_for_insertion(worker_ptrs(a.ws, a.L, r, best), paths.of(best), qs, hins, &rank_sh, &rank_ready_sh);
      } else {
        // the others compute the draw words, a round of 2*nd words at a
        // time (two independent words per lane), and publish each round
        // they complete
        const uint32_t nd = blockDim.x - (ranker ? 2u : 1u) * KVR_WAVE;
        uint32_t rounds = 0;
        for (uint32_t base = 0; base < rn; base += 2u * nd) {
          const uint32_t d0 = base + threadIdx.x - KVR_WAVE, d1 = d0 + nd;
          const uint64_t w0 = philox_word0(jg, best, d0, 0ull, a.C.seed, r);
          const uint64_t w1 = philox_word0(jg, best, d1, 0ull, a.C.seed, r);
          if (d0 < rn) rw[d0] = (uint32_t)(w0 >> 32);
          if (d1 < rn) rw[d1] = (uint32_t)(w1 >> 32);
          ++rounds;
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
          if (lane == 0)
            __hip_atomic_store(&prog_sh[wave - 1u], rounds, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
      }
      if (wave == 1) {
        if (has_next) {
          if ((uint32_t)lane < W)
            complete_and_decay(a.C, worker_ptrs(a.ws, a.L, r, (uint32_t)lane), a.arrival[k + 1], t);
          if (lane == 0) ell_sh[cur ^ 1u] = 0x7fffffff;
        }
        if (rtree) {
          int64_t rdbg[4] = {0, 0, 0, 0};
          const uint32_t rerr = router_admit(a, r, jg, best, qs, Lq, g_sh[cur][best], has_next, qn, Lnq, ell, rpaths,
                                             &g_sh[cur ^ 1u][best], rdbg);
          report_error(g, r, jg, rerr, rdbg, &abort_sh);
        }
      }
      if (has_next)
        take_matches(a, r, W, best, qn, Lnq, ell, h_sh[cur], h_sh[cur ^ 1u], g_sh[cur], g_sh[cur ^ 1u], paths,
                     rpaths, rtree, &next_sh);
    }
    __syncthreads();
    if (wave == 0) clock_mark<PT>(&clk, KVR_PHASE_JOIN);
    if (abort_sh) break;
  }
  if (threadIdx.x == 0) {
    if constexpr (PT)
      for (int p = 0; p < KVR_PHASES; ++p) rh->phase_ticks[p] += clk.acc[p];
    rh->route_digest = chain;
    rh->queries = routed;
    if (!abort_sh && a.n > 0) {
      rh->tprev = a.arrival[a.n - 1];
      if (r == 0) g->last_arrival = a.arrival[a.n - 1];
    }
  }
}

// ---------------------------------------------------------------- pipelined step kernel
//
// RLT with prompts only, LBGR or a baseline router, no approximate router
// and single-query processing (the benchmark's path).  The evictions of an
// insertion only touch the routed worker's cache, and nothing the routing of
// the next query reads depends on them but that worker's h of the next
// query.  So a separate wave, the evicting wave, runs the back half of each
// insertion (evictions, marks of the loaded tokens, header) while the
// routing wave routes the next query and runs the front half of its
// insertion (marking walk, split, rank, load of the new leaf).  The routing
// wave takes the routed worker's h of the next query on the tree after the
// load and before the evictions: the evictions never remove a token of the
// inserted path, so when that match ends on the inserted path (h equal to
// the two queries' longest common prefix) it is exact; otherwise it is taken
// again once the evictions are done.  One insertion is evicted at a time:
// the routing wave waits for the evicting wave before it hands it the next
// insertion or inserts into the worker being evicted.
//
// Waves: 0 routes and runs front halves, 1 evicts, 2.. are helpers (stage
// the next query, compute draw words, rank the new leaf, apply completions
// and decay, match the next query on the other workers).  They synchronise
// through the counters below (LDS, workgroup scope, release/acquire); every
// wait is bounded and checks the stop flag, so an error ends every loop.

struct PipeFlags {
  uint32_t top;         // the routing wave has begun query top - 1: q_top may be staged
  uint32_t routed;      // queries routed (route, evictions and slots of query routed - 1 published)
  uint32_t staged;      // staging waves done, over all queries
  uint32_t matched;     // helper matches done, over all queries (W - 1 per query)
  uint32_t decayed;     // arrivals whose completions and decay are applied
  uint32_t handed;      // insertions handed to the evicting wave
  uint32_t evicted;     // insertions it has finished
  uint32_t ework;       // worker of its current insertion, kNoWorker when idle
  uint32_t ework_size;  // that worker's |S| once the insertion is done
  uint32_t end;         // no more insertions will be handed
  uint32_t stop;        // an error stopped the replica
  uint32_t next[2];     // helper match items taken, by query parity
  uint32_t last_worker; // worker of the last insertion handed to the evicting wave
  uint32_t pad;
  // the next query's matches, claimed per worker (bit i) by the wave that
  // takes them, by query parity: a helper, or the evicting wave for its
  // worker once its evictions end
  unsigned long long claim[2];
};

constexpr uint32_t kNoWorker = 0xffffffffu;
// 16-byte compare loads in flight per lane in the pipelined kernel's matches
// (its next-query matches are on the routing wave's path)
#ifndef KVR_PIPE_MATCH_UNROLL
#define KVR_PIPE_MATCH_UNROLL 8
#endif
constexpr int kPipeMatchUnroll = KVR_PIPE_MATCH_UNROLL;
// ... in the matches taken from the shared item counter (most of them, on
// the helper waves, whose registers are not the kernel's peak)
#ifndef KVR_PIPE_ITEM_UNROLL
#define KVR_PIPE_ITEM_UNROLL 8
#endif
constexpr int kPipeItemUnroll = KVR_PIPE_ITEM_UNROLL;
constexpr uint32_t kSpinLimit = 1u << 24;
#ifndef KVR_PIPE_WAVES
#define KVR_PIPE_WAVES 8
#endif
constexpr uint32_t kPipeWaves = KVR_PIPE_WAVES;
// Waves per workgroup for replicas of many workers: four more helpers for
// the next query's matches, at a register cap of 168 VGPRs instead of 256
// (the routing wave's loop state then partly lives in scratch).  Measured
// faster at 32 workers and slower at 16, so used from 17 on.
#ifndef KVR_PIPE_WAVES_WIDE
#define KVR_PIPE_WAVES_WIDE 12
#endif
#ifndef KVR_PIPE_WIDE_WORKERS
#define KVR_PIPE_WIDE_WORKERS 17
#endif
constexpr uint32_t kPipeWavesWide = KVR_PIPE_WAVES_WIDE;
constexpr uint32_t kPipeWideWorkers = KVR_PIPE_WIDE_WORKERS;

__device__ __forceinline__ uint32_t ld_acq(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Publish v (lane 0, after every lane's earlier writes).
__device__ __forceinline__ void st_rel(uint32_t* p, uint32_t v) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  if (lane_id() == 0) __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ void add_rel(uint32_t* p, uint32_t v) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  if (lane_id() == 0) __hip_atomic_fetch_add(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Stop the replica: the first error of the run is recorded (check id, the
// query, values), the status bits are set and every wave's waits end.
__device__ __forceinline__ void pipe_stop(GlobalHdr* g, PipeFlags* f, uint32_t r, uint64_t jg, uint32_t err,
                                          const int64_t* dbg) {
  if (lane_id() == 0) {
    if (atomicCAS(&g->err_taken, 0u, 1u) == 0u) {
      g->err_check = (uint32_t)dbg[0];
      g->err_replica = r;
      g->err_query = jg;
      g->err_val[0] = dbg[1];
      g->err_val[1] = dbg[2];
      g->err_val[2] = dbg[3];
    }
    atomicOr(&g->status, err);
    __hip_atomic_store(&f->stop, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
}

// Wait until *p >= target (or, with ne, until *p != target).  False when
// the replica was stopped; a wait that runs out stops it (check id 90 +
// site, an internal error).
template <bool kNe = false>
__device__ __forceinline__ bool pipe_wait(const uint32_t* p, uint32_t target, PipeFlags* f, GlobalHdr* g, uint32_t r,
                                          uint64_t jg, int site) {
  uint32_t spins = 0;
  for (;;) {
    const uint32_t v = ld_acq(p);
    if (kNe ? v != target : v >= target) return true;
    if (__hip_atomic_load(&f->stop, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP)) return false;
    if (++spins > kSpinLimit) {
      const int64_t dbg[4] = {90 + site, (int64_t)v, (int64_t)target, 0};
      pipe_stop(g, f, r, jg, KVR_DEV_INTERNAL, dbg);
      return false;
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

// Root filters of the pipelined kernel: per worker a 256-bit Bloom filter
// (in LDS) of the first tokens of its root's children, two bits per token,
// built when the kernel starts and extended when an insertion adds a child
// to the root.  A clear bit proves that no cached path starts with the
// token, so a match that starts at the root is 0 without a memory access; a
// set bit (also one left by a child evicted since) only means the tree is
// walked.  (512- and 1,024-bit filters measured within 1% of this.)
#ifndef KVR_ROOT_FILTER_LOG2_BITS
#define KVR_ROOT_FILTER_LOG2_BITS 8
#endif
constexpr uint32_t kRootFilterBits = 1u << KVR_ROOT_FILTER_LOG2_BITS;
constexpr uint32_t kRootFilterWords = kRootFilterBits / 32u;

__device__ __forceinline__ uint32_t rf_bit1(int32_t t) {
  return ((uint32_t)t * 0x9E3779B1u) >> (32 - KVR_ROOT_FILTER_LOG2_BITS);
}
__device__ __forceinline__ uint32_t rf_bit2(int32_t t) {
  return ((uint32_t)t * 0x85EBCA6Bu + 0x632BE5ABu) >> (32 - KVR_ROOT_FILTER_LOG2_BITS);
}

__device__ __forceinline__ void rf_add(uint32_t* rf, int32_t t) {
  atomicOr(&rf[rf_bit1(t) >> 5], 1u << (rf_bit1(t) & 31u));
  atomicOr(&rf[rf_bit2(t) >> 5], 1u << (rf_bit2(t) & 31u));
}

__device__ __forceinline__ bool rf_may(const uint32_t* rf, int32_t t) {
  return ((rf[rf_bit1(t) >> 5] >> (rf_bit1(t) & 31u)) & 1u) && ((rf[rf_bit2(t) >> 5] >> (rf_bit2(t) & 31u)) & 1u);
}

// h of qn[0, Ln) on a worker from its recorded path (match_incremental);
// sel = the active semispace, or -1 to read it from the header when the tree
// is walked.  A match that would start at the root is settled by the root
// filter when it rules out qn[0].
template <int kU = kPipeMatchUnroll>
__device__ __forceinline__ int32_t match_pipe(const Ptrs& P, int32_t sel, const uint32_t* rf, const int32_t* qn,
                                              int32_t Ln, int32_t h_old, int32_t ell, const PathRef& pr) {
  if ((ell == 0 || *pr.cnt > kPathMax) && !rf_may(rf, qn[0])) {
    if (lane_id() == 0) *pr.cnt = 0;
    return 0;
  }
  if (sel < 0) return match_incremental_lazy<kU>(P, qn, Ln, h_old, ell, pr);
  return match_incremental<kU>(P, (uint32_t)sel, qn, Ln, h_old, ell, pr);
}

// The next query's h on the workers other than the routed one (best) of
// query parity cur, taken one item at a time from the LDS counter; the
// worker being evicted is left to the evicting wave, and every other is
// claimed first (the evicting wave may have taken it).  Returns the number
// of matches done (the caller publishes them).
template <int kU>
__device__ __forceinline__ uint32_t take_matches_pipe(const StepArgs& a, uint32_t r, uint32_t W, uint32_t cur,
                                                      uint32_t best, uint32_t prev, const int32_t* qn, int32_t Ln,
                                                      int32_t ell, const int32_t* h_cur, int32_t* h_next, PipeFlags* f,
                                                      unsigned long long* mtok, const uint32_t* rootf,
                                                      const PathArea& paths) {
  uint32_t mine = 0;
  for (uint32_t it = 0; it < W; ++it) {
    uint32_t got = 0;
    if (lane_id() == 0) got = atomicAdd(&f->next[cur], 1u);
    const uint32_t item = (uint32_t)__builtin_amdgcn_readlane((int)got, 0);
    if (item >= W) break;
    const uint32_t w = (prev + 1u + item) % W;
    if (w == best) continue;
    if (__hip_atomic_load(&f->ework, __ATOMIC_SEQ_CST, __HIP_MEMORY_SCOPE_WORKGROUP) == w) continue;
    unsigned long long old = 0ull;
    if (lane_id() == 0) old = atomicOr(&f->claim[cur], 1ull << w);
    const uint32_t taken = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((old >> w) & 1ull), 0);
    if (taken) continue;
    Ptrs Pw = worker_ptrs(a.ws, a.L, r, w);
    count_mtok(mtok, w,
               match_pipe<kU>(Pw, -1, rootf + w * kRootFilterWords, qn, Ln, h_cur[w], ell, paths.of(w)),
               &h_next[w]);
    ++mine;
  }
  return mine;
}

// NW = waves per workgroup (the kernel itself takes it from blockDim).
template <bool PT, uint32_t NW>
__global__ void __launch_bounds__(64 * NW) step_kernel_pipe(StepArgs a) {
  // dynamic LDS: two query buffers, the draw words of two insertions, the
  // match paths, the staged candidate list
  extern __shared__ int32_t smem[];
  const uint32_t W = a.L.W;
  const uint32_t qstride = (a.L.maxL + 3u) & ~3u;
  uint32_t* rwb = reinterpret_cast<uint32_t*>(smem + 2 * qstride);  // [2][rcap]
  PathArea paths;
  paths.base = reinterpret_cast<int32_t*>(rwb + 2 * a.rcap);
  paths.W = W;
  // root filters (kRootFilterWords words per worker), then the candidates
  uint32_t* rootf = reinterpret_cast<uint32_t*>(paths.base + (size_t)W * (3 * kPathMax + 1));
  UStage ustage;
  {
    int32_t* ub = reinterpret_cast<int32_t*>(rootf + (size_t)W * kRootFilterWords);
    ustage.node = ub;
    ustage.len = ub + a.ucap;
    ustage.top = ub + 2 * a.ucap;
    ustage.par = ub + 3 * a.ucap;
    ustage.cap = a.ucap;
  }
  __shared__ int32_t h_sh[2][kMaxWorkers];  // h of q_k in slot k & 1
  __shared__ double eh_sh[kMaxWorkers];
  __shared__ int32_t ell_sh[2];             // LCP(q_k, q_k+1) in slot k & 1
  __shared__ int32_t best_sh[2];
  __shared__ uint32_t rn_sh[2];             // draw words of insertion k precomputed in slot k & 1
  __shared__ uint32_t prog_sh[2][16];       // rounds of them each drawing wave has written
  __shared__ int32_t rank_sh;
  __shared__ uint32_t rank_ready_sh;
  __shared__ PipeFlags f;
  __shared__ EvictJob job_sh[2];            // by insertion count parity
  // per handed insertion (same parity): the routed worker's h of the next
  // query not taken yet (0), taken and exact (1), taken but to be taken
  // again after the evictions (2)
  __shared__ uint32_t early_sh[2];
  __shared__ unsigned long long eticks_sh[KVR_PHASES];  // evicting and helper waves' ticks
  // matched tokens per worker over the batch (added to the headers at the end)
  __shared__ unsigned long long mtok_sh[kMaxWorkers];

  const uint32_t r = blockIdx.x;
  const int lane = lane_id();
  const uint32_t wave = threadIdx.x / KVR_WAVE;
  const uint32_t nwaves = blockDim.x / KVR_WAVE;
  const uint32_t nh = nwaves - 2;  // helper waves (>= 2)
  // the last helper ranks new leaves; half of the helpers compute the draw
  // words first, the rest start on the next query's matches at once (both
  // are due about when the front half of the insertion ends)
  const uint32_t ndraw = nh / 2u < 16u ? nh / 2u : 16u;
  const uint32_t nd = ndraw * KVR_WAVE;  // drawing threads
  GlobalHdr* g = reinterpret_cast<GlobalHdr*>(a.ws + a.L.off_global);
  ReplicaHdr* rh = reinterpret_cast<ReplicaHdr*>(a.ws + a.L.off_rhdr) + r;

  if (threadIdx.x == 0) {
    f.top = 1;  // q_1 may be staged at once (its buffer is free)
    f.routed = f.staged = f.matched = f.handed = f.evicted = f.end = 0;
    f.decayed = 0;
    f.ework = kNoWorker;
    f.ework_size = 0;
    f.next[0] = f.next[1] = 0;
    f.claim[0] = f.claim[1] = 0ull;
    f.last_worker = kNoWorker;
    f.pad = 0;
    f.stop = __atomic_load_n(&g->status, __ATOMIC_RELAXED) ? 1u : 0u;
    ell_sh[0] = ell_sh[1] = 0x7fffffff;
    rank_ready_sh = 0;
    for (uint32_t i = 0; i < kMaxWorkers; ++i) mtok_sh[i] = 0ull;
    for (int p = 0; p < KVR_PHASES; ++p) eticks_sh[p] = 0;
  }
  for (uint32_t x = threadIdx.x; x < W * kRootFilterWords; x += blockDim.x) rootf[x] = 0u;
  __syncthreads();
  if (f.stop) return;

  // query 0: stage it; completions and decay at its arrival; full matches
  {
    const uint64_t o0 = a.offsets[0];
    const int32_t L0 = (int32_t)(a.offsets[1] - o0);
    for (int32_t x = (int32_t)threadIdx.x; x < L0; x += (int32_t)blockDim.x) smem[x] = a.tokens[o0 + x];
    if (wave == 0 && (uint32_t)lane < W)
      complete_and_decay(a.C, worker_ptrs(a.ws, a.L, r, (uint32_t)lane), a.arrival[0], rh->tprev);
    // the root filters: the first token of every child of every root
    for (uint32_t i = wave; i < W; i += nwaves) {
      Ptrs P = worker_ptrs(a.ws, a.L, r, i);
      const int32_t* ar = arena_of(P, P.hdr->arena_sel);
      const NodeRec root = P.nodes[0];
      for (int32_t c = lane; c < root.nchild; c += KVR_WAVE) rf_add(rootf + i * kRootFilterWords, ar[root.coff + 2 * c]);
    }
    __syncthreads();
    for (uint32_t i = wave; i < W; i += nwaves) {
      Ptrs P = worker_ptrs(a.ws, a.L, r, i);
      count_mtok(mtok_sh, i, match_lcp<kPipeMatchUnroll>(P, P.hdr->arena_sel, smem, L0, paths.of(i)), &h_sh[0][i]);
    }
    if (threadIdx.x == 0) f.decayed = 1;
    __syncthreads();
  }

  if (wave == 0) {
    // ---------------------------------------------------------- routing wave
    uint64_t chain = rh->route_digest, routed = rh->queries;
    PhaseClock clk;
    clock_start<PT>(&clk);
    uint32_t issued = 0;    // insertions handed to the evicting wave
    uint32_t last_job = 0;  // query index (in the batch) of the last one
    for (uint32_t k = 0; k < a.n; ++k) {
      const uint32_t cur = k & 1u;
      const uint64_t jg = a.j0 + k;
      const uint64_t o0 = a.offsets[k];
      const int32_t Lp = (int32_t)(a.offsets[k + 1] - o0);
      const int64_t t = a.arrival[k];
      const int32_t olen = query_out_len(a.out_len, k);
      const bool has_next = k + 1 < a.n;
      const int32_t Ln = has_next ? (int32_t)(a.offsets[k + 2] - a.offsets[k + 1]) : 0;
      int32_t* qs = smem + cur * qstride;
      const int32_t* qn = smem + (cur ^ 1u) * qstride;
      // h of q_k on every worker (taking any match no other wave has taken
      // yet), completions and decay at its arrival
      if (k > 0) {
        const uint32_t pc = cur ^ 1u;
        const int32_t Lprev = (int32_t)(a.offsets[k] - a.offsets[k - 1]);
        const int32_t ellp = ell_sh[pc];
        const int32_t ell_r = ellp < Lp ? ellp : Lp;
        const int32_t ell = ell_r < Lprev ? ell_r : Lprev;
        const uint32_t prev = k > 1 ? (uint32_t)best_sh[cur] : 0u;
        const uint32_t mine = take_matches_pipe<kPipeMatchUnroll>(a, r, W, pc, (uint32_t)best_sh[pc], prev, qs, Lp, ell, h_sh[pc],
                                                h_sh[cur], &f, mtok_sh, rootf, paths);
        if (mine) add_rel(&f.matched, mine);
        clock_mark<PT>(&clk, KVR_PHASE_MATCH);
      }
      // every worker's h of q_k: W per query from q_1 on (the routed
      // worker's from this wave or the evicting wave, the others' from the
      // helpers, this wave or the evicting wave)
      if (k > 0 && !pipe_wait(&f.matched, k * W, &f, g, r, jg, 0)) break;
      if (!pipe_wait(&f.decayed, k + 1, &f, g, r, jg, 1)) break;
      clock_mark<PT>(&clk, KVR_PHASE_JOIN);

      // the draw words and rounds of this parity are reused below: the
      // evicting wave must be done with the insertion that used them
      if (issued > 0 && (last_job & 1u) == cur && !pipe_wait(&f.evicted, issued, &f, g, r, jg, 11)) break;
      // ---- route: scores, argmin, commit
      const uint32_t ew = ld_acq(&f.ework);
      const uint32_t ew_size = __hip_atomic_load(&f.ework_size, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      double eh = __builtin_huge_val(), ch = 0.0;
      RouteView v{};
      if ((uint32_t)lane < W) {
        v = load_view(worker_ptrs(a.ws, a.L, r, (uint32_t)lane).hdr);
        // the worker being evicted: its size once the evictions are done
        if ((uint32_t)lane == ew) v.size = ew_size;
        eh = lbgr_score(a.C, v, h_sh[cur][lane], Lp, &ch);
        eh_sh[lane] = eh;
      }
      __builtin_amdgcn_wave_barrier();
      const uint32_t best = route_choice(a, r, k, W, eh, h_sh[cur], Lp, eh_sh, v);
      Ptrs P = worker_ptrs(a.ws, a.L, r, best);
      const int32_t hb = h_sh[cur][best];
      uint32_t cerr = 0;
      if ((uint32_t)lane == best) cerr = commit_route(a.C, P, v, ch, hb, hb, Lp, t, olen);
      const uint32_t err0 = (uint32_t)__builtin_amdgcn_readlane((int)cerr, (int)best);
      const uint32_t size = (uint32_t)__builtin_amdgcn_readlane((int)v.size, (int)best);
      const uint32_t nload = (uint32_t)(Lp - hb);
      const uint32_t nfree = a.L.B - size;
      const uint32_t nev = nload > nfree ? nload - nfree : 0u;
      const uint32_t rn = nev < a.rcap ? nev : a.rcap;
      if ((uint32_t)lane < 16u) prog_sh[cur][lane] = 0u;
      if (lane == 0) {
        best_sh[cur] = (int32_t)best;
        rn_sh[cur] = rn;
        f.next[cur] = 0;
        f.claim[cur] = 0ull;
        rank_ready_sh = 0;
        const uint64_t orow = (uint64_t)r * a.n + k;
        if (a.route) a.route[orow] = (int32_t)best;
        if (a.hits) a.hits[orow] = hb;
        if (!err0) {
          chain = route_chain(chain, jg, best, hb);
          routed += 1;
        }
      }
      if (a.all_hits && (uint32_t)lane < W) a.all_hits[((uint64_t)r * a.n + k) * W + (uint32_t)lane] = h_sh[cur][lane];
      if (err0) {
        const int64_t dbg[4] = {0, 0, 0, 0};
        pipe_stop(g, &f, r, jg, err0, dbg);
        break;
      }
      st_rel(&f.routed, k + 1);
      clock_mark<PT>(&clk, KVR_PHASE_ROUTE);

      // ---- front half of the insertion of q_k (the worker being evicted first
      // finishes its evictions)
      if (ew == best && !pipe_wait(&f.evicted, issued, &f, g, r, jg, 3)) break;
      clock_mark<PT>(&clk, KVR_PHASE_EVICTOR_WAIT);
      EvictJob& job = job_sh[issued & 1u];
      {
        InsertArgs ia;
        ia.seed = a.C.seed;
        ia.jg = jg;
        ia.worker = best;
        ia.replica = r;
        ia.B = a.L.B;
        ia.rn = rn;
        ia.rw = rwb + (size_t)cur * a.rcap;
        ia.prog = rn ? prog_sh[cur] : nullptr;
        ia.nprog = ndraw;
        ia.round = 2u * nd;
        ia.rank = hb < Lp ? &rank_sh : nullptr;
        ia.rank_ready = &rank_ready_sh;
        int64_t dbg[4] = {0, 0, 0, 0};
        const uint32_t err = rlt_insert_front<PT>(P, ia, qs, Lp, hb, paths.of(best), dbg, job, &clk);
        if (err) {
          pipe_stop(g, &f, r, jg, err, dbg);
          break;
        }
      }
      // a new child of the root: its first token joins the root filter
      if (hb == 0 && lane == 0) rf_add(rootf + best * kRootFilterWords, qs[0]);
      // q_k's buffer is free: q_k+2 may be staged (its LCP with q_k+1 goes to
      // the slot of LCP(q_k-1, q_k), which nothing reads any more)
      if (lane == 0) ell_sh[cur ^ 1u] = 0x7fffffff;
      st_rel(&f.top, k + 2);
      // ---- nothing to evict: the routed worker's h of the next query (on
      // the tree after the load, which is final) and the back half here;
      // else both on the evicting wave once it is free
      if (job.nev == 0) {
        if (has_next) {
          if (!pipe_wait(&f.staged, (k + 1) * nh, &f, g, r, jg, 4)) break;
          clock_mark<PT>(&clk, KVR_PHASE_STAGE_WAIT);
          const int32_t ellp = ell_sh[cur];
          const int32_t ell_r = ellp < Ln ? ellp : Ln;
          count_mtok(mtok_sh, best,
                     match_pipe(P, (int32_t)job.s.arena_sel, rootf + best * kRootFilterWords, qn, Ln, Lp, ell_r,
                                paths.of(best)),
                     &h_sh[cur ^ 1u][best]);
          add_rel(&f.matched, 1u);
          clock_mark<PT>(&clk, KVR_PHASE_MATCH);
        }
        int64_t dbg[4] = {0, 0, 0, 0};
        const uint32_t err = rlt_insert_back<PT>(P, job, ustage, dbg, &clk);
        if (err) {
          pipe_stop(g, &f, r, jg, err, dbg);
          break;
        }
      } else {
        // the evicting wave takes the routed worker's h of the next query
        // before its evictions; while it still evicts for an earlier
        // insertion, this wave takes that match here first
        uint32_t early = 0;
        if (has_next && ld_acq(&f.evicted) < issued) {
          if (!pipe_wait(&f.staged, (k + 1) * nh, &f, g, r, jg, 4)) break;
          clock_mark<PT>(&clk, KVR_PHASE_STAGE_WAIT);
          const int32_t ellp = ell_sh[cur];
          const int32_t ell_r = ellp < Ln ? ellp : Ln;
          const int32_t h = match_pipe(P, (int32_t)job.s.arena_sel, rootf + best * kRootFilterWords, qn, Ln, Lp,
                                       ell_r, paths.of(best));
          if (h == ell_r) {
            count_mtok(mtok_sh, best, h, &h_sh[cur ^ 1u][best]);
            add_rel(&f.matched, 1u);
            early = 1;
          } else {
            early = 2;
          }
          clock_mark<PT>(&clk, KVR_PHASE_MATCH);
        }
        if (!pipe_wait(&f.evicted, issued, &f, g, r, jg, 5)) break;
        clock_mark<PT>(&clk, KVR_PHASE_EVICTOR_WAIT);
        if (lane == 0) {
          early_sh[issued & 1u] = early;
          __hip_atomic_store(&f.ework, best, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
          __hip_atomic_store(&f.ework_size, job.final_size, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
        issued += 1;
        last_job = k;
        st_rel(&f.handed, issued);
      }
    }
    st_rel(&f.end, 1u);
    if (lane == 0) {
      rh->route_digest = chain;
      rh->queries = routed;
      if constexpr (PT)
        for (int p = 0; p < KVR_PHASES; ++p) rh->phase_ticks[p] += clk.acc[p];
    }
  } else if (wave == 1) {
    // ---------------------------------------------------------- evicting wave
    PhaseClock clk;
    clock_start<PT>(&clk);
    uint32_t done = 0;
    for (;;) {
      // the next insertion, or the end (the bound on the wait restarts
      // whenever the routing wave routes a query)
      uint32_t spins = 0, seen = ld_acq(&f.routed);
      bool quit = false;
      for (;;) {
        if (ld_acq(&f.handed) > done) break;
        const uint32_t now = ld_acq(&f.routed);
        if (now != seen) {
          seen = now;
          spins = 0;
        }
        if (ld_acq(&f.end) && ld_acq(&f.handed) == done) {
          quit = true;
          break;
        }
        if (__hip_atomic_load(&f.stop, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP)) {
          quit = true;
          break;
        }
        if (++spins > kSpinLimit) {
          const int64_t dbg[4] = {96, (int64_t)done, 0, 0};
          pipe_stop(g, &f, r, a.j0, KVR_DEV_INTERNAL, dbg);
          quit = true;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      if (quit) break;
      clock_mark<PT>(&clk, KVR_PHASE_E_IDLE);
      const EvictJob& job = job_sh[done & 1u];
      const uint32_t w = job.worker;
      const Ptrs Pw = worker_ptrs(a.ws, a.L, r, w);
      // the routed worker's h of the next query q_kq+1, first on the tree
      // after the load: exact when it ends where q_kq+1 leaves the inserted
      // path (depth LCP(q_kq, q_kq+1), marked, so no eviction shortens it;
      // no child can match there later, as evictions only remove tokens),
      // else taken again after the evictions
      const uint32_t kq = (uint32_t)(job.ia.jg - a.j0);
      const bool has_next = kq + 1u < a.n;
      const uint32_t early = early_sh[done & 1u];
      bool exact = early != 2u;
      int32_t Lnx = 0, ell_r = 0;
      const int32_t* qnx = smem + ((kq + 1u) & 1u) * qstride;
      if (has_next) {
        if (!pipe_wait(&f.staged, (kq + 1u) * nh, &f, g, r, job.ia.jg, 13)) break;
        Lnx = (int32_t)(a.offsets[kq + 2] - a.offsets[kq + 1]);
        const int32_t ellp = ell_sh[kq & 1u];
        ell_r = ellp < Lnx ? ellp : Lnx;
      }
      if (has_next && early == 0u) {
        const int32_t h = match_pipe(Pw, (int32_t)job.s.arena_sel, rootf + w * kRootFilterWords, qnx, Lnx, job.L,
                                     ell_r, paths.of(w));
        exact = h == ell_r;
        if (exact) {
          count_mtok(mtok_sh, w, h, &h_sh[(kq + 1u) & 1u][w]);
          add_rel(&f.matched, 1u);
        }
        clock_mark<PT>(&clk, KVR_PHASE_E_MATCH);
      }
      int64_t dbg[4] = {0, 0, 0, 0};
      const uint32_t err = rlt_insert_back<PT>(Pw, job, ustage, dbg, &clk, KVR_PHASE_E_EVICT, KVR_PHASE_E_FINISH);
      if (err) {
        pipe_stop(g, &f, r, job.ia.jg, err, dbg);
        break;
      }
      if (has_next && !exact) {
        count_mtok(mtok_sh, w,
                   match_pipe(Pw, -1, rootf + w * kRootFilterWords, qnx, Lnx, job.L, ell_r, paths.of(w)),
                   &h_sh[(kq + 1u) & 1u][w]);
        add_rel(&f.matched, 1u);
        clock_mark<PT>(&clk, KVR_PHASE_E_MATCH);
      }
      if (lane == 0) __hip_atomic_store(&f.ework, kNoWorker, __ATOMIC_SEQ_CST, __HIP_MEMORY_SCOPE_WORKGROUP);
      done += 1;
      st_rel(&f.evicted, done);
      // the helpers may be matching q_s+1 (s = the last query routed) and
      // have left this worker to this wave: take that match unless a helper
      // claimed it (or the worker is the one q_s went to)
      {
        const uint32_t rt = __hip_atomic_load(&f.routed, __ATOMIC_SEQ_CST, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (rt > 0 && rt < a.n) {
          const uint32_t sq = rt - 1u, sc = sq & 1u;
          unsigned long long old = 0ull;
          if ((uint32_t)best_sh[sc] != w && lane == 0) old = atomicOr(&f.claim[sc], 1ull << w);
          old = ((unsigned long long)(uint32_t)__builtin_amdgcn_readlane((int)(old >> 32), 0) << 32) |
                (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)old, 0);
          if ((uint32_t)best_sh[sc] != w && !(old & (1ull << w))) {
            if (!pipe_wait(&f.staged, rt * nh, &f, g, r, a.j0 + rt, 12)) break;
            const int32_t Ls = (int32_t)(a.offsets[sq + 1] - a.offsets[sq]);
            const int32_t Lnx = (int32_t)(a.offsets[sq + 2] - a.offsets[sq + 1]);
            const int32_t ellp = ell_sh[sc];
            const int32_t ell_r = ellp < Lnx ? ellp : Lnx;
            const int32_t ell = ell_r < Ls ? ell_r : Ls;
            Ptrs Pw = worker_ptrs(a.ws, a.L, r, w);
            count_mtok(mtok_sh, w,
                       match_pipe(Pw, -1, rootf + w * kRootFilterWords, smem + (sc ^ 1u) * qstride, Lnx, h_sh[sc][w],
                                  ell, paths.of(w)),
                       &h_sh[sc ^ 1u][w]);
            add_rel(&f.matched, 1u);
          }
        }
      }
    }
    if constexpr (PT)
      if (lane == 0)
        for (int p = KVR_PHASE_E_EVICT; p < KVR_PHASES; ++p)
          if (p <= KVR_PHASE_E_IDLE || p == KVR_PHASE_E_MATCH) atomicAdd(&eticks_sh[p], (unsigned long long)clk.acc[p]);
  } else {
    // ---------------------------------------------------------- helper waves
    const uint32_t hw = wave - 2u;  // 0 .. nh-1
    PhaseClock clk;
    clock_start<PT>(&clk);
    for (uint32_t k = 0; k < a.n; ++k) {
      const uint32_t cur = k & 1u;
      const uint64_t jg = a.j0 + k;
      const uint64_t o0 = a.offsets[k];
      const int32_t Lp = (int32_t)(a.offsets[k + 1] - o0);
      const int64_t t = a.arrival[k];
      const bool has_next = k + 1 < a.n;
      const uint64_t n0 = has_next ? a.offsets[k + 1] : 0;
      const int32_t Ln = has_next ? (int32_t)(a.offsets[k + 2] - n0) : 0;
      const int32_t* qs = smem + cur * qstride;
      int32_t* qn = smem + (cur ^ 1u) * qstride;
      // stage q_k+1 once the routing wave has begun q_k
      if (has_next) {
        if (!pipe_wait(&f.top, k + 1, &f, g, r, jg, 6)) break;
        clock_mark<PT>(&clk, KVR_PHASE_H_WAIT);
        stage_next(a.tokens, n0, Ln, qn, qs, Lp, hw * KVR_WAVE + (uint32_t)lane, nh * KVR_WAVE, &ell_sh[cur]);
        add_rel(&f.staged, 1u);
        clock_mark<PT>(&clk, KVR_PHASE_H_STAGE);
      }
      if (!pipe_wait(&f.routed, k + 1, &f, g, r, jg, 7)) break;
      clock_mark<PT>(&clk, KVR_PHASE_H_WAIT);
      const uint32_t best = (uint32_t)best_sh[cur];
      const uint32_t rn = rn_sh[cur];
      // completions and decay at the next arrival (the first helper)
      if (hw == 0 && has_next) {
        if ((uint32_t)lane < W)
          complete_and_decay(a.C, worker_ptrs(a.ws, a.L, r, (uint32_t)lane), a.arrival[k + 1], t);
        st_rel(&f.decayed, k + 2);
        clock_mark<PT>(&clk, KVR_PHASE_H_OTHER);
      }
      const int32_t hb = h_sh[cur][best];
      if (hw == nh - 1u) {
        // the last helper ranks the new leaf (on the tree before the
        // insertion; the worker's previous evictions come first)
        if (hb < Lp) {
          if (!pipe_wait<true>(&f.ework, best, &f, g, r, jg, 8)) break;
          rank_for_insertion(worker_ptrs(a.ws, a.L, r, best), paths.of(best), qs, hb, &rank_sh, &rank_ready_sh);
          clock_mark<PT>(&clk, KVR_PHASE_H_OTHER);
        }
      } else if (hw < ndraw) {
        // the drawing helpers compute the draw words, a round of 2*nd words
        // at a time, and publish each round they complete
        uint32_t* rw = rwb + (size_t)cur * a.rcap;
        uint32_t rounds = 0;
        for (uint32_t base = 0; base < rn; base += 2u * nd) {
          const uint32_t d0 = base + hw * KVR_WAVE + (uint32_t)lane, d1 = d0 + nd;
          const uint64_t w0 = philox_word0(jg, best, d0, 0ull, a.C.seed, r);
          const uint64_t w1 = philox_word0(jg, best, d1, 0ull, a.C.seed, r);
          if (d0 < rn) rw[d0] = (uint32_t)(w0 >> 32);
          if (d1 < rn) rw[d1] = (uint32_t)(w1 >> 32);
          ++rounds;
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
          if (lane == 0) __hip_atomic_store(&prog_sh[cur][hw], rounds, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
        clock_mark<PT>(&clk, KVR_PHASE_H_DRAW);
      }
      // h of q_k+1 on every worker but the routed one, the worker whose
      // evictions may still run taken last
      if (has_next) {
        if (!pipe_wait(&f.staged, (k + 1) * nh, &f, g, r, jg, 9)) break;
        clock_mark<PT>(&clk, KVR_PHASE_H_WAIT);
        const int32_t ellp = ell_sh[cur];
        const int32_t ell_r = ellp < Ln ? ellp : Ln;
        const int32_t ell = ell_r < Lp ? ell_r : Lp;
        const uint32_t prev = k > 0 ? (uint32_t)best_sh[cur ^ 1u] : 0u;
        bool ok = true;
        const uint32_t mine = take_matches_pipe<kPipeItemUnroll>(a, r, W, cur, best, prev, qn, Ln, ell, h_sh[cur], h_sh[cur ^ 1u], &f,
                                                mtok_sh, rootf, paths);
        // this wave's matches, published at once
        add_rel(&f.matched, mine);
        clock_mark<PT>(&clk, KVR_PHASE_H_MATCH);
        if (!ok) break;
      }
    }
    if constexpr (PT)
      if (lane == 0)
        for (int p = KVR_PHASE_H_STAGE; p <= KVR_PHASE_H_MATCH; ++p) atomicAdd(&eticks_sh[p], (unsigned long long)clk.acc[p]);
  }
  __syncthreads();
  if (threadIdx.x < W) worker_ptrs(a.ws, a.L, r, threadIdx.x).hdr->matched_tokens += mtok_sh[threadIdx.x];
  if (threadIdx.x == 0) {
    if constexpr (PT)
      for (int p = KVR_PHASE_E_EVICT; p < KVR_PHASES; ++p) rh->phase_ticks[p] += eticks_sh[p];
    if (!f.stop && a.n > 0) {
      rh->tprev = a.arrival[a.n - 1];
      if (r == 0) g->last_arrival = a.arrival[a.n - 1];
    }
  }
}

// Zero n 32-bit words (in-progress counts of continuous batching).
__global__ void zero_words_kernel(uint32_t* p, uint64_t n) {
  for (uint64_t x = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; x < n; x += (uint64_t)gridDim.x * blockDim.x)
    p[x] = 0u;
}

__global__ void init_kernel(char* ws, Layout L, double rls_p0) {
  const uint64_t RW = (uint64_t)L.R * L.W;
  const uint64_t tid = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid == 0) {
    GlobalHdr* g = reinterpret_cast<GlobalHdr*>(ws + L.off_global);
    g->status = 0;
    g->err_taken = 0;
    g->last_arrival = 0;
    g->err_check = 0;
    g->err_replica = 0;
    g->err_query = 0;
    g->err_val[0] = g->err_val[1] = g->err_val[2] = 0;
  }
  if (tid < L.R) {
    ReplicaHdr h;
    h.tprev = 0;
    h.queries = 0;
    h.route_digest = 0;
    for (int k = 0; k < KVR_PHASES; ++k) h.phase_ticks[k] = 0;
    for (int k = 0; k < 12; ++k) h.pad[k] = 0;
    reinterpret_cast<ReplicaHdr*>(ws + L.off_rhdr)[tid] = h;
  }
  if (tid < RW) {
    init_worker(worker_ptrs(ws, L, (uint32_t)(tid / L.W), (uint32_t)(tid % L.W)), rls_p0);
    if (L.has_router) init_worker(router_ptrs(ws, L, (uint32_t)(tid / L.W), (uint32_t)(tid % L.W)), rls_p0);
  }
}

// Batch checks before any state changes: lengths (with cached responses, a
// prompt of at least one token before the response) and arrival order.
__global__ void validate_kernel(char* ws, Layout L, const uint64_t* offsets, const int64_t* arrival,
                                const uint16_t* out_len, int32_t resp, uint32_t n) {
  GlobalHdr* g = reinterpret_cast<GlobalHdr*>(ws + L.off_global);
  uint32_t bits = 0;
  for (uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n;
       j += (uint64_t)gridDim.x * blockDim.x) {
    const uint64_t o0 = offsets[j], o1 = offsets[j + 1];
    if (o1 <= o0 || o1 - o0 > L.maxL) bits |= KVR_DEV_BAD_LENGTH;
    if (resp && o1 - o0 <= (uint64_t)query_out_len(out_len, j)) bits |= KVR_DEV_BAD_LENGTH;
    const int64_t prev = j == 0 ? g->last_arrival : arrival[j - 1];
    if (arrival[j] < prev) bits |= KVR_DEV_BAD_ARRIVAL;
  }
  if (bits) atomicOr(&g->status, bits);
}

// Token ids must be >= 0 (checked only when the offsets passed).
__global__ void validate_tokens_kernel(char* ws, Layout L, const int32_t* tokens,
                                       const uint64_t* offsets, uint32_t n) {
  GlobalHdr* g = reinterpret_cast<GlobalHdr*>(ws + L.off_global);
  if (__atomic_load_n(&g->status, __ATOMIC_RELAXED)) return;
  const uint64_t b = offsets[0], e = offsets[n];
  uint32_t bad = 0;
  for (uint64_t x = b + (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; x < e;
       x += (uint64_t)gridDim.x * blockDim.x)
    if (tokens[x] < 0) bad = 1;
  if (__ballot(bad != 0) && lane_id() == 0) atomicOr(&g->status, (uint32_t)KVR_DEV_BAD_TOKEN);
}

// Final state of every (replica, worker): one wave each, for the workers
// w0 .. w0 + gridDim.x - 1 (index r * W + i).  The digest walk's FIFO is
// fifo + (widx - w0) * fifo_words (fifo_words / 2 entries), or the worker's
// scratch region when fifo is null; the records go to out[widx - w0].  An
// inconsistent tree or a FIFO too short raises KVR_DEV_INTERNAL.
__global__ void __launch_bounds__(64) stats_kernel(char* ws, Layout L, uint64_t w0, uint64_t* fifo,
                                                   uint64_t fifo_words, kvr_worker_stats* out) {
  const uint64_t widx = w0 + blockIdx.x;
  const uint32_t r = (uint32_t)(widx / L.W), i = (uint32_t)(widx % L.W);
  kvr_worker_stats* o = out + blockIdx.x;
  uint64_t* q = fifo ? fifo + (uint64_t)blockIdx.x * fifo_words : nullptr;
  bool ok = worker_stats(worker_ptrs(ws, L, r, i), o, q, fifo_words / 2);
  if (L.has_router) {
    // the router's tree of the worker (its walk reuses the same FIFO once
    // the cache's is done): contents digest and evictions
    wave_mem_sync();
    Ptrs Pr = router_ptrs(ws, L, r, i);
    kvr_worker_stats t;
    ok = worker_stats(Pr, &t, q, fifo_words / 2) && ok;
    if (lane_id() == 0) {
      o->router_resident = t.resident;
      o->router_digest_sum = t.digest_sum;
      o->router_digest_xor = t.digest_xor;
      o->router_evictions = Pr.hdr->evictions;
    }
  }
  if (!ok && lane_id() == 0) atomicOr(&reinterpret_cast<GlobalHdr*>(ws + L.off_global)->status, (uint32_t)KVR_DEV_INTERNAL);
}

// ---------------------------------------------------------------- launchers (host)

size_t step_lds_bytes(uint32_t maxL, uint32_t W, uint32_t ucap, uint32_t rcap, uint32_t path_sets) {
  return 2 * (size_t)((maxL + 3u) & ~3u) * sizeof(int32_t) + (size_t)rcap * sizeof(uint32_t) +
         (size_t)path_sets * W * (3 * kPathMax + 1) * sizeof(int32_t) + (size_t)ucap * 4u * sizeof(int32_t);
}


// Dynamic LDS of the pipelined step kernel: two query buffers, the draw
// words of two insertions (rcap each), the match paths, the root filters,
// ucap staged candidates.
size_t step_lds_bytes_pipe(uint32_t maxL, uint32_t W, uint32_t ucap, uint32_t rcap) {
  return 2 * (size_t)((maxL + 3u) & ~3u) * sizeof(int32_t) + 2 * (size_t)rcap * sizeof(uint32_t) +
         (size_t)W * (3 * kPathMax + 1) * sizeof(int32_t) + (size_t)W * kRootFilterWords * sizeof(uint32_t) +
         (size_t)ucap * 4u * sizeof(int32_t);
}

hipError_t launch_init(char* ws, const Layout& L, double rls_p0, hipStream_t st) {
  const uint64_t work = (uint64_t)L.R * L.W > L.R ? (uint64_t)L.R * L.W : L.R;
  const uint32_t blocks = (uint32_t)((work + 255) / 256);
  hipLaunchKernelGGL(init_kernel, dim3(blocks), dim3(256), 0, st, ws, L, rls_p0);
  if (L.pin_stride) {
    const uint64_t words = (uint64_t)L.R * L.W * L.pin_stride / 4u;
    hipLaunchKernelGGL(zero_words_kernel, dim3(1024), dim3(256), 0, st, reinterpret_cast<uint32_t*>(ws + L.off_pin),
                       words);
  }
  return hipGetLastError();
}

hipError_t launch_step(const StepArgs& a, hipStream_t st) {
  const uint32_t blocks_v = (a.n + 255) / 256 < 1024 ? (a.n + 255) / 256 : 1024;
  hipLaunchKernelGGL(validate_kernel, dim3(blocks_v ? blocks_v : 1), dim3(256), 0, st, a.ws, a.L,
                     a.offsets, a.arrival, a.out_len, a.C.cache_responses, a.n);
  hipLaunchKernelGGL(validate_tokens_kernel, dim3(1024), dim3(256), 0, st, a.ws, a.L, a.tokens,
                     a.offsets, a.n);
  const uint32_t waves = a.L.W < kMaxWavesPerBlock ? a.L.W : kMaxWavesPerBlock;
  const size_t lds = step_lds_bytes(a.L.maxL, a.L.W, a.ucap, a.rcap, a.L.has_router ? 2u : 1u);
  const bool rt = a.L.has_router != 0, ba = a.L.beta > 1;
  if (a.pipe) {
    const size_t lds_p = step_lds_bytes_pipe(a.L.maxL, a.L.W, a.ucap, a.rcap);
    const bool wide = a.L.W >= kPipeWideWorkers;
    if (a.C.phase_timers) {
      if (wide)
        hipLaunchKernelGGL((step_kernel_pipe<true, kPipeWavesWide>), dim3(a.L.R), dim3(64 * kPipeWavesWide), lds_p, st,
                           a);
      else
        hipLaunchKernelGGL((step_kernel_pipe<true, kPipeWaves>), dim3(a.L.R), dim3(64 * kPipeWaves), lds_p, st, a);
    } else {
      if (wide)
        hipLaunchKernelGGL((step_kernel_pipe<false, kPipeWavesWide>), dim3(a.L.R), dim3(64 * kPipeWavesWide), lds_p,
                           st, a);
      else
        hipLaunchKernelGGL((step_kernel_pipe<false, kPipeWaves>), dim3(a.L.R), dim3(64 * kPipeWaves), lds_p, st, a);
    }
  } else if (rt && ba)
    hipLaunchKernelGGL((step_kernel<true, true, false>), dim3(a.L.R), dim3(64 * waves), lds, st, a);
  else if (rt)
    hipLaunchKernelGGL((step_kernel<true, false, false>), dim3(a.L.R), dim3(64 * waves), lds, st, a);
  else if (ba)
    hipLaunchKernelGGL((step_kernel<false, true, false>), dim3(a.L.R), dim3(64 * waves), lds, st, a);
  else if (a.C.phase_timers)
    hipLaunchKernelGGL((step_kernel<false, false, true>), dim3(a.L.R), dim3(64 * waves), lds, st, a);
  else
    hipLaunchKernelGGL((step_kernel<false, false, false>), dim3(a.L.R), dim3(64 * waves), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_stats(char* ws, const Layout& L, hipStream_t st) {
  hipLaunchKernelGGL(stats_kernel, dim3(L.R * L.W), dim3(64), 0, st, ws, L, 0ull, nullptr, 0ull,
                     reinterpret_cast<kvr_worker_stats*>(ws + L.off_stats));
  return hipGetLastError();
}

// ---------------------------------------------------------------- allocation-free statistics
//
// kvr_stats_noalloc keeps the digest walk's FIFO and the staged records in
// this array instead of the workspace; one copy per device, for the life of
// the process.  Host code uses its address from hipGetSymbolAddress, never
// its name.
constexpr size_t kScratchBytes = 32ull << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

// The device address of `scratch` on the current device (looked up once per
// device).
hipError_t noalloc_scratch(int device, void** ptr, size_t* bytes) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[device] = p;
  }
  *ptr = g_scratch_ptr[device];
  *bytes = kScratchBytes;
  return hipSuccess;
}

// Workers w0 .. w0 + n - 1 with their FIFOs (fifo_words each) and records
// in caller-given device memory.
hipError_t launch_stats_into(char* ws, const Layout& L, uint64_t w0, uint32_t n, uint64_t* fifo, uint64_t fifo_words,
                             kvr_worker_stats* out, hipStream_t st) {
  hipLaunchKernelGGL(stats_kernel, dim3(n), dim3(64), 0, st, ws, L, w0, fifo, fifo_words, out);
  return hipGetLastError();
}

static const void* const kStepKernels[9] = {
    reinterpret_cast<const void*>(step_kernel_pipe<false, kPipeWaves>),
    reinterpret_cast<const void*>(step_kernel_pipe<true, kPipeWaves>),
    reinterpret_cast<const void*>(step_kernel_pipe<false, kPipeWavesWide>),
    reinterpret_cast<const void*>(step_kernel_pipe<true, kPipeWavesWide>),
    reinterpret_cast<const void*>(step_kernel<false, false, false>),
    reinterpret_cast<const void*>(step_kernel<false, true, false>),
    reinterpret_cast<const void*>(step_kernel<true, false, false>),
    reinterpret_cast<const void*>(step_kernel<true, true, false>),
    reinterpret_cast<const void*>(step_kernel<false, false, true>)};

// Static LDS of the step kernels (their __shared__ variables, the largest),
// from the compiled kernels' attributes.
hipError_t step_static_lds(size_t* bytes) {
  size_t mx = 0;
  for (const void* f : kStepKernels) {
    hipFuncAttributes fa;
    const hipError_t e = hipFuncGetAttributes(&fa, f);
    if (e != hipSuccess) return e;
    if (fa.sharedSizeBytes > mx) mx = fa.sharedSizeBytes;
  }
  *bytes = mx;
  return hipSuccess;
}

hipError_t set_step_lds_limit(size_t bytes) {
  for (const void* f : kStepKernels) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace kvr
