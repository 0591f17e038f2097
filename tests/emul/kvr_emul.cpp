// kvr_emul.cpp - sequential CPU replay of the step kernel's logic (tests only).
// Includes the kernel's per-wave logic unchanged (one lane) and orchestrates
// it the way step_kernel does for each replica: completions and decay, match
// on every worker, LBGR score and argmin, commit, RLT insert.
#include "emul_wave.h"
#include "../../paper_2601_18999_amd/csrc/kvr_core.h"

#include <cstring>
#include <vector>

using namespace kvr;

// next-query matches on the routed worker that the pipelined order had to
// take again after the evictions (last emul_run call)
static uint64_t g_pipe_unsafe = 0, g_pipe_steps = 0;
extern "C" uint64_t emul_pipe_unsafe(void) { return g_pipe_unsafe; }
extern "C" uint64_t emul_pipe_steps(void) { return g_pipe_steps; }

extern "C" int emul_run(const kvr_config* cfg, uint64_t n, const int32_t* tokens, const uint64_t* offsets,
                        const int64_t* arrival, const uint16_t* out_len, int32_t* route, int32_t* hits,
                        int32_t* all_hits, kvr_worker_stats* out, char* ws_out, uint32_t ucap_in) {
  Layout L = make_layout(*cfg);
  std::vector<uint64_t> mem(ws_out ? 0 : (L.total + 7) / 8);  // zeroed: the in-progress counts start at 0
  char* ws = ws_out ? ws_out : reinterpret_cast<char*>(mem.data());
  Consts C;
  C.seed = cfg->seed;
  C.alpha_cached = cfg->alpha_cached;
  C.alpha_miss = cfg->alpha_miss;
  C.rho = cfg->rho;
  C.lr = cfg->lr;
  C.nlms_eps = cfg->nlms_eps;
  C.rls_p0 = cfg->rls_p0;
  C.dt_us = cfg->decay_interval_us;
  C.true_cached_us = cfg->true_cached_us;
  C.true_miss_us = cfg->true_miss_us;
  C.true_out_us = cfg->true_out_us;
  C.update = cfg->update;
  C.evict = cfg->evict;
  C.cache_responses = cfg->cache_responses;
  const bool resp = cfg->cache_responses != 0;
  const bool rtree = L.has_router != 0;
  const uint32_t W = L.W;
  // the order of the pipelined step kernel (RLT, no router tree, no
  // continuous batching, prompts only)
  const bool pipe = C.evict == KVR_EVICT_RLT && !rtree && L.beta == 1 && !resp;
  g_pipe_unsafe = g_pipe_steps = 0;
  // candidate list staging buffer (LDS on the device)
  const uint32_t ucap = ucap_in;
  std::vector<int32_t> ubuf(4 * (size_t)(ucap ? ucap : 1));
  UStage ustage;
  ustage.node = ubuf.data();
  ustage.len = ubuf.data() + ucap;
  ustage.top = ubuf.data() + 2 * ucap;
  ustage.par = ubuf.data() + 3 * ucap;
  ustage.cap = ucap;
  for (uint32_t r = 0; r < L.R; ++r)
    for (uint32_t i = 0; i < W; ++i) {
      init_worker(worker_ptrs(ws, L, r, i), cfg->rls_p0);
      if (rtree) init_worker(router_ptrs(ws, L, r, i), cfg->rls_p0);
    }
  if (L.pin_stride) std::memset(ws + L.off_pin, 0, (size_t)L.R * W * L.pin_stride);
  std::vector<uint32_t> rwbuf;
  // per-worker match paths (LDS on the device)
  std::vector<int32_t> pbuf((size_t)W * (3 * kPathMax + 1));
  auto path_of = [&](uint32_t i) {
    PathRef p;
    p.node = pbuf.data() + (size_t)i * kPathMax;
    p.start = pbuf.data() + (size_t)(W + i) * kPathMax;
    p.end = pbuf.data() + (size_t)(2 * W + i) * kPathMax;
    p.cnt = pbuf.data() + (size_t)3 * W * kPathMax + i;
    return p;
  };
  // the router trees' recorded matches (approximate router)
  std::vector<int32_t> rbuf((size_t)W * (3 * kPathMax + 1));
  auto rpath_of = [&](uint32_t i) {
    PathRef p;
    p.node = rbuf.data() + (size_t)i * kPathMax;
    p.start = rbuf.data() + (size_t)(W + i) * kPathMax;
    p.end = rbuf.data() + (size_t)(2 * W + i) * kPathMax;
    p.cnt = rbuf.data() + (size_t)3 * W * kPathMax + i;
    return p;
  };
  for (uint32_t r = 0; r < L.R; ++r) {
    // the schedule of step_kernel for one replica, one batch: completions of
    // query 0 and full matches first; then per query the scores, route,
    // commit and insertion, the routed worker's match of the next query, the
    // completions at the next arrival, the router's tree of the routed
    // worker, and the next query's matches on the other workers.  h = the
    // caches' matches, g = the router trees' (approximate router); the
    // router scores with est = g or h.
    int32_t h[2][kMaxWorkers], g[2][kMaxWorkers];
    int32_t(*est)[kMaxWorkers] = rtree ? g : h;
    int64_t tprev = 0;
    if (n > 0) {
      for (uint32_t i = 0; i < W; ++i) complete_and_decay(C, worker_ptrs(ws, L, r, i), arrival[0], tprev);
      const int32_t L0 = (int32_t)(offsets[1] - offsets[0]);
      const int32_t L0q = resp ? L0 - query_out_len(out_len, 0) : L0;
      for (uint32_t i = 0; i < W; ++i) {
        Ptrs P = worker_ptrs(ws, L, r, i);
        h[0][i] = match_lcp(P, P.hdr->arena_sel, tokens + offsets[0], L0q, path_of(i));
        if (rtree) {
          Ptrs Pr = router_ptrs(ws, L, r, i);
          g[0][i] = match_lcp(Pr, Pr.hdr->arena_sel, tokens + offsets[0], L0q, rpath_of(i));
        }
        P.hdr->matched_tokens += (uint64_t)est[0][i];
      }
    }
    for (uint64_t j = 0; j < n; ++j) {
      const int cur = (int)(j & 1u);
      const int32_t* qs = tokens + offsets[j];
      // path Lp (inserted) and prompt Lq (matched, scored, committed)
      const int32_t Lp = (int32_t)(offsets[j + 1] - offsets[j]);
      const int64_t t = arrival[j];
      const int32_t olen = query_out_len(out_len, j);
      const int32_t Lq = resp ? Lp - olen : Lp;
      const bool has_next = j + 1 < n;
      const int32_t* qn = has_next ? tokens + offsets[j + 1] : nullptr;
      const int32_t Ln = has_next ? (int32_t)(offsets[j + 2] - offsets[j + 1]) : 0;
      const int32_t Lnq = has_next && resp ? Ln - query_out_len(out_len, j + 1) : Ln;
      double eh[kMaxWorkers], ch[kMaxWorkers];
      RouteView view[kMaxWorkers];
      for (uint32_t i = 0; i < W; ++i) {
        view[i] = load_view(worker_ptrs(ws, L, r, i).hdr);
        eh[i] = lbgr_score(C, view[i], est[cur][i], Lq, &ch[i]);
      }
      uint32_t best = 0;
      for (uint32_t i = 1; i < W; ++i)
        if (eh[i] < eh[best]) best = i;
      // the baseline routers, as step_kernel's route_choice takes them
      if (cfg->router == KVR_ROUTE_RANDOM) {
        best = (uint32_t)__umul64hi(philox_word0(j, 0ull, 0ull, 1ull, C.seed, r), (uint64_t)W);
      } else if (cfg->router == KVR_ROUTE_ROUND_ROBIN) {
        best = (uint32_t)(j % W);
      } else if (cfg->router == KVR_ROUTE_CACHE_AWARE) {
        uint32_t lo = 0, hi = 0, hmax = 0, small = 0;
        auto load = [&](uint32_t i) { return worker_ptrs(ws, L, r, i).hdr->pend_count; };
        auto size = [&](uint32_t i) { return worker_ptrs(ws, L, r, i).hdr->size; };
        for (uint32_t i = 1; i < W; ++i) {
          if (load(i) < load(lo)) lo = i;
          if (load(i) > load(hi)) hi = i;
          if (est[cur][i] > est[cur][hmax]) hmax = i;
          if (size(i) < size(small)) small = i;
        }
        if (load(hi) - load(lo) > (uint32_t)cfg->ca_balance_abs &&
            (double)load(hi) > cfg->ca_balance_rel * (double)load(lo))
          best = lo;
        else if ((double)est[cur][hmax] > cfg->ca_cache_threshold * (double)Lq)
          best = hmax;
        else
          best = small;
      }
      Ptrs P = worker_ptrs(ws, L, r, best);
      uint32_t err = commit_route(C, P, view[best], ch[best], h[cur][best], est[cur][best], Lq, t, olen);
      if (route) route[r * n + j] = (int32_t)best;
      if (hits) hits[r * n + j] = h[cur][best];
      if (all_hits)
        for (uint32_t i = 0; i < W; ++i) all_hits[(r * n + j) * W + i] = est[cur][i];
      // LCP of this path and the next; then of the next prompt with this
      // path (routed cache) and with this prompt (the other caches and
      // every router tree)
      int32_t ellp = 0;
      if (has_next) {
        const int32_t m = Lp < Ln ? Lp : Ln;
        while (ellp < m && qs[ellp] == qn[ellp]) ++ellp;
      }
      const int32_t ell_r = ellp < Lnq ? ellp : Lnq;
      const int32_t ell = ell_r < Lq ? ell_r : Lq;
      // the cached length of the whole path, continued from the prompt's match
      int32_t hins = h[cur][best];
      if (resp && hins == Lq && Lp > Lq) hins = match_incremental(P, P.hdr->arena_sel, qs, Lp, Lq, Lq, path_of(best));
      if (!err) {
        // high halves of the insertion's draw words, as the helper waves
        // compute them on the device
        const uint32_t nload = (uint32_t)(Lp - hins);
        const uint32_t nfree = L.B - P.hdr->size;
        const uint32_t nev = nload > nfree ? nload - nfree : 0u;
        rwbuf.resize(nev ? nev : 1);
        for (uint32_t d = 0; d < nev; ++d) rwbuf[d] = (uint32_t)(philox_word0(j, best, d, 0ull, C.seed, r) >> 32);
        InsertArgs ia;
        ia.seed = C.seed;
        ia.jg = j;
        ia.worker = best;
        ia.replica = r;
        ia.B = L.B;
        ia.rn = nev;
        ia.rw = rwbuf.data();
        ia.prog = nullptr;
        ia.nprog = 0;
        ia.round = 1;
        // the new leaf's rank as the device's last helper wave computes it,
        // from the recorded match path on the tree before the insertion
        int32_t rank = -1;
        uint32_t rank_ready = 0;
        ia.rank = nullptr;
        ia.rank_ready = nullptr;
        if (C.evict == KVR_EVICT_RLT && hins < Lp) {
          rank_for_insertion(P, path_of(best), qs, hins, &rank, &rank_ready);
          ia.rank = &rank;
          ia.rank_ready = &rank_ready;
        }
        if (pipe) {
          // the pipelined kernel's order: the front half of the insertion;
          // the routed worker's h of the next query on the tree before the
          // evictions (exact when it stays on the inserted path, which no
          // eviction touches); the back half; a new match if it was not
          EvictJob job;
          err = rlt_insert_front(P, ia, qs, Lp, hins, path_of(best), nullptr, job);
          int32_t hspec = -1;
          bool safe = false;
          if (!err && has_next) {
            hspec = match_incremental(P, job.s.arena_sel, qn, Lnq, Lp, ell_r, path_of(best));
            safe = hspec == ell_r || job.nev == 0;
          }
          if (!err) err = rlt_insert_back(P, job, ustage, nullptr);
          if (!err && has_next) {
            const int32_t hpost = match_incremental(P, P.hdr->arena_sel, qn, Lnq, Lp, ell_r, path_of(best));
            if (safe && hpost != hspec) return -8;  // the early match was not exact
            g_pipe_unsafe += safe ? 0 : 1;
            g_pipe_steps += 1;
          }
        } else {
          err = C.evict == KVR_EVICT_RLT ? rlt_insert(P, ia, qs, Lp, hins, ustage, path_of(best), nullptr)
                                         : lru_insert(P, ia, qs, Lp, hins, path_of(best), nullptr);
        }
        if (!err && P.beta > 1) err = batch_admit(P, path_of(best), qs, Lp, nullptr);
      }
      if (err) return (int)err;
      if (has_next) {
        h[cur ^ 1][best] = match_incremental(P, P.hdr->arena_sel, qn, Lnq, Lp, ell_r, path_of(best));
        if (!rtree) P.hdr->matched_tokens += (uint64_t)h[cur ^ 1][best];
        for (uint32_t i = 0; i < W; ++i) complete_and_decay(C, worker_ptrs(ws, L, r, i), arrival[j + 1], t);
      }
      if (rtree) {
        // the router adds the prompt to its tree of the routed worker
        Ptrs Pr = router_ptrs(ws, L, r, best);
        InsertArgs ia;
        ia.seed = C.seed;
        ia.jg = j;
        ia.worker = best;
        ia.replica = r;
        ia.B = L.RB;
        ia.rn = 0;
        ia.rw = nullptr;
        ia.prog = nullptr;
        ia.nprog = 0;
        ia.round = 1;
        ia.rank = nullptr;
        ia.rank_ready = nullptr;
        err = lru_insert(Pr, ia, qs, Lq, g[cur][best], rpath_of(best), nullptr);
        if (err) return (int)err;
        if (has_next) {
          g[cur ^ 1][best] = match_incremental(Pr, Pr.hdr->arena_sel, qn, Lnq, Lq, ell, rpath_of(best));
          P.hdr->matched_tokens += (uint64_t)g[cur ^ 1][best];
        }
      }
      if (has_next) {
        for (uint32_t i = 0; i < W; ++i) {
          if (i == best) continue;
          Ptrs Pi = worker_ptrs(ws, L, r, i);
          h[cur ^ 1][i] = match_incremental(Pi, Pi.hdr->arena_sel, qn, Lnq, h[cur][i], ell, path_of(i));
          if (rtree) {
            Ptrs Pr = router_ptrs(ws, L, r, i);
            g[cur ^ 1][i] = match_incremental(Pr, Pr.hdr->arena_sel, qn, Lnq, g[cur][i], ell, rpath_of(i));
          }
          Pi.hdr->matched_tokens += (uint64_t)est[cur ^ 1][i];
        }
      }
      tprev = t;
    }
  }
  for (uint32_t r = 0; r < L.R; ++r)
    for (uint32_t i = 0; i < W; ++i) {
      kvr_worker_stats* o = out + (uint64_t)r * W + i;
      if (!worker_stats(worker_ptrs(ws, L, r, i), o)) return -7;  // the digest walk could not finish
      if (rtree) {
        Ptrs Pr = router_ptrs(ws, L, r, i);
        kvr_worker_stats t;
        if (!worker_stats(Pr, &t)) return -7;
        o->router_resident = t.resident;
        o->router_digest_sum = t.digest_sum;
        o->router_digest_xor = t.digest_xor;
        o->router_evictions = Pr.hdr->evictions;
      }
    }
  return 0;
}

// The draw index of the eviction blocks: from the high half of the word when
// that decides it, else from the whole word.
extern "C" uint32_t emul_draw_index(uint64_t r64, uint32_t n) {
  uint32_t k = 0;
  if (draw_index_hi((uint32_t)(r64 >> 32), n, k)) return k;
  return (uint32_t)__umul64hi(r64, (uint64_t)n);
}

extern "C" int emul_draw_index_decided(uint64_t r64, uint32_t n) {
  uint32_t k = 0;
  return draw_index_hi((uint32_t)(r64 >> 32), n, k) ? 1 : 0;
}
