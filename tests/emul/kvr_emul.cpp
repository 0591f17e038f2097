// kvr_emul.cpp - sequential CPU replay of the step kernel's logic (tests only).
// Includes the kernel's per-wave logic unchanged (one lane) and orchestrates
// it the way step_kernel does for each replica: completions and decay, match
// on every worker, LBGR score and argmin, commit, RLT insert.
#include "emul_wave.h"
#include "../../paper_2601_18999_amd/csrc/kvr_core.h"

#include <vector>

using namespace kvr;

extern "C" int emul_run(const kvr_config* cfg, uint64_t n, const int32_t* tokens, const uint64_t* offsets,
                        const int64_t* arrival, const uint16_t* out_len, int32_t* route, int32_t* hits,
                        int32_t* all_hits, kvr_worker_stats* out, char* ws_out, uint32_t ucap_in) {
  Layout L = make_layout(*cfg);
  std::vector<uint64_t> mem(ws_out ? 0 : (L.total + 7) / 8);
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
  const uint32_t W = L.W;
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
    for (uint32_t i = 0; i < W; ++i) init_worker(worker_ptrs(ws, L, r, i), cfg->rls_p0);
  for (uint32_t r = 0; r < L.R; ++r) {
    int64_t tprev = 0;
    for (uint64_t j = 0; j < n; ++j) {
      const int32_t* qs = tokens + offsets[j];
      const int32_t Lq = (int32_t)(offsets[j + 1] - offsets[j]);
      const int64_t t = arrival[j];
      const int32_t olen = out_len ? (int32_t)out_len[j] : 4;
      int32_t h[kMaxWorkers];
      double eh[kMaxWorkers], ch[kMaxWorkers];
      for (uint32_t i = 0; i < W; ++i) complete_and_decay(C, worker_ptrs(ws, L, r, i), t, tprev);
      for (uint32_t i = 0; i < W; ++i) {
        Ptrs P = worker_ptrs(ws, L, r, i);
        h[i] = match_lcp(P, P.hdr->arena_sel, qs, Lq);
        P.hdr->matched_tokens += (uint64_t)h[i];
      }
      for (uint32_t i = 0; i < W; ++i) eh[i] = lbgr_score(C, worker_ptrs(ws, L, r, i).hdr, h[i], Lq, &ch[i]);
      uint32_t best = 0;
      for (uint32_t i = 1; i < W; ++i)
        if (eh[i] < eh[best]) best = i;
      tprev = t;
      Ptrs P = worker_ptrs(ws, L, r, best);
      uint32_t err = commit_route(C, P, ch[best], h[best], Lq, t, olen);
      if (route) route[r * n + j] = (int32_t)best;
      if (hits) hits[r * n + j] = h[best];
      if (all_hits)
        for (uint32_t i = 0; i < W; ++i) all_hits[(r * n + j) * W + i] = h[i];
      if (!err) {
        InsertArgs ia;
        ia.seed = C.seed;
        ia.jg = j;
        ia.worker = best;
        ia.replica = r;
        ia.B = L.B;
        ia.rn = 0;
        ia.rw = nullptr;
        err = rlt_insert(P, ia, qs, Lq, h[best], ustage, nullptr);
      }
      if (err) return (int)err;
    }
  }
  for (uint32_t r = 0; r < L.R; ++r)
    for (uint32_t i = 0; i < W; ++i) worker_stats(worker_ptrs(ws, L, r, i), out + (uint64_t)r * W + i);
  return 0;
}
