// kvr_oracle.cpp - plain, slow, single-threaded CPU oracle of the batched
// KV-cache routing/eviction simulation.
//
// TEST INFRASTRUCTURE ONLY.  Only tests/, the smoke entry point and the
// benchmark's CPU-baseline leg may load this library.  It shares no code,
// header, table or helper with the HIP path.
//
// What it computes (one replica, one query at a time, in stream order):
//   * the online model of Sec. 3.1: per worker i a load and a cache state;
//     the cache changes only on the worker a query is routed to (Eq. 3);
//   * cache matching = longest prefix of the query present in the worker's
//     token-level prefix tree (Sec. 3.2 "Cache Matching");
//   * LBGR routing (Algorithm 2, Eq. "LBGR-score", Sec. 4.2, App. A
//     constants): estimated service time + decayed queue load + a per-worker
//     linear residual model, argmin over workers, load increment on the
//     routed worker, release of the remaining load and an online update of
//     the residual model when a query completes, exponential decay every
//     decay interval;
//   * RLT insertion/eviction (Algorithm 1, Sec. 4.1): every token of the
//     path is marked; the marking set is reset to the current token when it
//     would exceed B; a missing token is loaded after evicting, when the
//     cache is full, an unmarked leaf token chosen uniformly at random;
//   * L-LRU (Sec. 3.2): evict the least recently used leaf token.
//
// Representation: one trie node per cached token (a token is a position in
// the prefix tree, i.e. a root path), children kept in an ordered map so a
// depth-first walk visits leaves in lexicographic order of their root paths.
//
// Readings of points the paper leaves open (each one is listed with its
// reason in the design notes of the repository):
//   - by default only the prompt q_j is inserted (synthetic responses never
//     recur); with cache_responses the stream holds complete token paths
//     Gamma_j = q_j || a_j (Sec. 3.2 "Cache Matching and Arrival Model")
//     whose last o_j tokens are the response: the whole path is inserted,
//     while the match, the routing features and the cost use the prompt
//     (the response is not known when the query is routed);
//   - the insertion point (the parent of the token being loaded) is never
//     evicted while its child is loaded, so the tree stays prefix-closed;
//   - with continuous batching of batch size beta the running batch of a
//     worker is the beta - 1 queries routed to it before the current one:
//     their whole paths are pinned (no token on them is evicted), and a
//     path is released when beta - 1 later queries have been routed there;
//     batching changes nothing else (matching, routing, observed latency);
//   - "uniformly at random" = index floor(r * |U| / 2^64) into U sorted by
//     root path, r = word 0 of Philox4x64-10 with key (seed, replica) and
//     counter (global query index, worker, draw index, 0);
//   - if U is empty while the cache is full a new phase is forced
//     (marking set reset to the current token) and U is recomputed;
//   - the hit estimate used by the router is the exact per-worker match, or
//     with router_tree the match against a tree the router keeps per worker:
//     the prompts routed there (the router never sees a response), inserted
//     when routed, under L-LRU eviction of its own budget (App. E: a global
//     tree that drifts from the workers' caches); the routing features and
//     decision use that estimate, the observed latency and the hit counts use
//     the worker's true match;
//   - LBGR quantities are in seconds with the per-1k-token scaling of App. A
//     (features 0.001*h, 0.001*(|q|-h), load, 1);
//   - the residual model is updated by normalised LMS (step = the paper's
//     learning rate) or, optionally, recursive least squares (forgetting
//     factor = the paper's learning rate); update NONE leaves it at zero;
//     the error fed to the update is E minus the prediction of the current
//     model on the features stored at routing time (the squared loss of
//     Sec. 4.2 is minimised at the current parameters);
//   - the observed latency comes from a per-worker FIFO fluid queue whose
//     service time per query is the paper's Cost_ij (Eq. 1) in integer us;
//   - decay ticks are multiples of the decay interval of simulated time;
//     pending completions are applied, in FIFO order, at the first arrival
//     at or after their completion time, before the decay to that arrival.
//
// Floating point: IEEE double, every sum left to right, compiled with
// -ffp-contract=off so no multiply-add is fused.
#include <cstdint>
#include <cstring>
#include <ctime>
#include <deque>
#include <map>
#include <set>
#include <vector>

extern "C" {

// ---------------------------------------------------------------------------
// public structs (ctypes mirrors them in oracle/oracle.py)

typedef struct orc_config {
  uint32_t num_workers;       // M in the paper
  uint32_t cache_tokens;      // B_i (same for every worker)
  uint64_t seed;              // Philox key word 0
  int32_t evict;              // 0 = RLT, 1 = L-LRU
  int32_t update;             // 0 = NLMS, 1 = RLS, 2 = none
  int32_t u_mode;             // 0 = maintained ordered candidate list (RLT) or ordered leaf set
                              // (L-LRU), 1 = recompute U / scan every leaf at each eviction
  int32_t check;              // 1 = check invariants after every step
  double alpha_cached;        // s per 1k tokens (App. A: 0 ms per 1k tokens)
  double alpha_miss;          // s per 1k tokens (App. A: 1000 ms per 1k tokens)
  double rho;                 // decay factor (App. A: 31/32)
  int64_t decay_interval_us;  // Delta t (App. A: 20 ms)
  double lr;                  // App. A: 0.992
  double nlms_eps;
  double rls_p0;
  int64_t true_cached_us;     // observed-latency model, us per cached token
  int64_t true_miss_us;       // us per missed token
  int64_t true_out_us;        // us per output token
  // routing (Sec. 5 "Baselines"): 0 = LBGR, 1 = random, 2 = round robin,
  // 3 = cache-aware (highest hit or least loaded, by a load-balance threshold)
  int32_t router;
  int32_t ca_balance_abs;     // cache-aware: imbalance when max - min in-flight > this ...
  double ca_balance_rel;      // ... and max > this * min
  double ca_cache_threshold;  // cache-aware: best hit / |q| above this routes to the best hit
  // 1 = a path is q_j || a_j with |a_j| = out_len[j]; insert all of it
  int32_t cache_responses;
  // continuous batching with batch size beta (Sec. 3.2, Theorem 2): the
  // paths of the beta - 1 queries routed to a worker before the one being
  // inserted are in progress there and none of their tokens is evicted;
  // 1 = single-query processing (only the insertion point is protected)
  int32_t batch_size;
  // approximate router tree (App. E): 1 = the router estimates h from a tree
  // of its own per worker, holding the prompts routed there (inserted when
  // routed) under its own L-LRU eviction with budget router_tree_tokens
  // (0 = cache_tokens); 0 = the router sees the workers' true caches
  int32_t router_tree;
  uint32_t router_tree_tokens;
} orc_config;

typedef struct orc_worker_stats {
  uint64_t routed, prompt_tokens, hit_tokens, matched_tokens;
  uint64_t loads, evictions, phase, cnt, forced_resets, resident;
  uint64_t digest_sum, digest_xor, marked_count, marked_sum;
  uint64_t completions, pending_depth, pending_max;
  uint64_t latency_sum_us, latency_max_us;
  int64_t backlog_us, last_decay_us;
  double load_est;
  double theta[4];
  // the router's tree of this worker (router_tree = 1): tokens held, digest
  // as above, L-LRU evictions
  uint64_t router_resident, router_digest_sum, router_digest_xor, router_evictions;
} orc_worker_stats;

// Options of orc_run_ex (all optional; zero-initialise).
typedef struct orc_run_opts {
  uint64_t snap_every;       // > 0: snapshot the per-worker state every snap_every queries
  orc_worker_stats* snaps;   // [ceil(n / snap_every) * W] snapshots
  uint64_t time_from;        // first query of the timed window
  double time_budget_s;      // > 0: stop once the window has taken this much thread CPU time
  double window_cpu_s;       // out: thread CPU seconds of the window
  double window_wall_s;      // out: wall seconds of the window
  uint64_t done;             // out: queries processed
} orc_run_opts;

}  // extern "C"

namespace {

// ---------------------------------------------------------------------------
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
// easy as 1, 2, 3", SC'11): ten rounds of two 64x64->128 multiplications,
// key bumped by the Weyl constants between rounds.
const uint64_t kPhiloxM0 = 0xD2E7470EE14C6C93ULL;
const uint64_t kPhiloxM1 = 0xCA5A826395121157ULL;
const uint64_t kPhiloxW0 = 0x9E3779B97F4A7C15ULL;
const uint64_t kPhiloxW1 = 0xBB67AE8584CAA73BULL;

void philox4x64_10(const uint64_t ctr_in[4], const uint64_t key_in[2], uint64_t out[4]) {
  uint64_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
  uint64_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += kPhiloxW0;
      k1 += kPhiloxW1;
    }
    unsigned __int128 p0 = (unsigned __int128)kPhiloxM0 * c[0];
    unsigned __int128 p1 = (unsigned __int128)kPhiloxM1 * c[2];
    uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
    uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    uint64_t n0 = hi1 ^ c[1] ^ k0;
    uint64_t n1 = lo1;
    uint64_t n2 = hi0 ^ c[3] ^ k1;
    uint64_t n3 = lo0;
    c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
  }
  out[0] = c[0]; out[1] = c[1]; out[2] = c[2]; out[3] = c[3];
}

// SplitMix64 finaliser, used only for the cache digest.
uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

// rho^k by square-and-multiply, least significant bit first.
double pow_int(double rho, uint64_t k) {
  double res = 1.0, b = rho;
  while (k) {
    if (k & 1) res = res * b;
    b = b * b;
    k >>= 1;
  }
  return res;
}

struct Node {
  int32_t tok = 0;
  int32_t parent = -1;
  uint32_t mark = 0;      // phase in which the token was last marked (0 = never)
  uint64_t stamp = 0;     // L-LRU access stamp
  uint32_t pin = 0;       // number of in-progress paths through this token
  bool alive = false;
  std::map<int32_t, int32_t> kids;  // child token -> node id, ordered
};

struct Pending {
  int64_t t_route, t_done;
  double chat;   // estimated service time at routing
  double base;   // estimated service time + queue load at routing
  double e_obs;  // observed latency (s)
  double phi[4];
};

struct Worker {
  std::vector<Node> nodes;     // node 0 = root (the empty path)
  std::vector<int32_t> free_ids;
  uint64_t size = 0;           // |S_i| in tokens
  uint32_t phase = 1, cnt = 0; // marking set T = {v : mark(v) == phase}, |T| = cnt
  std::vector<int32_t> U;      // ordered candidate list (RLT, u_mode 0)
  std::set<std::pair<uint64_t, int32_t>> lru_leaves;  // (stamp, id) of every leaf (L-LRU, u_mode 0)
  bool U_valid = false;
  double P = 0.0;              // estimated queue load
  double theta[4] = {0, 0, 0, 0};
  double Pm[16];               // RLS inverse-correlation matrix
  int64_t tl = 0;              // time of the last decay (us)
  int64_t Wb = 0;              // observed-latency backlog (us)
  std::deque<Pending> pend;
  std::deque<std::vector<int32_t>> running;  // paths of the running batch (oldest first)
  orc_worker_stats st;
};

struct Sim {
  orc_config cfg;
  uint32_t replica;
  std::vector<Worker> w;
  std::vector<Worker> rt;  // the router's tree of each worker (router_tree = 1)
  int64_t tprev = 0;
  int error = 0;
};

int32_t new_node(Worker& w, int32_t tok, int32_t parent) {
  int32_t id;
  if (!w.free_ids.empty()) {
    id = w.free_ids.back();
    w.free_ids.pop_back();
  } else {
    id = (int32_t)w.nodes.size();
    w.nodes.emplace_back();
  }
  Node& n = w.nodes[id];
  n.tok = tok;
  n.parent = parent;
  n.mark = 0;
  n.stamp = 0;
  n.pin = 0;
  n.alive = true;
  n.kids.clear();
  w.nodes[parent].kids[tok] = id;
  w.size += 1;
  return id;
}

void remove_leaf(Worker& w, int32_t id) {
  Node& n = w.nodes[id];
  w.nodes[n.parent].kids.erase(n.tok);
  n.alive = false;
  n.kids.clear();
  w.free_ids.push_back(id);
  w.size -= 1;
}

bool is_leaf(const Worker& w, int32_t id) { return id != 0 && w.nodes[id].kids.empty(); }

// U by definition: the leaf tokens of S that are not marked in the current
// phase, minus the pinned insertion point and the tokens of in-progress
// paths, in lexicographic order of their root paths (= pre-order of a
// depth-first walk with ordered children).
std::vector<int32_t> candidates(const Worker& w, int32_t pinned) {
  std::vector<int32_t> out, stack;
  stack.push_back(0);
  while (!stack.empty()) {
    int32_t x = stack.back();
    stack.pop_back();
    const Node& n = w.nodes[x];
    if (x != 0 && n.kids.empty()) {
      if (n.mark != w.phase && x != pinned && n.pin == 0) out.push_back(x);
      continue;
    }
    for (auto it = n.kids.rbegin(); it != n.kids.rend(); ++it) stack.push_back(it->second);
  }
  return out;
}

int32_t lcp(const Worker& w, const int32_t* q, int32_t L) {
  int32_t u = 0, h = 0;
  while (h < L) {
    auto it = w.nodes[u].kids.find(q[h]);
    if (it == w.nodes[u].kids.end()) break;
    u = it->second;
    h += 1;
  }
  return h;
}

// Mark token v (already in S, or about to be loaded when v < 0), Algorithm 1:
// add it to T; if |T| reaches B+1 the marking set becomes {v}.
// Returns true when a new phase started.
bool mark_token(Worker& w, uint32_t B, int32_t v) {
  bool newly = (v < 0) || (w.nodes[v].mark != w.phase);
  bool reset = false;
  if (newly) {
    w.cnt += 1;
    if (w.cnt == B + 1) {
      w.phase += 1;
      w.cnt = 1;
      reset = true;
    }
    if (v >= 0) w.nodes[v].mark = w.phase;
  }
  return reset;
}

void erase_value(std::vector<int32_t>& v, int32_t x) {
  for (size_t k = 0; k < v.size(); ++k)
    if (v[k] == x) {
      v.erase(v.begin() + (long)k);
      return;
    }
}

// RLT insertion of path q into worker i (Algorithm 1 for one path).
void insert_rlt(Sim& s, uint32_t i, const int32_t* q, int32_t L, uint64_t jg) {
  Worker& w = s.w[i];
  const uint32_t B = s.cfg.cache_tokens;
  uint64_t d = 0;  // draw index within this query
  int32_t u = 0;   // node of q[0:p)
  for (int32_t p = 0; p < L; ++p) {
    auto it = w.nodes[u].kids.find(q[p]);
    int32_t v = (it == w.nodes[u].kids.end()) ? -1 : it->second;
    bool was_leaf_cand = (v >= 0) && is_leaf(w, v) && w.nodes[v].mark != w.phase;
    if (mark_token(w, B, v)) {
      w.U_valid = false;
      w.st.phase = w.phase;
    } else if (was_leaf_cand && w.U_valid) {
      erase_value(w.U, v);  // a candidate leaf got marked
    }
    if (v >= 0) {  // hit: continue along the path
      u = v;
      continue;
    }
    if (w.size == B) {
      std::vector<int32_t> Udef;
      std::vector<int32_t>* Up;
      if (s.cfg.u_mode == 1) {
        Udef = candidates(w, u);
        Up = &Udef;
      } else {
        if (!w.U_valid) {
          w.U = candidates(w, u);
          w.U_valid = true;
        }
        Up = &w.U;
      }
      if (Up->empty()) {
        // no unmarked leaf: start a new phase with T = {t} and recompute U
        w.phase += 1;
        w.cnt = 1;
        w.st.forced_resets += 1;
        w.st.phase = w.phase;
        *Up = candidates(w, u);
        w.U_valid = (s.cfg.u_mode == 0);
        if (Up->empty()) {
          s.error |= 4;  // the path alone exceeds the cache (|q| > B)
          return;
        }
      }
      uint64_t ctr[4] = {jg, (uint64_t)i, d, 0};
      uint64_t key[2] = {s.cfg.seed, (uint64_t)s.replica};
      uint64_t r[4];
      philox4x64_10(ctr, key, r);
      d += 1;
      uint64_t k = (uint64_t)(((unsigned __int128)r[0] * (uint64_t)Up->size()) >> 64);
      int32_t victim = (*Up)[k];
      int32_t par = w.nodes[victim].parent;
      remove_leaf(w, victim);
      w.st.evictions += 1;
      if (s.cfg.u_mode == 0) {
        // the parent of the evicted leaf takes its place in the ordered list
        // if it is now an unmarked, unpinned leaf; otherwise the entry goes.
        if (par != 0 && w.nodes[par].kids.empty() && w.nodes[par].mark != w.phase && par != u &&
            w.nodes[par].pin == 0)
          w.U[k] = par;
        else
          w.U.erase(w.U.begin() + (long)k);
      }
    }
    int32_t nv = new_node(w, q[p], u);
    w.nodes[nv].mark = w.phase;  // marked before it was loaded
    w.st.loads += 1;
    u = nv;
  }
}

// L-LRU insertion (Sec. 3.2): every access stamps the token; a miss with a
// full cache evicts the leaf (other than the insertion point) with the
// oldest stamp.  Stamps (query index, position) are unique, so there are no
// ties.  u_mode 1 scans every node for that leaf; u_mode 0 keeps the leaves
// in a set ordered by stamp (the same leaf, found faster).
void lru_set_stamp(Sim& s, Worker& w, int32_t id, uint64_t stamp) {
  Node& n = w.nodes[id];
  if (s.cfg.u_mode == 0 && id != 0 && n.kids.empty()) {
    w.lru_leaves.erase({n.stamp, id});
    w.lru_leaves.insert({stamp, id});
  }
  n.stamp = stamp;
}

void insert_lru(Sim& s, Worker& w, uint32_t B, const int32_t* q, int32_t L, uint64_t jg) {
  const bool scan = s.cfg.u_mode == 1;
  int32_t u = 0;
  for (int32_t p = 0; p < L; ++p) {
    uint64_t stamp = (jg << 32) | (uint64_t)(uint32_t)p;
    auto it = w.nodes[u].kids.find(q[p]);
    if (it != w.nodes[u].kids.end()) {
      u = it->second;
      lru_set_stamp(s, w, u, stamp);
      continue;
    }
    if (w.size == B) {
      int32_t best = -1;
      if (scan) {
        for (int32_t x = 1; x < (int32_t)w.nodes.size(); ++x) {
          const Node& n = w.nodes[x];
          if (!n.alive || !n.kids.empty() || x == u || n.pin > 0) continue;
          if (best < 0 || n.stamp < w.nodes[best].stamp) best = x;
        }
      } else {
        for (auto jt = w.lru_leaves.begin(); jt != w.lru_leaves.end(); ++jt)
          if (jt->second != u && w.nodes[jt->second].pin == 0) {
            best = jt->second;
            break;
          }
      }
      if (best < 0) {
        s.error |= 4;
        return;
      }
      const int32_t par = w.nodes[best].parent;
      if (!scan) w.lru_leaves.erase({w.nodes[best].stamp, best});
      remove_leaf(w, best);
      if (!scan && par != 0 && w.nodes[par].kids.empty()) w.lru_leaves.insert({w.nodes[par].stamp, par});
      w.st.evictions += 1;
    }
    if (!scan && u != 0 && w.nodes[u].kids.empty()) w.lru_leaves.erase({w.nodes[u].stamp, u});
    int32_t nv = new_node(w, q[p], u);
    w.nodes[nv].stamp = stamp;
    if (!scan) w.lru_leaves.insert({stamp, nv});
    w.st.loads += 1;
    u = nv;
  }
}

// Residual-model update with error e = E - E_hat on features phi.
void online_update(Sim& s, Worker& w, const double phi[4], double e) {
  const orc_config& c = s.cfg;
  if (c.update == 0) {  // normalised LMS
    double ss = phi[0] * phi[0];
    ss = ss + phi[1] * phi[1];
    ss = ss + phi[2] * phi[2];
    ss = ss + phi[3] * phi[3];
    double g = (c.lr * e) / (c.nlms_eps + ss);
    for (int a = 0; a < 4; ++a) w.theta[a] = w.theta[a] + g * phi[a];
  } else if (c.update == 1) {  // recursive least squares, forgetting factor lr
    double pi[4];
    for (int a = 0; a < 4; ++a) {
      double acc = w.Pm[a * 4 + 0] * phi[0];
      acc = acc + w.Pm[a * 4 + 1] * phi[1];
      acc = acc + w.Pm[a * 4 + 2] * phi[2];
      acc = acc + w.Pm[a * 4 + 3] * phi[3];
      pi[a] = acc;
    }
    double den = phi[0] * pi[0];
    den = den + phi[1] * pi[1];
    den = den + phi[2] * pi[2];
    den = den + phi[3] * pi[3];
    den = c.lr + den;
    double k[4];
    for (int a = 0; a < 4; ++a) k[a] = pi[a] / den;
    for (int a = 0; a < 4; ++a) w.theta[a] = w.theta[a] + k[a] * e;
    for (int a = 0; a < 4; ++a)
      for (int b = 0; b < 4; ++b) w.Pm[a * 4 + b] = (w.Pm[a * 4 + b] - k[a] * pi[b]) / c.lr;
  }
}

int64_t tick(const orc_config& c, int64_t t) { return t / c.decay_interval_us; }

// Add d to the in-progress count of every token of path q (all cached).
void pin_path(Sim& s, Worker& w, const std::vector<int32_t>& q, int d) {
  int32_t u = 0;
  for (int32_t tok : q) {
    auto it = w.nodes[u].kids.find(tok);
    if (it == w.nodes[u].kids.end()) {
      s.error |= 2;  // an in-progress token was evicted
      return;
    }
    u = it->second;
    w.nodes[u].pin = (uint32_t)((int64_t)w.nodes[u].pin + d);
    // a released leaf that is not marked is a candidate again: the ordered
    // list is rebuilt from its definition at the next draw
    if (d < 0 && w.nodes[u].pin == 0 && w.nodes[u].kids.empty() && w.nodes[u].mark != w.phase)
      w.U_valid = false;
  }
}

// The path just inserted joins the running batch of worker i; the oldest
// path leaves it once beta - 1 later ones are running.
void batch_admit(Sim& s, uint32_t i, const int32_t* q, int32_t L) {
  const uint32_t beta = s.cfg.batch_size;
  if (beta <= 1) return;
  Worker& w = s.w[i];
  w.running.emplace_back(q, q + L);
  pin_path(s, w, w.running.back(), +1);
  if (w.running.size() > beta - 1) {
    pin_path(s, w, w.running.front(), -1);
    w.running.pop_front();
  }
}

// Query jg: prompt q[0, L), inserted path q[0, Lpath) (Lpath = L unless
// responses are cached), arrival t, output length o.
void step(Sim& s, uint64_t jg, const int32_t* q, int32_t L, int32_t Lpath, int64_t t, int32_t o,
          int32_t* route_out, int32_t* hit_out, int32_t* all_hits_row) {
  const orc_config& c = s.cfg;
  const uint32_t W = c.num_workers;
  // 1. completions (update thread) and decay (background thread)
  for (uint32_t i = 0; i < W; ++i) {
    Worker& w = s.w[i];
    while (!w.pend.empty() && w.pend.front().t_done <= t) {
      Pending pc = w.pend.front();
      w.pend.pop_front();
      w.P = w.P * pow_int(c.rho, (uint64_t)(tick(c, pc.t_done) - tick(c, w.tl)));
      w.tl = pc.t_done;
      double rem = pc.chat * pow_int(c.rho, (uint64_t)(tick(c, pc.t_done) - tick(c, pc.t_route)));
      double np = w.P - rem;
      w.P = np > 0.0 ? np : 0.0;
      // the squared loss (E - E_hat)^2 is minimised at the current model:
      // E_hat is re-evaluated with the current theta on the stored features
      double res = w.theta[0] * pc.phi[0];
      res = res + w.theta[1] * pc.phi[1];
      res = res + w.theta[2] * pc.phi[2];
      res = res + w.theta[3] * pc.phi[3];
      double ehat_now = pc.base + res;
      online_update(s, w, pc.phi, pc.e_obs - ehat_now);
      w.st.completions += 1;
    }
    w.P = w.P * pow_int(c.rho, (uint64_t)(tick(c, t) - tick(c, w.tl)));
    w.tl = t;
    int64_t nb = w.Wb - (t - s.tprev);
    w.Wb = nb > 0 ? nb : 0;
  }
  s.tprev = t;
  // 2. match on every worker (no state changes): the worker's cache, or the
  // router's tree of it
  const bool approx = c.router_tree != 0;
  std::vector<int32_t> h(W);
  for (uint32_t i = 0; i < W; ++i) {
    h[i] = approx ? lcp(s.rt[i], q, L) : lcp(s.w[i], q, L);
    s.w[i].st.matched_tokens += (uint64_t)h[i];
    if (all_hits_row) all_hits_row[i] = h[i];
  }
  // 3-4. LBGR score and argmin (lowest index on ties)
  std::vector<double> chat(W), ehat(W), phis(4 * W);
  uint32_t best = 0;
  for (uint32_t i = 0; i < W; ++i) {
    Worker& w = s.w[i];
    double x1 = (double)h[i] * 0.001;
    double x2 = (double)(L - h[i]) * 0.001;
    double x3 = w.P;
    double x4 = 1.0;
    double ch = c.alpha_cached * x1 + c.alpha_miss * x2;
    double res = w.theta[0] * x1;
    res = res + w.theta[1] * x2;
    res = res + w.theta[2] * x3;
    res = res + w.theta[3] * x4;
    double eh = (ch + w.P) + res;
    chat[i] = ch;
    ehat[i] = eh;
    phis[4 * i + 0] = x1;
    phis[4 * i + 1] = x2;
    phis[4 * i + 2] = x3;
    phis[4 * i + 3] = x4;
    if (i == 0 || eh < ehat[best]) best = i;
  }
  // 4'. the baseline routers of Sec. 5 replace the LBGR choice
  if (c.router == 1) {
    // random: a uniform worker from word 0 of Philox4x64-10, key
    // (seed, replica), counter (query index, 0, 0, 1)
    const uint64_t ctr[4] = {jg, 0, 0, 1}, key[2] = {c.seed, s.replica};
    uint64_t out[4];
    philox4x64_10(ctr, key, out);
    best = (uint32_t)(((unsigned __int128)out[0] * W) >> 64);
  } else if (c.router == 2) {
    // round robin over the global query index
    best = (uint32_t)(jg % W);
  } else if (c.router == 3) {
    // cache-aware: in-flight load = queries routed and not completed by t
    uint32_t lo = 0, hi = 0, hmax = 0, small = 0;
    for (uint32_t i = 1; i < W; ++i) {
      if (s.w[i].pend.size() < s.w[lo].pend.size()) lo = i;
      if (s.w[i].pend.size() > s.w[hi].pend.size()) hi = i;
      if (h[i] > h[hmax]) hmax = i;
      if (s.w[i].size < s.w[small].size) small = i;
    }
    const uint64_t lmin = s.w[lo].pend.size(), lmax = s.w[hi].pend.size();
    if (lmax - lmin > (uint64_t)c.ca_balance_abs && (double)lmax > c.ca_balance_rel * (double)lmin)
      best = lo;  // imbalanced: the least loaded
    else if ((double)h[hmax] > c.ca_cache_threshold * (double)L)
      best = hmax;  // the highest hit
    else
      best = small;  // low hits everywhere: the emptiest cache
  }
  // 5. commit: load increment, observed latency, pending completion; the
  // observed latency and the hit count take the worker's true match
  Worker& w = s.w[best];
  double base_route = chat[best] + w.P;
  w.P = w.P + chat[best];
  int64_t hb = approx ? lcp(w, q, L) : h[best];
  int64_t cost_us = c.true_cached_us * hb + c.true_miss_us * ((int64_t)L - hb) + c.true_out_us * (int64_t)o;
  int64_t e_us = w.Wb + cost_us;
  w.Wb = w.Wb + cost_us;
  Pending pc;
  pc.t_route = t;
  pc.t_done = t + e_us;
  pc.chat = chat[best];
  pc.base = base_route;
  pc.e_obs = (double)e_us * 1e-6;
  for (int a = 0; a < 4; ++a) pc.phi[a] = phis[4 * best + a];
  w.pend.push_back(pc);
  if (w.pend.size() > w.st.pending_max) w.st.pending_max = w.pend.size();
  w.st.routed += 1;
  w.st.prompt_tokens += (uint64_t)L;
  w.st.hit_tokens += (uint64_t)hb;
  w.st.latency_sum_us += (uint64_t)e_us;
  if ((uint64_t)e_us > w.st.latency_max_us) w.st.latency_max_us = (uint64_t)e_us;
  if (route_out) *route_out = (int32_t)best;
  if (hit_out) *hit_out = (int32_t)hb;
  // 6. insert the path into the routed worker's cache; it joins that
  // worker's running batch
  if (c.evict == 0)
    insert_rlt(s, best, q, Lpath, jg);
  else
    insert_lru(s, w, c.cache_tokens, q, Lpath, jg);
  if (!s.error) batch_admit(s, best, q, Lpath);
  // the router adds the prompt to its tree of the routed worker
  if (!s.error && approx)
    insert_lru(s, s.rt[best], c.router_tree_tokens ? c.router_tree_tokens : c.cache_tokens, q, L, jg);
}

// Per-token path hash H(v) = mix64(H(parent) + GOLDEN * (tok + 1)), H(root) = 0.
void digest(const Worker& w, orc_worker_stats& st) {
  st.digest_sum = st.digest_xor = st.marked_count = st.marked_sum = 0;
  std::vector<std::pair<int32_t, uint64_t>> stack;
  stack.push_back({0, 0});
  uint64_t count = 0;
  while (!stack.empty()) {
    auto [x, hx] = stack.back();
    stack.pop_back();
    for (auto& kv : w.nodes[x].kids) {
      uint64_t hv = mix64(hx + 0x9E3779B97F4A7C15ULL * (uint64_t)(int64_t)(kv.first + 1));
      st.digest_sum += hv;
      st.digest_xor ^= hv;
      count += 1;
      if (w.nodes[kv.second].mark == w.phase) {
        st.marked_count += 1;
        st.marked_sum += hv;
      }
      stack.push_back({kv.second, hv});
    }
  }
  st.resident = count;
}

bool check_invariants(const Sim& s) {
  for (const Worker& w : s.w) {
    if (w.size > s.cfg.cache_tokens) return false;  // |S_i| <= B_i (Sec. 3.1)
    if (!(w.P >= 0.0)) return false;                // the load estimate never goes negative
    uint64_t alive = 0, marked = 0;
    for (size_t x = 1; x < w.nodes.size(); ++x) {
      const Node& n = w.nodes[x];
      if (!n.alive) continue;
      alive += 1;
      if (!w.nodes[n.parent].alive && n.parent != 0) return false;  // prefix-closed
      if (n.mark == w.phase) marked += 1;
    }
    if (alive != w.size) return false;
    if (s.cfg.evict == 0 && marked != w.cnt) return false;  // T is a subset of S after an insert
    if (w.cnt > s.cfg.cache_tokens) return false;
    // the running batch is cached whole, and the in-progress counts are
    // exactly the number of running paths through each token
    std::vector<uint32_t> pins(w.nodes.size(), 0);
    for (const auto& q : w.running) {
      int32_t u = 0;
      for (int32_t tok : q) {
        auto it = w.nodes[u].kids.find(tok);
        if (it == w.nodes[u].kids.end()) return false;
        u = it->second;
        pins[u] += 1;
      }
    }
    for (size_t x = 1; x < w.nodes.size(); ++x)
      if (w.nodes[x].alive && w.nodes[x].pin != pins[x]) return false;
  }
  // the router's trees: within their budget, prefix-closed
  const uint64_t rb = s.cfg.router_tree_tokens ? s.cfg.router_tree_tokens : s.cfg.cache_tokens;
  for (const Worker& w : s.rt) {
    if (w.size > rb) return false;
    uint64_t alive = 0;
    for (size_t x = 1; x < w.nodes.size(); ++x) {
      const Node& n = w.nodes[x];
      if (!n.alive) continue;
      alive += 1;
      if (!w.nodes[n.parent].alive && n.parent != 0) return false;
    }
    if (alive != w.size) return false;
  }
  return true;
}

// Signature of everything a cache holds: its tokens, marks, marking phase
// and count, access stamps and in-progress counts.  A step may change only
// the routed worker's (Eq. 3); the check compares these before and after.
uint64_t cache_sig(const Worker& w) {
  uint64_t h = mix64(w.size + 1);
  h = mix64(h ^ w.phase);
  h = mix64(h ^ w.cnt);
  for (size_t x = 0; x < w.nodes.size(); ++x) {
    const Node& n = w.nodes[x];
    if (!n.alive) continue;
    h = mix64(h + x);
    h = mix64(h ^ (uint64_t)(uint32_t)n.tok);
    h = mix64(h ^ (uint64_t)(uint32_t)n.parent);
    h = mix64(h ^ n.mark);
    h = mix64(h ^ n.stamp);
    h = mix64(h ^ n.pin);
    h = mix64(h ^ n.kids.size());
  }
  return h;
}

// The per-worker statistics of the current state (the counters plus the
// path-hash digest of the cache and, with router_tree, of the router's tree).
void snapshot(const Sim& s, uint32_t i, orc_worker_stats& out) {
  const Worker& w = s.w[i];
  out = w.st;
  digest(w, out);
  out.phase = w.phase;
  out.cnt = w.cnt;
  out.pending_depth = w.pend.size();
  out.backlog_us = w.Wb;
  out.last_decay_us = w.tl;
  out.load_est = w.P;
  for (int a = 0; a < 4; ++a) out.theta[a] = w.theta[a];
  if (s.cfg.router_tree) {
    const Worker& rw = s.rt[i];
    orc_worker_stats rs;
    std::memset(&rs, 0, sizeof(rs));
    digest(rw, rs);
    out.router_resident = rs.resident;
    out.router_digest_sum = rs.digest_sum;
    out.router_digest_xor = rs.digest_xor;
    out.router_evictions = rw.st.evictions;
  }
}

double thread_cpu_seconds() {
  timespec ts;
  clock_gettime(CLOCK_THREAD_CPUTIME_ID, &ts);
  return (double)ts.tv_sec + 1e-9 * (double)ts.tv_nsec;
}

double wall_seconds() {
  timespec ts;
  clock_gettime(CLOCK_MONOTONIC, &ts);
  return (double)ts.tv_sec + 1e-9 * (double)ts.tv_nsec;
}

}  // namespace

extern "C" {

// Run replica `replica` over queries [0, n) of the stream from the initial
// state (empty caches, zero loads, phase 1; Sec. 3.1, Table 1).  Outputs:
// route[j], hits[j] and, if all_hits != NULL, all_hits[j*W + i].  wstats[W]
// receives the final per-worker state.  opts (optional) asks for snapshots of
// the per-worker state every snap_every queries (snapshot k, after query
// (k+1)*snap_every - 1 or the last one, in snaps[k*W + i]) and times the
// queries from time_from on (thread CPU and wall seconds), stopping once
// they have taken time_budget_s of CPU time when that is positive.
// Returns 0, or a bit set: 1 = bad argument, 2 = invariant violated (with
// check = 1), 4 = a path longer than the cache.
int orc_run_ex(const orc_config* cfg, uint32_t replica, uint64_t n, const int32_t* tokens,
               const uint64_t* offsets, const int64_t* arrival_us, const uint16_t* out_len,
               int32_t* route, int32_t* hits, int32_t* all_hits, orc_worker_stats* wstats,
               orc_run_opts* opts) {
  if (!cfg || cfg->num_workers == 0 || cfg->cache_tokens == 0 || cfg->decay_interval_us <= 0) return 1;
  const uint32_t W = cfg->num_workers;
  Sim s;
  s.cfg = *cfg;
  s.replica = replica;
  s.w.resize(W);
  s.rt.resize(cfg->router_tree ? W : 0);
  for (Worker& w : s.w) {
    w.nodes.emplace_back();
    w.nodes[0].alive = true;
    std::memset(&w.st, 0, sizeof(w.st));
    w.st.phase = 1;
    for (int a = 0; a < 16; ++a) w.Pm[a] = (a % 5 == 0) ? cfg->rls_p0 : 0.0;
  }
  for (Worker& w : s.rt) {
    w.nodes.emplace_back();
    w.nodes[0].alive = true;
    std::memset(&w.st, 0, sizeof(w.st));
  }
  const uint64_t snap_every = opts ? opts->snap_every : 0;
  const uint64_t time_from = opts ? opts->time_from : n;
  double cpu0 = 0.0, wall0 = 0.0;
  std::vector<uint64_t> sig_w, sig_rt;
  uint64_t j = 0;
  for (; j < n; ++j) {
    if (j == time_from) {
      cpu0 = thread_cpu_seconds();
      wall0 = wall_seconds();
    } else if (j > time_from && opts && opts->time_budget_s > 0.0 &&
               thread_cpu_seconds() - cpu0 >= opts->time_budget_s) {
      break;
    }
    const int32_t* q = tokens + offsets[j];
    const int32_t Lpath = (int32_t)(offsets[j + 1] - offsets[j]);
    int32_t o = out_len ? (int32_t)out_len[j] : 4;
    const int32_t L = cfg->cache_responses ? Lpath - o : Lpath;  // the prompt
    if (L < 1) {
      s.error |= 1;
      break;
    }
    if (cfg->check) {
      sig_w.resize(W);
      sig_rt.resize(s.rt.size());
      for (uint32_t i = 0; i < W; ++i) sig_w[i] = cache_sig(s.w[i]);
      for (size_t i = 0; i < s.rt.size(); ++i) sig_rt[i] = cache_sig(s.rt[i]);
    }
    int32_t routed = -1;
    step(s, j, q, L, Lpath, arrival_us[j], o, &routed, hits ? hits + j : nullptr,
         all_hits ? all_hits + j * W : nullptr);
    if (route) route[j] = routed;
    if (s.error) break;
    if (cfg->check) {
      if (!check_invariants(s)) s.error |= 2;
      // Eq. 3: no cache but the routed worker's changed (nor its router tree)
      for (uint32_t i = 0; i < W; ++i)
        if ((int32_t)i != routed && cache_sig(s.w[i]) != sig_w[i]) s.error |= 2;
      for (size_t i = 0; i < s.rt.size(); ++i)
        if ((int32_t)i != routed && cache_sig(s.rt[i]) != sig_rt[i]) s.error |= 2;
      if (s.error) {
        ++j;
        break;
      }
    }
    if (snap_every && opts->snaps && ((j + 1) % snap_every == 0 || j + 1 == n)) {
      const uint64_t k = j / snap_every;
      for (uint32_t i = 0; i < W; ++i) snapshot(s, i, opts->snaps[k * W + i]);
    }
  }
  if (opts) {
    opts->done = j;
    if (j > time_from) {
      opts->window_cpu_s = thread_cpu_seconds() - cpu0;
      opts->window_wall_s = wall_seconds() - wall0;
    } else {
      opts->window_cpu_s = opts->window_wall_s = 0.0;
    }
  }
  if (wstats)
    for (uint32_t i = 0; i < W; ++i) snapshot(s, i, wstats[i]);
  return s.error;
}

int orc_run(const orc_config* cfg, uint32_t replica, uint64_t n, const int32_t* tokens,
            const uint64_t* offsets, const int64_t* arrival_us, const uint16_t* out_len,
            int32_t* route, int32_t* hits, int32_t* all_hits, orc_worker_stats* wstats) {
  return orc_run_ex(cfg, replica, n, tokens, offsets, arrival_us, out_len, route, hits, all_hits, wstats,
                    nullptr);
}

// Self-test of the invariant checks: build a two-worker state, plant one
// violation (1 = a negative load estimate on a worker, 2 = a changed mark on
// a worker the step did not route to, 3 = a token whose parent is gone) and
// return 1 when the checks report it, 0 when they miss it.
int orc_check_selftest(int which) {
  Sim s;
  s.replica = 0;
  std::memset(&s.cfg, 0, sizeof(s.cfg));
  s.cfg.num_workers = 2;
  s.cfg.cache_tokens = 64;
  s.cfg.decay_interval_us = 20000;
  s.cfg.rho = 1.0;
  s.cfg.lr = 0.992;
  s.cfg.alpha_miss = 1.0;
  s.cfg.true_miss_us = 1000;
  s.cfg.batch_size = 1;
  s.w.resize(2);
  for (Worker& w : s.w) {
    w.nodes.emplace_back();
    w.nodes[0].alive = true;
    std::memset(&w.st, 0, sizeof(w.st));
  }
  const int32_t qa[4] = {1, 2, 3, 4}, qb[3] = {7, 8, 9};
  int32_t r0 = -1, r1 = -1;
  step(s, 0, qa, 4, 4, 0, 4, &r0, nullptr, nullptr);
  step(s, 1, qb, 3, 3, 1000, 4, &r1, nullptr, nullptr);
  if (!check_invariants(s)) return 0;  // the clean state must pass
  const uint64_t sig1 = cache_sig(s.w[1]);
  if (which == 1) {
    s.w[1].P = -1e-3;
    return check_invariants(s) ? 0 : 1;
  }
  if (which == 2) {
    // worker 1 holds qb (routed away from the loaded worker 0); re-mark one
    // of its tokens as if a step routed to worker 0 had touched it
    for (size_t x = 1; x < s.w[1].nodes.size(); ++x)
      if (s.w[1].nodes[x].alive) {
        s.w[1].nodes[x].mark += 1;
        break;
      }
    return cache_sig(s.w[1]) != sig1 ? 1 : 0;
  }
  if (which == 3) {
    Worker& w = s.w[r1];
    for (size_t x = 1; x < w.nodes.size(); ++x)
      if (w.nodes[x].alive && w.nodes[x].parent == 0) {
        w.nodes[x].alive = false;  // an internal token gone: its child dangles
        w.size -= 1;
        break;
      }
    return check_invariants(s) ? 0 : 1;
  }
  return 0;
}

// Philox4x64-10 block for (counter, key); exported for the known-answer test.
void orc_philox4x64_10(const uint64_t* ctr, const uint64_t* key, uint64_t* out) {
  philox4x64_10(ctr, key, out);
}

double orc_pow_int(double rho, uint64_t k) { return pow_int(rho, k); }

}  // extern "C"
