// kvr_core.h - per-wave logic of the simulator (included by kvr_device.hip).
//
// Every function here is executed by one whole wavefront with wave-uniform
// control flow; lane-parallel loops step by KVR_WAVE lanes (64 on gfx950).
// Writes of shared scalars are done by lane 0.
#ifndef KVR_CORE_H
#define KVR_CORE_H

#include <stdint.h>

#include "kvr_layout.h"

#ifndef KVR_WAVE
#define KVR_WAVE 64
#endif

namespace kvr {


// ---------------------------------------------------------------- wave tools

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (KVR_WAVE - 1u)); }

__device__ __forceinline__ uint64_t lanemask_lt() {
  return (1ull << (uint32_t)lane_id()) - 1ull;
}

__device__ __forceinline__ uint64_t lanemask_le() {
  return (2ull << (uint32_t)lane_id()) - 1ull;
}

#ifndef KVR_SYNC_SCOPE
#define KVR_SYNC_SCOPE "workgroup"
#endif
// Global stores of one lane are read back by the other lanes of the same
// wave (the tree, leaf and candidate arrays are shared by the whole wave):
// complete them before any later load.
__device__ __forceinline__ void wave_mem_sync() { __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, KVR_SYNC_SCOPE); }

__device__ __forceinline__ int first_lane(uint64_t m) { return __ffsll((unsigned long long)m) - 1; }

// Wave reductions with DPP lane moves (no LDS round trip): shifts by 1, 2,
// 4 and 8 lanes within each row of 16 leave the row's result in its lane 15,
// then the broadcasts of lanes 15 and 31 to the following rows leave the
// wave's result in lane 63, which is returned to every lane.  A lane whose
// DPP source lies outside its row keeps its own value.  Call with the whole
// wave active.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, kCtrl, kRowMask, 0xf, false);
}

template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
  const uint32_t lo = dpp_u32<kCtrl, kRowMask>((uint32_t)v);
  const uint32_t hi = dpp_u32<kCtrl, kRowMask>((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}

template <bool kMax>
__device__ __forceinline__ uint64_t wave_reduce_u64(uint64_t v) {
#define KVR_RED_STEP(ctrl, rows)                  \
  {                                               \
    const uint64_t w = dpp_u64<ctrl, rows>(v);    \
    v = kMax ? (w > v ? w : v) : (w < v ? w : v); \
  }
  KVR_RED_STEP(0x111, 0xf)  // row_shr:1
  KVR_RED_STEP(0x112, 0xf)  // row_shr:2
  KVR_RED_STEP(0x114, 0xf)  // row_shr:4
  KVR_RED_STEP(0x118, 0xf)  // row_shr:8
  KVR_RED_STEP(0x142, 0xa)  // row_bcast:15 into rows 1 and 3
  KVR_RED_STEP(0x143, 0xc)  // row_bcast:31 into rows 2 and 3
#undef KVR_RED_STEP
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, KVR_WAVE - 1);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), KVR_WAVE - 1);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) { return wave_reduce_u64<false>(v); }

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) { return wave_reduce_u64<true>(v); }

// ---------------------------------------------------------------- phase timers
// Per-part timing of a step (phase_timers): ticks of the 100 MHz real-time
// counter, accumulated in registers by the routing wave.  A no-op unless kOn.
struct PhaseClock {
  uint64_t t;
  uint64_t acc[KVR_PHASES];
};

template <bool kOn>
__device__ __forceinline__ void clock_start(PhaseClock* c) {
  if constexpr (kOn) {
    c->t = (uint64_t)wall_clock64();
    for (int k = 0; k < KVR_PHASES; ++k) c->acc[k] = 0;
  }
}

template <bool kOn>
__device__ __forceinline__ void clock_mark(PhaseClock* c, int part) {
  if constexpr (kOn) {
    const uint64_t now = (uint64_t)wall_clock64();
    c->acc[part] += now - c->t;
    c->t = now;
  }
}

// ---------------------------------------------------------------- Philox4x64-10
// Salmon et al., SC'11: ten rounds, two 64x64->128 products per round, key
// bumped by the Weyl increments between rounds.  Only word 0 is used.
__device__ __forceinline__ uint64_t philox_word0(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                                 uint64_t k0, uint64_t k1) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
#pragma unroll
  for (int rnd = 0; rnd < 10; ++rnd) {
    if (rnd) {
      k0 += 0x9E3779B97F4A7C15ull;
      k1 += 0xBB67AE8584CAA73Bull;
    }
    uint64_t lo0 = M0 * c0, hi0 = __umul64hi(M0, c0);
    uint64_t lo1 = M1 * c2, hi1 = __umul64hi(M1, c2);
    uint64_t n0 = hi1 ^ c1 ^ k0;
    uint64_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return c0;
}

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// One link of a replica's route digest: D' = mix64(mix64(D + G*(j+1)) +
// ((route << 32) | hit)), so the chain over the queries in order changes
// with any routing decision or routed hit.
__device__ __forceinline__ uint64_t route_chain(uint64_t d, uint64_t jg, uint32_t route, int32_t hit) {
  d = mix64(d + 0x9E3779B97F4A7C15ull * (jg + 1ull));
  return mix64(d + (((uint64_t)route << 32) | (uint64_t)(uint32_t)hit));
}

// rho^k, square-and-multiply from the least significant bit
__device__ double pow_int(double rho, uint64_t k) {
  double res = 1.0, b = rho;
  while (k) {
    if (k & 1) res = res * b;
    b = b * b;
    k >>= 1;
  }
  return res;
}

// ---------------------------------------------------------------- worker view

struct Ptrs {
  WorkerHdr* hdr;
  NodeRec* nodes;
  int32_t* arena0;  // semispace 0; semispace 1 follows at arena0 + A
  int32_t* leaf;
  int32_t* U;
  PendRec* pend;
  uint64_t* scratch;
  int32_t* stamp0;  // L-LRU: last access of each arena word (semispace 1 at + A); null for RLT
  int32_t* pin;     // continuous batching: running paths through each node; null otherwise
  int32_t* run;     // continuous batching: end nodes of the running batch (ring of beta - 1)
  uint32_t A, NC, PC, beta;
};

__device__ __forceinline__ Ptrs worker_ptrs(char* ws, const Layout& L, uint32_t r, uint32_t i) {
  const uint64_t w = (uint64_t)r * L.W + i;
  Ptrs P;
  P.hdr = reinterpret_cast<WorkerHdr*>(ws + L.off_whdr) + w;
  P.nodes = reinterpret_cast<NodeRec*>(ws + L.off_nodes + w * L.node_stride);
  P.arena0 = reinterpret_cast<int32_t*>(ws + L.off_arena + w * L.arena_stride);
  P.leaf = reinterpret_cast<int32_t*>(ws + L.off_leaf + w * L.leaf_stride);
  P.U = reinterpret_cast<int32_t*>(ws + L.off_U + w * L.leaf_stride);
  P.pend = reinterpret_cast<PendRec*>(ws + L.off_pend + w * L.pend_stride);
  P.scratch = reinterpret_cast<uint64_t*>(ws + L.off_scratch + w * L.scratch_stride);
  P.stamp0 = L.has_stamp ? reinterpret_cast<int32_t*>(ws + L.off_stamp + w * L.arena_stride) : nullptr;
  P.pin = L.beta > 1 ? reinterpret_cast<int32_t*>(ws + L.off_pin + w * L.pin_stride) : nullptr;
  P.run = L.beta > 1 ? reinterpret_cast<int32_t*>(ws + L.off_run + w * L.run_stride) : nullptr;
  P.A = L.A;
  P.NC = L.NC;
  P.PC = L.PC;
  P.beta = L.beta;
  return P;
}

// The router's tree of worker i (approximate router): an L-LRU token tree
// laid out like a cache, with its own header, budget and regions.  It has
// no candidate list, completion ring or running batch; the digest walk
// borrows the worker's scratch.
__device__ __forceinline__ Ptrs router_ptrs(char* ws, const Layout& L, uint32_t r, uint32_t i) {
  const uint64_t w = (uint64_t)r * L.W + i;
  Ptrs P;
  P.hdr = reinterpret_cast<WorkerHdr*>(ws + L.off_rt_hdr) + w;
  P.nodes = reinterpret_cast<NodeRec*>(ws + L.off_rt_nodes + w * L.rt_node_stride);
  P.arena0 = reinterpret_cast<int32_t*>(ws + L.off_rt_arena + w * L.rt_arena_stride);
  P.leaf = reinterpret_cast<int32_t*>(ws + L.off_rt_leaf + w * L.rt_leaf_stride);
  P.U = nullptr;
  P.pend = nullptr;
  P.scratch = reinterpret_cast<uint64_t*>(ws + L.off_scratch + w * L.scratch_stride);
  P.stamp0 = reinterpret_cast<int32_t*>(ws + L.off_rt_stamp + w * L.rt_arena_stride);
  P.pin = nullptr;
  P.run = nullptr;
  P.A = L.Ar;
  P.NC = L.NCr;
  P.PC = 0;
  P.beta = 1;
  return P;
}

// Is node x on a path of the worker's running batch (continuous batching)?
// Such a node is never evicted, and is no candidate while it is a leaf.
__device__ __forceinline__ bool pinned(const Ptrs& P, int32_t x) { return P.pin != nullptr && P.pin[x] > 0; }

// Wave-uniform copy of the cache part of a worker header.
struct St {
  uint32_t phase, cnt, size, hwm;
  int32_t free_head;
  uint32_t nleaves, nU, U_valid;
  int32_t rnode, rlo, rhi;
  uint32_t rphase;
  uint32_t arena_sel, arena_top, nnodes;
  uint32_t err;
  // first failing internal check (diagnostics only)
  int32_t dbg_check;
  int64_t dbg_val[3];
};

#define KVR_FAIL_CHECK(s, id, a, b, c) \
  do {                                 \
    (s).err |= KVR_DEV_INTERNAL;       \
    if ((s).dbg_check == 0) {          \
      (s).dbg_check = (id);            \
      (s).dbg_val[0] = (int64_t)(a);   \
      (s).dbg_val[1] = (int64_t)(b);   \
      (s).dbg_val[2] = (int64_t)(c);   \
    }                                  \
  } while (0)

__device__ __forceinline__ St load_st(const WorkerHdr* h) {
  St s;
  s.phase = h->phase;
  s.cnt = h->cnt;
  s.size = h->size;
  s.hwm = h->hwm;
  s.free_head = h->free_head;
  s.nleaves = h->nleaves;
  s.nU = h->nU;
  s.U_valid = h->U_valid;
  s.rnode = h->rnode;
  s.rlo = h->rlo;
  s.rhi = h->rhi;
  s.rphase = h->rphase;
  s.arena_sel = h->arena_sel;
  s.arena_top = h->arena_top;
  s.nnodes = h->nnodes;
  s.err = 0;
  s.dbg_check = 0;
  s.dbg_val[0] = s.dbg_val[1] = s.dbg_val[2] = 0;
  return s;
}

__device__ __forceinline__ void store_st(WorkerHdr* h, const St& s) {
  if (lane_id() != 0) return;
  h->phase = s.phase;
  h->cnt = s.cnt;
  h->size = s.size;
  h->hwm = s.hwm;
  h->free_head = s.free_head;
  h->nleaves = s.nleaves;
  h->nU = s.nU;
  h->U_valid = s.U_valid;
  h->rnode = s.rnode;
  h->rlo = s.rlo;
  h->rhi = s.rhi;
  h->rphase = s.rphase;
  h->arena_sel = s.arena_sel;
  h->arena_top = s.arena_top;
  h->nnodes = s.nnodes;
}

// Add v to one of a worker's 64-bit event counters (loads, evictions,
// forced resets, collections), which are kept out of St so that they do not
// occupy registers through an insertion.  Lane 0; the result is not used,
// so nothing waits for it.
__device__ __forceinline__ void hdr_count(uint64_t* c, uint64_t v) {
  if (lane_id() == 0) __hip_atomic_fetch_add(c, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ int32_t* arena_of(const Ptrs& P, uint32_t sel) {
  return P.arena0 + (size_t)sel * P.A;
}

__device__ __forceinline__ void node_put(const Ptrs& P, int32_t id, const NodeRec& n) {
  if (lane_id() == 0) P.nodes[id] = n;
  wave_mem_sync();
}

// Is edge position `pos` of node `id` in the marking set of the current phase?
__device__ __forceinline__ bool is_marked(const St& s, const NodeRec& nd, int32_t id, int32_t pos) {
  if (nd.mphase == s.phase && pos < nd.ma) return true;
  if (s.rphase == s.phase && s.rnode == id && pos >= s.rlo && pos < s.rhi) return true;
  return false;
}

// First edge position from which the tail of a leaf is unmarked: every
// position >= mark_top is evictable (the marked positions form [0, ma) and,
// on one node per phase, [rlo, rhi)).
__device__ __forceinline__ int32_t mark_top(const St& s, const NodeRec& nd, int32_t id) {
  int32_t top = (nd.mphase == s.phase) ? nd.ma : 0;
  if (s.rphase == s.phase && s.rnode == id && s.rhi > top) top = s.rhi;
  return top;
}

// ---------------------------------------------------------------- array tools (wave)

__device__ int32_t arr_find(const int32_t* a, uint32_t n, int32_t v) {
  constexpr int kUnroll = 8;  // eight chunks per round trip
  for (uint32_t b = 0; b < n; b += kUnroll * KVR_WAVE) {
    int32_t x[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t k = b + (uint32_t)(u * KVR_WAVE) + (uint32_t)lane_id();
      x[u] = k < n ? a[k] : 0;
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t k = b + (uint32_t)(u * KVR_WAVE) + (uint32_t)lane_id();
      const uint64_t m = __ballot(k < n && x[u] == v);
      if (m) return (int32_t)(b + (uint32_t)(u * KVR_WAVE) + (uint32_t)first_lane(m));
    }
  }
  return -1;
}

// a[pos+1 .. n+1) = a[pos .. n); a[pos] = v.  Top-down rounds of eight
// chunks: every load of a round completes before its stores are issued (a
// round's stores and the next round's loads touch disjoint words).  With
// fence = false the stores are left outstanding: the caller fences before
// anything reads the array.
__device__ void arr_insert(int32_t* a, uint32_t n, uint32_t pos, int32_t v, bool fence = true) {
  constexpr int kUnroll = 8;
  constexpr int64_t kSpan = (int64_t)kUnroll * KVR_WAVE;
  for (int64_t hi = (int64_t)n; hi > (int64_t)pos; hi -= kSpan) {
    const int64_t lo = hi - kSpan > (int64_t)pos ? hi - kSpan : (int64_t)pos;
    int32_t x[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t k = lo + u * KVR_WAVE + lane_id();
      x[u] = k < hi ? a[k] : 0;
    }
    wave_mem_sync();
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t k = lo + u * KVR_WAVE + lane_id();
      if (k < hi) a[k + 1] = x[u];
    }
    if (fence) wave_mem_sync();
  }
  if (lane_id() == 0) a[pos] = v;
  if (fence) wave_mem_sync();
}

// a[pos .. n-1) = a[pos+1 .. n), bottom-up rounds of eight chunks
__device__ void arr_erase(int32_t* a, uint32_t n, uint32_t pos) {
  constexpr int kUnroll = 8;
  constexpr uint32_t kSpan = (uint32_t)kUnroll * KVR_WAVE;
  for (uint32_t lo = pos; lo + 1 < n; lo += kSpan) {
    int32_t x[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t k = lo + (uint32_t)(u * KVR_WAVE) + (uint32_t)lane_id();
      x[u] = k + 1 < n ? a[k + 1] : 0;
    }
    wave_mem_sync();
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t k = lo + (uint32_t)(u * KVR_WAVE) + (uint32_t)lane_id();
      if (k + 1 < n) a[k] = x[u];
    }
    wave_mem_sync();
  }
}

// ---------------------------------------------------------------- child arrays

// Child of a node whose edge starts with `tok`, or -1.  (One chunk of 64
// entries per round trip: most child arrays are short, and measured faster
// than several chunks in flight.)
__device__ int32_t child_find(const int32_t* ar, const NodeRec& nd, int32_t tok) {
  if (nd.nchild > KVR_WAVE) {
    // a wide node (the root of many prefix groups): four chunks per round trip
    constexpr int kC = 4;
    for (int32_t b = 0; b < nd.nchild; b += kC * KVR_WAVE) {
      int2 e[kC];
#pragma unroll
      for (int u = 0; u < kC; ++u) {
        const int32_t k = b + u * KVR_WAVE + lane_id();
        e[u].x = e[u].y = -1;
        if (k < nd.nchild) e[u] = *reinterpret_cast<const int2*>(ar + nd.coff + 2 * k);
      }
#pragma unroll
      for (int u = 0; u < kC; ++u) {
        const int32_t k = b + u * KVR_WAVE + lane_id();
        const uint64_t m = __ballot(k < nd.nchild && e[u].x == tok);
        if (m) return __builtin_amdgcn_readlane(e[u].y, first_lane(m));
      }
    }
    return -1;
  }
  for (int32_t b = 0; b < nd.nchild; b += KVR_WAVE) {
    int32_t k = b + lane_id();
    bool hit = false;
    int32_t id = -1;
    if (k < nd.nchild) {
      int2 e = *reinterpret_cast<const int2*>(ar + nd.coff + 2 * k);
      hit = (e.x == tok);
      id = e.y;
    }
    uint64_t m = __ballot(hit);
    if (m) return __builtin_amdgcn_readlane(id, first_lane(m));
  }
  return -1;
}

// Child with the largest first token < tok (below) or the smallest > tok.
__device__ int32_t child_neighbor(const int32_t* ar, const NodeRec& nd, int64_t tok, bool below) {
  uint64_t best = below ? 0ull : ~0ull;
  for (int32_t b = 0; b < nd.nchild; b += KVR_WAVE) {
    int32_t k = b + lane_id();
    if (k < nd.nchild) {
      int2 e = *reinterpret_cast<const int2*>(ar + nd.coff + 2 * k);
      uint64_t key = ((uint64_t)(uint32_t)e.x << 32) | (uint32_t)e.y;
      if (below && (int64_t)e.x < tok && key > best) best = key;
      if (!below && (int64_t)e.x > tok && key < best) best = key;
    }
  }
  best = below ? wave_max_u64(best) : wave_min_u64(best);
  if (below ? best == 0ull : best == ~0ull) return -1;
  return (int32_t)(uint32_t)(best & 0xffffffffull);
}

// First (last=false) or last leaf of the subtree of x in lexicographic order
// (-1 on an inconsistency).
__device__ int32_t extreme_leaf(const Ptrs& P, const int32_t* ar, int32_t x, bool last, uint32_t hwm) {
  for (uint32_t steps = 0; steps < hwm; ++steps) {
    if (x <= 0 || (uint32_t)x >= hwm) return -1;
    NodeRec nx = P.nodes[x];
    if (nx.nchild == 0) return x;
    x = last ? child_neighbor(ar, nx, (int64_t)1 << 32, true) : child_neighbor(ar, nx, -1, false);
  }
  return -1;
}

// Index of the first (after=false) or one past the last (after=true) leaf of
// the subtree of x in the leaf list, or -1.
__device__ __forceinline__ int32_t leaf_rank(const Ptrs& P, const St& s, const int32_t* ar, int32_t x, bool after) {
  int32_t lf = extreme_leaf(P, ar, x, after, s.hwm);
  if (lf < 0) return -1;
  int32_t pos = arr_find(P.leaf, s.nleaves, lf);
  if (pos < 0) return -1;
  return after ? pos + 1 : pos;
}

// Rank in the leaf list (lexicographic order) of the leaf that the insertion
// of a path creates, on the tree as it is before that insertion: the path's
// cached part ends in node `last` (0: the root) after `lastcov` of its
// `lastlen` edge tokens, and tok is the path's first token not cached.  A
// match ending inside the edge of last will split it there, and the new leaf
// goes before or after every leaf below last; ending at a leaf, the new leaf
// takes its place; else it goes next to its neighbours among last's
// children.  -1 on an inconsistency.
__device__ int32_t new_leaf_rank(const Ptrs& P, const St& s, const int32_t* ar, int32_t last, int32_t lastcov,
                                 int32_t lastlen, int32_t tok) {
  if (last != 0 && lastcov < lastlen) {
    const int32_t tail_tok = ar[P.nodes[last].off + (uint32_t)lastcov];
    return leaf_rank(P, s, ar, last, !(tok < tail_tok));
  }
  const NodeRec na = P.nodes[last];
  if (last != 0 && na.nchild == 0) return arr_find(P.leaf, s.nleaves, last);
  if (na.nchild == 0) return 0;  // the empty tree
  const int32_t cb = child_neighbor(ar, na, tok, true);
  if (cb >= 0) return leaf_rank(P, s, ar, cb, true);
  const int32_t ca = child_neighbor(ar, na, tok, false);
  return leaf_rank(P, s, ar, ca, false);
}

// ---------------------------------------------------------------- allocation

// Wave-cooperative copy of n words (eight loads in flight per lane).
__device__ __forceinline__ void wave_copy(int32_t* dst, const int32_t* src, int32_t n) {
  constexpr int kU = 8;
  for (int32_t b = 0; b < n; b += kU * KVR_WAVE) {
    int32_t v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int32_t k = b + u * KVR_WAVE + lane_id();
      v[u] = k < n ? src[k] : 0;
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int32_t k = b + u * KVR_WAVE + lane_id();
      if (k < n) dst[k] = v[u];
    }
  }
}

// Inclusive prefix sum over the wave's lanes.
__device__ __forceinline__ uint32_t wave_inclusive_sum(uint32_t v) {
  for (int o = 1; o < KVR_WAVE; o <<= 1) {
    const uint32_t w = (uint32_t)__shfl_up((int)v, o, KVR_WAVE);
    if (lane_id() >= o) v += w;
  }
  return v;
}

// Copying collector: move every live edge and child array of the active
// semispace to the other one, compacted, and switch semispaces.  Node slots
// are taken 64 at a time: one lane reads each node, a prefix sum gives the
// new offsets (edge padded to an even length, then the child array), and
// the wave copies the blocks.  False (and nothing switched) when the live
// data does not fit a semispace.
// Out of line (it runs rarely) and with scalar arguments only, so the
// caller's cache state never has to live in memory.  Returns the new arena
// top, or ~0 when the live data does not fit.
__device__ __noinline__ uint64_t collect_arena(NodeRec* nodes, const int32_t* src, int32_t* dst, uint32_t hwm,
                                               uint32_t A, const int32_t* ssrc, int32_t* sdst) {
  wave_mem_sync();  // the caller's stores (e.g. a new edge) before they are copied
  uint64_t top = 0;
  // sizes first: the live data must fit
  for (uint32_t b = 0; b < hwm; b += KVR_WAVE) {
    const uint32_t x = b + (uint32_t)lane_id();
    uint32_t sz = 0;
    if (x < hwm) {
      const NodeRec nd = nodes[x];
      if (nd.parent != -2) sz = (((uint32_t)nd.len + 1u) & ~1u) + 2u * (uint32_t)nd.ccap;
    }
    top += (uint32_t)__builtin_amdgcn_readlane((int)wave_inclusive_sum(sz), KVR_WAVE - 1);
  }
  if (top > A) return ~0ull;
  top = 0;
  for (uint32_t b = 0; b < hwm; b += KVR_WAVE) {
    const uint32_t x = b + (uint32_t)lane_id();
    NodeRec nd;
    nd.parent = -2;
    nd.len = 0;
    nd.ccap = 0;
    nd.nchild = 0;
    nd.off = 0;
    nd.coff = 0;
    if (x < hwm) nd = nodes[x];
    const bool live = x < hwm && nd.parent != -2;
    const uint32_t elen = live ? (((uint32_t)nd.len + 1u) & ~1u) : 0u;
    const uint32_t sz = live ? elen + 2u * (uint32_t)nd.ccap : 0u;
    const uint32_t incl = wave_inclusive_sum(sz);
    const uint32_t noff = (uint32_t)top + incl - sz;
    const uint32_t ncoff = noff + elen;
    uint64_t todo = __ballot(live);
    while (todo) {
      const int j = first_lane(todo);
      todo &= todo - 1;
      const uint32_t so = (uint32_t)__builtin_amdgcn_readlane((int)nd.off, j);
      const int32_t sl = __builtin_amdgcn_readlane(nd.len, j);
      const uint32_t sc = (uint32_t)__builtin_amdgcn_readlane((int)nd.coff, j);
      const int32_t snc = __builtin_amdgcn_readlane(nd.nchild, j);
      const uint32_t dO = (uint32_t)__builtin_amdgcn_readlane((int)noff, j);
      const uint32_t dC = (uint32_t)__builtin_amdgcn_readlane((int)ncoff, j);
      wave_copy(dst + dO, src + so, sl);
      if (ssrc) wave_copy(sdst + dO, ssrc + so, sl);
      if (snc > 0) wave_copy(dst + dC, src + sc, 2 * snc);
    }
    if (live) {
      nodes[x].off = noff;
      nodes[x].coff = nd.ccap > 0 ? ncoff : 0u;
    }
    top += (uint32_t)__builtin_amdgcn_readlane((int)incl, KVR_WAVE - 1);
  }
  wave_mem_sync();
  return top;
}

__device__ __forceinline__ bool collect(const Ptrs& P, St& s) {
  const uint64_t top =
      collect_arena(P.nodes, arena_of(P, s.arena_sel), arena_of(P, s.arena_sel ^ 1u), s.hwm, P.A,
                    P.stamp0 ? P.stamp0 + (size_t)s.arena_sel * P.A : nullptr,
                    P.stamp0 ? P.stamp0 + (size_t)(s.arena_sel ^ 1u) * P.A : nullptr);
  if (top == ~0ull) return false;
  s.arena_sel ^= 1u;
  s.arena_top = (uint32_t)top;
  hdr_count(&P.hdr->gc_runs, 1u);
  return true;
}

__device__ __forceinline__ bool arena_alloc(const Ptrs& P, St& s, uint32_t words, bool even, uint32_t& off) {
  uint64_t top = s.arena_top;
  if (even) top = (top + 1u) & ~1ull;
  if (top + words > P.A) {
    if (!collect(P, s)) {
      s.err |= KVR_DEV_ARENA_FULL;
      return false;
    }
    top = s.arena_top;
    if (even) top = (top + 1u) & ~1ull;
    if (top + words > P.A) {
      s.err |= KVR_DEV_ARENA_FULL;
      return false;
    }
  }
  off = (uint32_t)top;
  s.arena_top = (uint32_t)(top + words);
  return true;
}

__device__ __forceinline__ int32_t node_alloc(const Ptrs& P, St& s) {
  int32_t id;
  if (s.free_head >= 0) {
    id = s.free_head;
    s.free_head = (int32_t)P.nodes[id].off;
  } else if (s.hwm < P.NC) {
    id = (int32_t)s.hwm;
    s.hwm += 1;
  } else {
    s.err |= KVR_DEV_NODES_FULL;
    return -1;
  }
  s.nnodes += 1;
  return id;
}

// No fence: a freed record is read again only by a later allocation, after
// the fences that end this insertion.
__device__ __forceinline__ void node_free(const Ptrs& P, St& s, int32_t id) {
  if (lane_id() == 0) {
    P.nodes[id].parent = -2;
    P.nodes[id].off = (uint32_t)s.free_head;
  }
  s.free_head = id;
  s.nnodes -= 1;
}

// Add child c (first token tok) to node a.  When the caller has read a's
// child count, capacity and array offset (in semispace sel_read), they are
// used unless a collection has switched semispaces since.  With fence =
// false the final stores are left outstanding (the caller fences before
// anything reads them).
__device__ __forceinline__ bool child_add(const Ptrs& P, St& s, int32_t a, int32_t tok, int32_t c,
                                          const int32_t* known = nullptr, uint32_t sel_read = 0,
                                          bool fence = true) {
  NodeRec na;
  if (known != nullptr && s.arena_sel == sel_read) {
    na.nchild = known[0];
    na.ccap = known[1];
    na.coff = (uint32_t)known[2];
  } else {
    na = P.nodes[a];
  }
  if (na.nchild == na.ccap) {
    int32_t ncap = na.ccap ? 2 * na.ccap : 2;
    uint32_t off;
    if (!arena_alloc(P, s, 2u * (uint32_t)ncap, true, off)) return false;
    wave_mem_sync();
    na = P.nodes[a];  // the collector may have moved the old array
    int32_t* ar = arena_of(P, s.arena_sel);
    for (int32_t k = lane_id(); k < 2 * na.nchild; k += KVR_WAVE) ar[off + k] = ar[na.coff + k];
    wave_mem_sync();
    na.coff = off;
    na.ccap = ncap;
  }
  int32_t* ar = arena_of(P, s.arena_sel);
  if (lane_id() == 0) {
    ar[na.coff + 2 * na.nchild] = tok;
    ar[na.coff + 2 * na.nchild + 1] = c;
    P.nodes[a].coff = na.coff;
    P.nodes[a].ccap = na.ccap;
    P.nodes[a].nchild = na.nchild + 1;
  }
  if (fence) wave_mem_sync();
  return true;
}

__device__ int32_t child_slot(const int32_t* ar, const NodeRec& na, int32_t c) {
  for (int32_t b = 0; b < na.nchild; b += KVR_WAVE) {
    int32_t k = b + lane_id();
    bool hit = (k < na.nchild) && (ar[na.coff + 2 * k + 1] == c);
    uint64_t m = __ballot(hit);
    if (m) return b + first_lane(m);
  }
  return -1;
}

// Remove child c of node a, whose record (as read by the caller) is na; na
// is updated to the new child count.  The last entry, which moves into the
// removed one's slot, is taken from the chunk just read when it is there
// (every array of up to 64 children).
__device__ __forceinline__ bool child_remove_rec(const Ptrs& P, const St& s, int32_t a, NodeRec& na, int32_t c) {
  int32_t* ar = arena_of(P, s.arena_sel);
  const int32_t last = na.nchild - 1;
  int32_t pos = -1;
  int2 lst = {0, 0};
  bool have_last = false;
  for (int32_t b = 0; b < na.nchild; b += KVR_WAVE) {
    const int32_t k = b + lane_id();
    int2 e = {0, -1};
    if (k < na.nchild) e = *reinterpret_cast<const int2*>(ar + na.coff + 2 * k);
    if (last >= b && last < b + KVR_WAVE) {
      lst.x = __builtin_amdgcn_readlane(e.x, last - b);
      lst.y = __builtin_amdgcn_readlane(e.y, last - b);
      have_last = true;
    }
    const uint64_t m = __ballot(k < na.nchild && e.y == c);
    if (m) {
      pos = b + first_lane(m);
      break;
    }
  }
  if (pos < 0) return false;
  if (pos != last && !have_last) lst = *reinterpret_cast<const int2*>(ar + na.coff + 2 * last);
  if (lane_id() == 0) {
    if (pos != last) *reinterpret_cast<int2*>(ar + na.coff + 2 * pos) = lst;
    P.nodes[a].nchild = last;
  }
  wave_mem_sync();
  na.nchild = last;
  return true;
}

__device__ __forceinline__ bool child_remove(const Ptrs& P, const St& s, int32_t a, int32_t c) {
  NodeRec na = P.nodes[a];
  int32_t* ar = arena_of(P, s.arena_sel);
  int32_t pos = child_slot(ar, na, c);
  if (pos < 0) return false;
  int32_t last = na.nchild - 1;
  if (lane_id() == 0) {
    if (pos != last) {
      ar[na.coff + 2 * pos] = ar[na.coff + 2 * last];
      ar[na.coff + 2 * pos + 1] = ar[na.coff + 2 * last + 1];
    }
    P.nodes[a].nchild = last;
  }
  wave_mem_sync();
  return true;
}

__device__ __forceinline__ bool child_replace(const Ptrs& P, const St& s, int32_t a, int32_t oldc, int32_t newc) {
  NodeRec na = P.nodes[a];
  int32_t* ar = arena_of(P, s.arena_sel);
  int32_t pos = child_slot(ar, na, oldc);
  if (pos < 0) return false;
  if (lane_id() == 0) ar[na.coff + 2 * pos + 1] = newc;
  wave_mem_sync();
  return true;
}

// Split node x at edge offset k (0 < k < len): a new head node takes
// positions [0, k) and x keeps [k, len) below it, so every leaf keeps its id.
__device__ __forceinline__ int32_t split_node(const Ptrs& P, St& s, int32_t x, int32_t k) {
  uint32_t coff;
  if (!arena_alloc(P, s, 4u, true, coff)) return -1;
  int32_t hd = node_alloc(P, s);
  if (hd < 0) return -1;
  NodeRec nx = P.nodes[x];
  int32_t* ar = arena_of(P, s.arena_sel);
  int32_t tail_tok = ar[nx.off + (uint32_t)k];
  NodeRec nh;
  nh.parent = nx.parent;
  nh.off = nx.off;
  nh.len = k;
  nh.nchild = 1;
  nh.coff = coff;
  nh.ccap = 2;
  nh.mphase = nx.mphase;
  nh.ma = nx.ma < k ? nx.ma : k;
  NodeRec nt;
  nt.parent = hd;
  nt.off = nx.off + (uint32_t)k;
  nt.len = nx.len - k;
  nt.nchild = nx.nchild;
  nt.coff = nx.coff;
  nt.ccap = nx.ccap;
  nt.mphase = nx.mphase;
  nt.ma = nx.ma - k > 0 ? nx.ma - k : 0;
  if (s.rnode == x) {
    if (s.rphase != s.phase) {
      s.rphase = 0;
    } else if (s.rhi <= k) {
      s.rnode = hd;
    } else if (s.rlo >= k) {
      s.rlo -= k;
      s.rhi -= k;
    } else {
      int32_t t = s.rhi - k;
      s.rnode = hd;
      s.rhi = k;
      if (nt.mphase == s.phase) {
        nt.ma = nt.ma > t ? nt.ma : t;
      } else {
        nt.mphase = s.phase;
        nt.ma = t;
      }
    }
  }
  if (lane_id() == 0) {
    ar[coff] = tail_tok;
    ar[coff + 1] = x;
  }
  node_put(P, hd, nh);
  node_put(P, x, nt);
  // every running path through x passes through its head
  if (P.pin != nullptr && lane_id() == 0) P.pin[hd] = P.pin[x];
  if (!child_replace(P, s, nx.parent, x, hd)) {
    KVR_FAIL_CHECK(s, 3, x, nx.parent, hd);
    return -1;
  }
  return hd;
}

// ---------------------------------------------------------------- match paths

// The nodes a match entered, kept (in LDS) per worker so that the next match
// on the same worker, and the insertion of a query routed there, can start
// from them instead of walking the tree again.  Entry e = (node, depth
// before its edge, depth after its edge); *cnt = number of entries, or
// kPathMax + 1 when the path was longer than kPathMax or is unknown.
constexpr int32_t kPathMax = 16;

struct PathRef {
  int32_t* node;
  int32_t* start;
  int32_t* end;
  int32_t* cnt;
};

__device__ __forceinline__ void path_add(const PathRef& pr, int32_t& pc, int32_t node, int32_t start, int32_t end) {
  if (pc < kPathMax && lane_id() == 0) {
    pr.node[pc] = node;
    pr.start[pc] = start;
    pr.end[pc] = end;
  }
  pc = pc < kPathMax ? pc + 1 : kPathMax + 1;
}

// ---------------------------------------------------------------- RLT pieces

// U := the leaves (other than `excl` and the running batch's nodes) whose
// leaf token is unmarked, in the order of the leaf list (lexicographic order
// of root paths).
__device__ __forceinline__ void rebuild_U(const Ptrs& P, St& s, int32_t excl) {
  constexpr int kUnroll = 4;  // four chunks of the leaf list per round trip
  uint32_t n = 0;
  for (uint32_t b = 0; b < s.nleaves; b += kUnroll * KVR_WAVE) {
    int32_t id[kUnroll];
#pragma unroll
    for (int v = 0; v < kUnroll; ++v) {
      const uint32_t k = b + (uint32_t)(v * KVR_WAVE) + (uint32_t)lane_id();
      id[v] = k < s.nleaves ? P.leaf[k] : -1;
    }
    NodeRec nd[kUnroll];
    bool pn[kUnroll];
#pragma unroll
    for (int v = 0; v < kUnroll; ++v) {
      pn[v] = false;
      if (id[v] > 0 && id[v] != excl) {
        nd[v] = P.nodes[id[v]];
        pn[v] = pinned(P, id[v]);
      }
    }
#pragma unroll
    for (int v = 0; v < kUnroll; ++v) {
      const bool cand = id[v] > 0 && id[v] != excl && !pn[v] && !is_marked(s, nd[v], id[v], nd[v].len - 1);
      const uint64_t m = __ballot(cand);
      if (cand) P.U[n + (uint32_t)__popcll(m & lanemask_lt())] = id[v];
      n += (uint32_t)__popcll(m);
    }
  }
  wave_mem_sync();
  s.nU = n;
  s.U_valid = 1;
}

// The candidate at U[kk], node n with parent p, has just lost its last
// token: drop it from the tree and the leaf list; its parent, if that became
// an unmarked leaf off the running batch, takes its place (and rank) in U,
// else the entry goes.
__device__ __forceinline__ bool remove_emptied(const Ptrs& P, St& s, uint32_t kk, int32_t n, int32_t p) {
  int32_t li = arr_find(P.leaf, s.nleaves, n);
  if (li < 0) {
    KVR_FAIL_CHECK(s, 12, n, s.nleaves, kk);
    return false;
  }
  if (!child_remove(P, s, p, n)) {
    KVR_FAIL_CHECK(s, 13, n, p, 0);
    return false;
  }
  node_free(P, s, n);
  NodeRec np = P.nodes[p];
  if (p != 0 && np.nchild == 0) {
    if (lane_id() == 0) P.leaf[li] = p;
    wave_mem_sync();
    if (!is_marked(s, np, p, np.len - 1) && !pinned(P, p)) {
      if (lane_id() == 0) P.U[kk] = p;
      wave_mem_sync();
    } else {
      arr_erase(P.U, s.nU, kk);
      s.nU -= 1;
    }
  } else {
    arr_erase(P.leaf, s.nleaves, (uint32_t)li);
    s.nleaves -= 1;
    arr_erase(P.U, s.nU, kk);
    s.nU -= 1;
  }
  return true;
}

// draws per lane in one staged eviction block
#ifndef KVR_EVICT_DRAWS
#define KVR_EVICT_DRAWS 4
#endif
constexpr int kEvictDraws = KVR_EVICT_DRAWS;

struct InsertArgs {
  uint64_t seed;
  uint64_t jg;        // global query index
  uint32_t worker;    // routed worker
  uint32_t replica;
  uint32_t B;
  uint32_t rn;        // the high halves of draw words 0..rn-1 are precomputed in rw
  const uint32_t* rw;
  // when non-null: the words are being written by nprog other waves in
  // rounds of `round` words (words [k*round, (k+1)*round) in round k), and
  // prog[w] (LDS, workgroup scope) counts the rounds drawing wave w has
  // completed
  const uint32_t* prog;
  uint32_t nprog;
  uint32_t round;
  // when non-null: another wave computes the new leaf's rank in the leaf
  // list from the recorded match path (new_leaf_rank on the tree before the
  // insertion) into *rank and then sets *rank_ready to 1, or to 2 when it
  // could not or the match ends inside an edge (LDS, workgroup scope)
  const int32_t* rank;
  const uint32_t* rank_ready;
};

// The new leaf's rank from the other wave (bounded wait), or -1 if it could
// not compute it or the wait ran out.
__device__ __forceinline__ int32_t await_rank(const InsertArgs& ia) {
  uint32_t spins = 0, rd;
  while ((rd = __hip_atomic_load(ia.rank_ready, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP)) == 0u) {
    if (++spins > (1u << 22)) break;
    __builtin_amdgcn_s_sleep(2);
  }
  return rd == 1u ? *ia.rank : -1;
}


// An insertion whose draw words take at most this many rounds waits for all
// of them at once (measured faster than starting on the first rounds).
constexpr uint32_t kAwaitAllRounds = 4;

// Wait (bounded) until draw words [0, need) of rw are written (need <= rn).
// Returns the count of words known to be there, at least need, or 0 if the
// wait ran out (the caller then computes every word itself).
__device__ __forceinline__ uint32_t await_words(const InsertArgs& ia, uint32_t need) {
  if (ia.rn <= kAwaitAllRounds * ia.round) need = ia.rn;
  const uint32_t want = (need + ia.round - 1u) / ia.round;  // rounds
  uint32_t spins = 0;
  for (;;) {
    bool late = false;
    if ((uint32_t)lane_id() < ia.nprog)
      late = __hip_atomic_load(ia.prog + lane_id(), __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < want;
    if (!__ballot(late)) {
      const uint64_t have = (uint64_t)want * ia.round;
      return have < ia.rn ? (uint32_t)have : ia.rn;
    }
    if (++spins > (1u << 22)) return 0u;
    __builtin_amdgcn_s_sleep(2);
  }
}

// Word 0 of Philox4x64-10 for draw d of this insertion: key (seed, replica),
// counter (query index, worker, d, 0).
__device__ __noinline__ uint64_t draw_word_slow(uint64_t jg, uint64_t worker, uint64_t d, uint64_t seed,
                                                uint64_t replica) {
  return philox_word0(jg, worker, d, 0ull, seed, replica);
}

__device__ __forceinline__ uint64_t draw_word(const InsertArgs& ia, uint64_t d) {
  return draw_word_slow(ia.jg, ia.worker, d, ia.seed, ia.replica);
}

// Index floor(r * n / 2^64) of a draw from the high half of r alone: with
// A = r_hi * n, the index is (A + floor(r_lo * n / 2^32)) / 2^32, and the
// second term (< n) can carry into the high half only when the low half of A
// is above 2^32 - n.  Returns false in that case (the full word decides).
__device__ __forceinline__ bool draw_index_hi(uint32_t r_hi, uint32_t n, uint32_t& k) {
  const uint64_t A = (uint64_t)r_hi * n;
  k = (uint32_t)(A >> 32);
  return (uint32_t)A <= 0xffffffffu - n + 1u;
}

// Evict with draws dctr .. dctr+cnt-1 (cnt <= wave width), one lane per
// draw, all taken against the current U: a draw only trims the leaf token of
// its candidate, so draws commute until one takes a candidate's last
// evictable token (the next token is marked, or the node empties), which is
// the only event that changes U.  Commits the draws up to and including the
// first such one, applies it, and returns the number of draws consumed in
// `done`.  Identical to taking the draws one at a time.
__device__ __forceinline__ bool evict_block(const Ptrs& P, St& s, const InsertArgs& ia, uint64_t dctr, uint32_t cnt,
                            uint32_t& done) {
  const int lane = lane_id();
  const bool act = (uint32_t)lane < cnt;
  uint32_t kk = 0;
  int32_t n = 0;
  const uint64_t d = dctr + (uint64_t)lane;
  bool exact = false;
  if (act && d < ia.rn) exact = draw_index_hi(ia.rw[d], s.nU, kk);
  if (act && !exact) kk = (uint32_t)__umul64hi(draw_word(ia, d), (uint64_t)s.nU);
  if (act) n = P.U[kk];
  if (__ballot(act && (n <= 0 || (uint32_t)n >= s.hwm))) {
    KVR_FAIL_CHECK(s, 10, kk, n, s.nU);
    return false;
  }
  NodeRec nd = P.nodes[act ? n : 0];
  int32_t top = (nd.mphase == s.phase) ? nd.ma : 0;
  if (s.rphase == s.phase && s.rnode == n && s.rhi > top) top = s.rhi;
  const int32_t e = nd.len - top;  // evictable tail tokens of my candidate
  if (__ballot(act && (e <= 0 || nd.nchild != 0 || nd.parent < 0))) {
    KVR_FAIL_CHECK(s, 11, n, nd.len, nd.nchild);
    return false;
  }
  // c = draws on my candidate up to and including mine; grp = their lanes
  uint64_t todo = __ballot(act);
  uint64_t grp = 0;
  int32_t c = 0;
  while (todo) {
    const int ld = first_lane(todo);
    const uint32_t v = (uint32_t)__builtin_amdgcn_readlane((int)kk, ld);
    const bool same = act && kk == v;
    const uint64_t m = __ballot(same);
    if (same) {
      grp = m;
      c = __popcll(m & lanemask_le());
    }
    todo &= ~m;
  }
  const uint64_t exm = __ballot(act && c == e);
  const int f = exm ? first_lane(exm) : (int)cnt - 1;  // last committed draw
  const uint64_t commit = (2ull << (uint32_t)f) - 1ull;
  const uint64_t mine = grp & commit;
  // the last committed draw on each candidate writes its new length
  if (act && lane <= f && mine && 63 - __clzll((long long)mine) == lane)
    P.nodes[n].len = nd.len - __popcll(mine);
  wave_mem_sync();
  done = (uint32_t)f + 1u;
  if (exm) {
    const uint32_t kkf = (uint32_t)__builtin_amdgcn_readlane((int)kk, f);
    const int32_t nf = __builtin_amdgcn_readlane(n, f);
    const int32_t pf = __builtin_amdgcn_readlane(nd.parent, f);
    const int32_t left = __builtin_amdgcn_readlane(top, f);
    if (left > 0) {  // the next token is marked: no longer a candidate
      arr_erase(P.U, s.nU, kkf);
      s.nU -= 1;
    } else if (!remove_emptied(P, s, kkf, nf, pf)) {
      return false;
    }
  }
  return true;
}

// The candidate list staged in LDS for the eviction phase of an insertion:
// entry k = (node, length, mark_top, parent) of U[k].  While staged, the LDS
// copy is authoritative for U and for the lengths of the staged nodes; the
// tree, leaf list and child arrays stay in global memory.
struct UStage {
  int32_t* node;
  int32_t* len;
  int32_t* top;
  int32_t* par;
  uint32_t cap;
};

__device__ __forceinline__ bool stage_in(const Ptrs& P, St& s, const UStage& u) {
  constexpr int kUnroll = 4;  // four chunks of the list per round trip
  bool bad = false;
  for (uint32_t b = 0; b < s.nU; b += kUnroll * KVR_WAVE) {
    int32_t n[kUnroll];
#pragma unroll
    for (int v = 0; v < kUnroll; ++v) {
      const uint32_t k = b + (uint32_t)(v * KVR_WAVE) + (uint32_t)lane_id();
      n[v] = k < s.nU ? P.U[k] : 0;
    }
    NodeRec nd[kUnroll];
#pragma unroll
    for (int v = 0; v < kUnroll; ++v) {
      const uint32_t k = b + (uint32_t)(v * KVR_WAVE) + (uint32_t)lane_id();
      const bool ok = k < s.nU && n[v] > 0 && (uint32_t)n[v] < s.hwm;
      if (k < s.nU && !ok) bad = true;
      if (ok) nd[v] = P.nodes[n[v]];
    }
#pragma unroll
    for (int v = 0; v < kUnroll; ++v) {
      const uint32_t k = b + (uint32_t)(v * KVR_WAVE) + (uint32_t)lane_id();
      if (k < s.nU && n[v] > 0 && (uint32_t)n[v] < s.hwm) {
        u.node[k] = n[v];
        u.len[k] = nd[v].len;
        u.top[k] = mark_top(s, nd[v], n[v]);
        u.par[k] = nd[v].parent;
      }
    }
  }
  if (__ballot(bad)) {
    KVR_FAIL_CHECK(s, 14, s.nU, s.hwm, 0);
    return false;
  }
  return true;
}

// Write the staged list back.  fence = false when the caller's own fence
// follows before anything reads U or the node lengths again.
__device__ __forceinline__ void stage_out(const Ptrs& P, const St& s, const UStage& u, bool fence = true) {
  for (uint32_t b = 0; b < s.nU; b += KVR_WAVE) {
    const uint32_t k = b + (uint32_t)lane_id();
    if (k < s.nU) {
      const int32_t n = u.node[k];
      P.U[k] = n;
      P.nodes[n].len = u.len[k];
    }
  }
  if (fence) wave_mem_sync();
}

// remove entry pos of the staged list (n entries); LDS only, so the wave's
// in-order LDS accesses need no fence
__device__ __forceinline__ void stage_erase(const UStage& u, uint32_t n, uint32_t pos) {
  for (uint32_t lo = pos; lo + 1 < n; lo += KVR_WAVE) {
    const uint32_t k = lo + (uint32_t)lane_id();
    int32_t a = 0, b = 0, c = 0, d = 0;
    if (k + 1 < n) {
      a = u.node[k + 1];
      b = u.len[k + 1];
      c = u.top[k + 1];
      d = u.par[k + 1];
    }
    __builtin_amdgcn_wave_barrier();
    if (k + 1 < n) {
      u.node[k] = a;
      u.len[k] = b;
      u.top[k] = c;
      u.par[k] = d;
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// evict_block with U staged in LDS (same draws, same result), kDraws draws
// per lane: draw j of the block is taken by lane j % wave in slot j / wave.
// Every draw of the block first trims its candidate with an LDS atomic; the
// values the atomics return show whether some candidate ran out of
// evictable tokens.  Only then (rarely) is the first exhausting draw in draw
// order found exactly and the draws after it are undone.
template <int kDraws>
__device__ __forceinline__ bool evict_block_staged(const Ptrs& P, St& s, const InsertArgs& ia, const UStage& u,
                                                   uint64_t dctr, uint32_t cnt, uint32_t& done, bool& changed) {
  changed = false;
  const int lane = lane_id();
  bool act[kDraws];
  uint32_t kk[kDraws];
  int32_t top[kDraws], old[kDraws];
  // no divergent branch around the LDS accesses, so all of them can be in
  // flight at once: inactive lanes read entry 0 and subtract 0
  bool exact = true;
  if (dctr + cnt <= ia.rn) {
    // every active draw's high half is precomputed; inactive lanes read the
    // last one.  All the loads first, so they are in flight together.
    uint32_t wv[kDraws];
#pragma unroll
    for (int r = 0; r < kDraws; ++r) {
      uint64_t d = dctr + (uint64_t)(r * KVR_WAVE + lane);
      if (d >= dctr + cnt) d = dctr + cnt - 1u;
      wv[r] = ia.rw[d];
    }
#pragma unroll
    for (int r = 0; r < kDraws; ++r) {
      act[r] = (uint32_t)(r * KVR_WAVE + lane) < cnt;
      uint32_t k = 0;
      const bool ok = draw_index_hi(wv[r], s.nU, k);
      kk[r] = act[r] ? k : 0u;
      if (act[r] && !ok) exact = false;
    }
  } else {
#pragma unroll
    for (int r = 0; r < kDraws; ++r) act[r] = (uint32_t)(r * KVR_WAVE + lane) < cnt;
    exact = false;
  }
  if (__ballot(!exact)) {
    // rare: whole words for this block
#pragma unroll
    for (int r = 0; r < kDraws; ++r)
      kk[r] = act[r] ? (uint32_t)__umul64hi(draw_word(ia, dctr + (uint64_t)(r * KVR_WAVE + lane)), (uint64_t)s.nU)
                     : 0u;
  }
#pragma unroll
  for (int r = 0; r < kDraws; ++r) {
    top[r] = u.top[kk[r]];
    old[r] = atomicSub(&u.len[kk[r]], act[r] ? 1 : 0);
  }
  // the decrements of one candidate return distinct values len, len-1, ...;
  // the one returning top + 1 took its last evictable token
  uint64_t exm[kDraws];
  uint64_t anyx = 0, over = 0;
#pragma unroll
  for (int r = 0; r < kDraws; ++r) {
    exm[r] = __ballot(act[r] && old[r] == top[r] + 1);
    anyx |= exm[r];
    over |= __ballot(act[r] && old[r] <= top[r]);
  }
  int f = (int)cnt - 1;  // last committed draw
  if (anyx) {
    // exhausting draw of each exhausted candidate, in draw order: the e-th
    // of the draws on it, e = its evictable tokens before the block
#pragma unroll
    for (int rx = 0; rx < kDraws; ++rx) {
      uint64_t todo = exm[rx];
      while (todo) {
        const int x = first_lane(todo);
        todo &= todo - 1ull;
        const uint32_t v = (uint32_t)__builtin_amdgcn_readlane((int)kk[rx], x);
        const int32_t tv = __builtin_amdgcn_readlane(top[rx], x);
        int e = 0;
#pragma unroll
        for (int r = 0; r < kDraws; ++r) e += __popcll(__ballot(act[r] && kk[r] == v && old[r] > tv));
        int fx = -1;
#pragma unroll
        for (int r = 0; r < kDraws; ++r) {
          uint64_t m = __ballot(act[r] && kk[r] == v);
          const int c = __popcll(m);
          if (fx < 0) {
            if (e <= c) {
              for (int q = 1; q < e; ++q) m &= m - 1ull;
              fx = r * KVR_WAVE + first_lane(m);
            } else {
              e -= c;
            }
          }
        }
        if (fx >= 0 && fx < f) f = fx;
      }
    }
    bool bad = false;
#pragma unroll
    for (int r = 0; r < kDraws; ++r) {
      const int j = r * KVR_WAVE + lane;
      atomicAdd(&u.len[kk[r]], (act[r] && j > f) ? 1 : 0);
    }
    // every committed draw leaves its candidate with len >= top
#pragma unroll
    for (int r = 0; r < kDraws; ++r) {
      const int j = r * KVR_WAVE + lane;
      if (act[r] && j <= f && u.len[kk[r]] < top[r]) bad = true;
    }
    if (__ballot(bad)) {
      KVR_FAIL_CHECK(s, 11, (int32_t)cnt, f, 1);
      return false;
    }
  } else if (over) {
    // a candidate without an evictable token
    KVR_FAIL_CHECK(s, 11, (int32_t)cnt, first_lane(over), 0);
    return false;
  }
  // the exhausting draw's slot and lane
  const int rf = f / KVR_WAVE, lf = f % KVR_WAVE;
  uint32_t kkr = kk[0];
  int32_t topr = top[0];
#pragma unroll
  for (int r = 1; r < kDraws; ++r)
    if (rf == r) {
      kkr = kk[r];
      topr = top[r];
    }
  done = (uint32_t)f + 1u;
  if (anyx) {
    changed = true;
    const uint32_t kkf = (uint32_t)__builtin_amdgcn_readlane((int)kkr, lf);
    const int32_t nf = u.node[kkf];
    const int32_t pf = u.par[kkf];
    const int32_t left = __builtin_amdgcn_readlane(topr, lf);
    if (pf < 0 || nf <= 0) {
      KVR_FAIL_CHECK(s, 11, nf, pf, 2);
      return false;
    }
    if (left > 0) {  // the next token is marked: no longer a candidate
      if (lane == 0) P.nodes[nf].len = left;
      wave_mem_sync();
      stage_erase(u, s.nU, kkf);
      s.nU -= 1;
      return true;
    }
    // the node is empty: drop it; its parent may take its place.  The
    // parent's record is read together with the leaf list.
    NodeRec np = P.nodes[pf];
    const int32_t li = arr_find(P.leaf, s.nleaves, nf);
    if (li < 0) {
      KVR_FAIL_CHECK(s, 12, nf, s.nleaves, kkf);
      return false;
    }
    // unless the parent takes the leaf-list entry over, the entry goes: the
    // first chunk of that shift is read together with the child array
    const bool takeover = pf != 0 && np.nchild == 1;
    int32_t shift0 = 0;
    const uint32_t k0 = (uint32_t)li + (uint32_t)lane_id();
    if (!takeover && k0 + 1u < s.nleaves) shift0 = P.leaf[k0 + 1u];
    if (!child_remove_rec(P, s, pf, np, nf)) {
      KVR_FAIL_CHECK(s, 13, nf, pf, 0);
      return false;
    }
    node_free(P, s, nf);
    if (takeover) {
      if (lane == 0) P.leaf[li] = pf;
      wave_mem_sync();
      const int32_t ptop = mark_top(s, np, pf);
      if (ptop < np.len && !pinned(P, pf)) {
        if (lane == 0) {
          u.node[kkf] = pf;
          u.len[kkf] = np.len;
          u.top[kkf] = ptop;
          u.par[kkf] = np.parent;
        }
      } else {
        stage_erase(u, s.nU, kkf);
        s.nU -= 1;
      }
    } else {
      if (k0 + 1u < s.nleaves) P.leaf[k0] = shift0;
      wave_mem_sync();
      if ((uint32_t)li + (uint32_t)KVR_WAVE + 1u < s.nleaves)
        arr_erase(P.leaf, s.nleaves, (uint32_t)li + (uint32_t)KVR_WAVE);
      s.nleaves -= 1;
      stage_erase(u, s.nU, kkf);
      s.nU -= 1;
    }
  }
  return true;
}

// RLT insertion of q[0, L) into the worker's cache; h = LCP(q, cache).
// Returns the KVR_DEV_* error bits (0 on success).
__device__ __forceinline__ NodeRec node_from_lane(const NodeRec& v, int e) {
  NodeRec r;
  r.parent = __builtin_amdgcn_readlane(v.parent, e);
  r.off = (uint32_t)__builtin_amdgcn_readlane((int)v.off, e);
  r.len = __builtin_amdgcn_readlane(v.len, e);
  r.nchild = __builtin_amdgcn_readlane(v.nchild, e);
  r.coff = (uint32_t)__builtin_amdgcn_readlane((int)v.coff, e);
  r.ccap = __builtin_amdgcn_readlane(v.ccap, e);
  r.mphase = (uint32_t)__builtin_amdgcn_readlane((int)v.mphase, e);
  r.ma = __builtin_amdgcn_readlane(v.ma, e);
  return r;
}

// The eviction half of an RLT insertion, as the front half leaves it: the
// cache state after the marks of the cached part and the load of the new
// leaf, and what the evictions of the loaded tokens need.  The front half
// may run on one wave and the back half on another.
struct EvictJob {
  St s;
  InsertArgs ia;
  int32_t h, L;       // cached length and length of the inserted path
  int32_t l;          // the new leaf node holding q[h, L) (when h < L)
  uint32_t nfree;     // free token slots before the load
  uint32_t nev;       // evictions the load needs
  uint32_t c0;        // |T| before the loaded tokens were marked
  int32_t reset_at;   // path position at which |T| reaches B+1 among the loads, or -1
  uint32_t worker;
  uint32_t final_size;  // |S| after the insertion
};

// Front half of the RLT insertion of q[0, L) into the worker's cache (h =
// LCP(q, cache); pr holds the path of that match, or is marked unknown):
// the marking walk over the cached part (Algorithm 1: each token joins T,
// with the reset to {t} when |T| reaches B+1), the split of the edge the
// match ends in, the new leaf's rank in the leaf list, and the load of
// q[h, L) as one new leaf node.  pr then holds the path of q in the updated
// cache, which the evictions never touch.  The evictions and the marks of
// the loaded tokens are left in *job for rlt_insert_back.  Returns the
// KVR_DEV_* error bits (0 on success).
template <bool PT = false>
__device__ __forceinline__ uint32_t rlt_insert_front(const Ptrs& P, const InsertArgs& ia, const int32_t* qs, int32_t L,
                                                     int32_t h, const PathRef& pr, int64_t* dbg, EvictJob& job,
                                                     PhaseClock* clk = nullptr) {
  St s = load_st(P.hdr);
  const uint32_t B = ia.B;
  int32_t* ar = arena_of(P, s.arena_sel);
  const int32_t pc = *pr.cnt;
  const bool have_path = pc <= kPathMax;
  bool split = false;
  int32_t a = 0, l = 0, laststart = 0, pe = 0;

  // ---- walk the cached part of the path and mark it: along the recorded
  // path (node records of all its entries loaded at once) or, when there is
  // none, by child lookups
  NodeRec pre;
  pre.parent = pre.len = pre.nchild = pre.ccap = pre.ma = 0;
  pre.off = pre.coff = pre.mphase = 0;
  if (KVR_WAVE >= kPathMax && have_path && lane_id() < pc) pre = P.nodes[pr.node[lane_id()]];
  int32_t x = 0, d = 0, last = 0, lastcov = 0;
  // the record of `last` (its length and child array: the marks below do
  // not change them)
  NodeRec lastrec = pre;
  while (d < h) {
    int32_t c;
    NodeRec nc;
    if (have_path) {
      if (pe >= pc || pr.start[pe] != d) {
        KVR_FAIL_CHECK(s, 1, pe, d, h);
        goto fail;
      }
      c = pr.node[pe];
      if (c <= 0 || (uint32_t)c >= s.hwm) {
        KVR_FAIL_CHECK(s, 1, c, d, h);
        goto fail;
      }
      if (KVR_WAVE >= kPathMax) {
        nc = node_from_lane(pre, pe);
      } else {
        nc = P.nodes[c];
      }
      ++pe;
    } else {
      NodeRec nx = P.nodes[x];
      c = child_find(ar, nx, qs[d]);
      if (c <= 0 || (uint32_t)c >= s.hwm) {
        KVR_FAIL_CHECK(s, 1, x, d, h);
        goto fail;
      }
      nc = P.nodes[c];
    }
    int32_t cov = nc.len < h - d ? nc.len : h - d;
    if (cov <= 0) {
      KVR_FAIL_CHECK(s, 2, c, nc.len, d);
      goto fail;
    }
    bool was_cand = (nc.nchild == 0) && !is_marked(s, nc, c, nc.len - 1);
    int32_t ma = (nc.mphase == s.phase) ? nc.ma : 0;
    bool rv = (s.rphase == s.phase) && (s.rnode == c);
    int32_t rlo = s.rlo, rhi = s.rhi;
    if (rv && rlo <= ma) {  // the reset interval touches the prefix: merge
      ma = ma > rhi ? ma : rhi;
      rv = false;
      s.rphase = 0;
    }
    int32_t m1 = ma < cov ? ma : cov;
    int32_t m2 = 0;
    if (rv) {
      int32_t e = rhi < cov ? rhi : cov;
      m2 = e - rlo > 0 ? e - rlo : 0;
    }
    int32_t newly = cov - m1 - m2;
    if (s.cnt + (uint32_t)newly <= B) {
      s.cnt += (uint32_t)newly;
      int32_t nma = ma > cov ? ma : cov;
      if (rv && rlo <= nma) {
        nma = nma > rhi ? nma : rhi;
        s.rphase = 0;
      }
      if (lane_id() == 0) {
        P.nodes[c].mphase = s.phase;
        P.nodes[c].ma = nma;
      }
    } else {
      // |T| reaches B+1 at the `need`-th newly marked position of this edge
      int32_t need = (int32_t)(B + 1u - s.cnt);
      int32_t rp;
      if (!rv) {
        rp = ma + need - 1;
      } else {
        int32_t e1 = rlo < cov ? rlo : cov;
        int32_t s1 = e1 - ma > 0 ? e1 - ma : 0;
        rp = need <= s1 ? ma + need - 1 : rhi + (need - s1) - 1;
      }
      s.phase += 1;
      s.U_valid = 0;
      s.cnt = (uint32_t)(cov - rp);
      if (rp == 0) {
        if (lane_id() == 0) {
          P.nodes[c].mphase = s.phase;
          P.nodes[c].ma = cov;
        }
      } else {
        s.rnode = c;
        s.rlo = rp;
        s.rhi = cov;
        s.rphase = s.phase;
      }
    }
    if (was_cand && s.U_valid && cov == nc.len) {
      // a candidate's leaf token was marked
      int32_t pos = arr_find(P.U, s.nU, c);
      if (pos >= 0) {
        arr_erase(P.U, s.nU, (uint32_t)pos);
        s.nU -= 1;
      }
    }
    laststart = d;
    d += cov;
    last = c;
    lastcov = cov;
    lastrec = nc;
    x = c;
  }
  wave_mem_sync();  // the marks above are read again below
  clock_mark<PT>(clk, KVR_PHASE_MARK);

  if (h < L) {
    const int32_t nload = L - h;
    // ---- attachment point: end of `last`, splitting it if needed
    a = last;
    if (h > 0 && lastcov < lastrec.len) {
      a = split_node(P, s, last, lastcov);
      if (a < 0) goto fail;
      split = true;
      ar = arena_of(P, s.arena_sel);
    }
    // ---- rank of the new leaf in the leaf list: from another wave, which
    // computes it on the tree before this insertion while this one marks
    // (only when no edge is split: that would change what it reads), or here
    int32_t pos = -1;
    const bool rank_helper = ia.rank != nullptr && have_path && !split;
    // a's child count, capacity and array offset, for the child added below
    int32_t a_known[3];
    if (h > 0 && !split) {
      a_known[0] = lastrec.nchild;
      a_known[1] = lastrec.ccap;
      a_known[2] = (int32_t)lastrec.coff;
    } else {
      const NodeRec na = P.nodes[a];
      a_known[0] = na.nchild;
      a_known[1] = na.ccap;
      a_known[2] = (int32_t)na.coff;
    }
    const uint32_t a_sel = s.arena_sel;
    const bool replace = a != 0 && a_known[0] == 0;
    // the free list's next entry, loaded before the stores below (an
    // allocation after them would wait for them)
    const int32_t fh = s.free_head;
    uint32_t fh_next = 0;
    if (fh >= 0) fh_next = P.nodes[fh].off;
    if (!rank_helper) pos = new_leaf_rank(P, s, ar, split ? last : a, 0, split ? 1 : 0, qs[h]);
    // ---- the new leaf node holding q[h, L)
    bool ranked = false;
    if (rank_helper && (uint64_t)s.arena_top + (uint32_t)nload > P.A) {
      // a collection is coming, which moves what the other wave reads
      pos = await_rank(ia);
      if (pos < 0) pos = new_leaf_rank(P, s, ar, a, 0, 0, qs[h]);
      ranked = true;
    }
    uint32_t eoff;
    if (!arena_alloc(P, s, (uint32_t)nload, false, eoff)) goto fail;
    ar = arena_of(P, s.arena_sel);
    // no fence here: nothing in this insertion reads the new edge's tokens
    // except a collection, which fences first; the fence at the end of the
    // insertion orders them before the next match
    wave_copy(ar + eoff, qs + h, nload);
    if (rank_helper && !ranked) {
      // if the other wave could not, or takes too long, rank here (the tree
      // is as the local ranking above would see it)
      pos = await_rank(ia);
      if (pos < 0) pos = new_leaf_rank(P, s, ar, a, 0, 0, qs[h]);
    }
    if (fh >= 0 && s.free_head == fh) {
      l = fh;
      s.free_head = (int32_t)fh_next;
      s.nnodes += 1;
    } else {
      l = node_alloc(P, s);
    }
    if (l < 0) goto fail;
    // the new node, child entry and leaf-list entry: none of these stores is
    // read again before the fence that ends this half (a collection fences
    // first), so they are not fenced one by one
    if (lane_id() == 0) {
      NodeRec nl;
      nl.parent = a;
      nl.off = eoff;
      nl.len = nload;
      nl.nchild = 0;
      nl.coff = 0;
      nl.ccap = 0;
      nl.mphase = 0;
      nl.ma = 0;
      P.nodes[l] = nl;
    }
    if (!child_add(P, s, a, qs[h], l, a_known, a_sel, false)) goto fail;
    ar = arena_of(P, s.arena_sel);
    if (pos < 0 || (uint32_t)pos > s.nleaves) {
      KVR_FAIL_CHECK(s, 4, pos, s.nleaves, a);
      goto fail;
    }
    if (replace) {
      if (lane_id() == 0) P.leaf[pos] = l;
    } else {
      arr_insert(P.leaf, s.nleaves, (uint32_t)pos, l, false);
      s.nleaves += 1;
    }
    clock_mark<PT>(clk, KVR_PHASE_LOAD);

    // ---- what the evictions of the loaded tokens need
    job.nfree = B - s.size;
    job.nev = (uint32_t)nload > job.nfree ? (uint32_t)nload - job.nfree : 0u;
    job.c0 = s.cnt;
    job.reset_at = (job.c0 + (uint32_t)nload >= B + 1u) ? h + (int32_t)(B - job.c0) : -1;
    job.l = l;
  } else {
    job.nfree = B - s.size;
    job.nev = 0;
    job.c0 = s.cnt;
    job.reset_at = -1;
    job.l = 0;
  }
  // ---- the path of q in the updated cache: the walked entries (the split
  // head in place of the split node) and the new leaf
  {
    int32_t fc = have_path ? pe : kPathMax + 1;
    if (fc <= kPathMax) {
      if (split) {
        int32_t f1 = fc - 1;
        path_add(pr, f1, a, laststart, laststart + lastcov);
      }
      if (h < L) path_add(pr, fc, l, h, L);
    }
    if (lane_id() == 0) *pr.cnt = fc;
  }
  job.s = s;
  job.ia = ia;
  job.h = h;
  job.L = L;
  job.worker = ia.worker;
  job.final_size = s.size + (uint32_t)(L - h) - job.nev;
  wave_mem_sync();  // the tree edits before the back half reads them (maybe on another wave)
  return 0;
fail:
  if (lane_id() == 0) *pr.cnt = kPathMax + 1;
  store_st(P.hdr, s);
  if (dbg) {
    dbg[0] = s.dbg_check;
    dbg[1] = s.dbg_val[0];
    dbg[2] = s.dbg_val[1];
    dbg[3] = s.dbg_val[2];
  }
  return s.err ? s.err : (uint32_t)KVR_DEV_INTERNAL;
}

// Back half of the RLT insertion (after rlt_insert_front, on the state in
// *job): for each loaded token into a full cache, evict the candidate
// U[floor(r * |U| / 2^64)] (Algorithm 1; U in lexicographic order; r the
// draw's Philox word), in blocks of draws that commute; the phase reset
// where |T| reaches B+1 among the loaded tokens; then the marks of the
// loaded tokens and the cache header.  Returns the KVR_DEV_* error bits.
template <bool PT = false>
__device__ __forceinline__ uint32_t rlt_insert_back(const Ptrs& P, const EvictJob& job, const UStage& ustage,
                                                    int64_t* dbg, PhaseClock* clk = nullptr,
                                                    int ph_evict = KVR_PHASE_EVICT, int ph_finish = KVR_PHASE_FINISH) {
  St s = job.s;
  const int32_t h = job.h, L = job.L, l = job.l;
  if (h < L) {
    const int32_t nload = L - h;
    const uint32_t nfree = job.nfree;
    const uint32_t nev = job.nev;
    const uint32_t c0 = job.c0;
    int32_t reset_at = job.reset_at;
    bool applied = false;
    uint64_t dctr = 0;
    uint32_t k = 0;
    bool staged = false;
    InsertArgs iq = job.ia;
    // draw words [0, have) are known to be written; before a block reads
    // words past that, wait for the drawing waves' rounds to cover them
    // (bounded: past it the words are computed here instead)
    uint32_t have = iq.prog ? 0u : iq.rn;
    while (k < nev) {
      const int32_t p = h + (int32_t)nfree + (int32_t)k;
      if (reset_at >= 0 && !applied && p >= reset_at) {
        if (staged) {
          stage_out(P, s, ustage);
          staged = false;
        }
        s.phase += 1;
        s.U_valid = 0;
        applied = true;
      }
      if (!s.U_valid) rebuild_U(P, s, l);
      if (s.nU == 0) {
        // no unmarked leaf: a new phase starts with the current token
        if (staged) {
          stage_out(P, s, ustage);
          staged = false;
        }
        s.phase += 1;
        hdr_count(&P.hdr->forced_resets, 1u);
        rebuild_U(P, s, l);
        reset_at = p;
        applied = true;
        if (s.nU == 0) {  // only possible for a path longer than the cache
          KVR_FAIL_CHECK(s, 6, p, s.nleaves, L);
          goto fail;
        }
      }
      if (!staged && s.nU <= ustage.cap) {
        if (!stage_in(P, s, ustage)) goto fail;
        staged = true;
      }
      // draws for positions p, p+1, ...: never across a pending phase reset
      uint32_t lim = nev;
      if (reset_at >= 0 && !applied && (uint32_t)(reset_at - p) < nev - k) lim = k + (uint32_t)(reset_at - p);
      if (staged) {
        // blocks against the staged list until the limit or until U changes;
        // the loop state is wave-uniform, so keep it in scalar registers
        uint32_t ku = (uint32_t)__builtin_amdgcn_readfirstlane((int)k);
        const uint32_t limu = (uint32_t)__builtin_amdgcn_readfirstlane((int)lim);
        uint32_t du = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)dctr);
        s.nU = (uint32_t)__builtin_amdgcn_readfirstlane((int)s.nU);
        bool ok = true;
        while (ku < limu) {
          constexpr uint32_t kSpan = (uint32_t)kEvictDraws * KVR_WAVE;
          const uint32_t cnt = limu - ku < kSpan ? limu - ku : kSpan;
          if (du + cnt > have && have < iq.rn) {
            const uint32_t need = du + cnt < iq.rn ? du + cnt : iq.rn;
            have = await_words(iq, need);
            if (have == 0u) iq.rn = 0;
          }
          uint32_t done = 0;
          bool changed = false;
          ok = evict_block_staged<kEvictDraws>(P, s, iq, ustage, (uint64_t)du, cnt, done, changed);
          if (!ok) break;
          done = (uint32_t)__builtin_amdgcn_readfirstlane((int)done);
          du += done;
          ku += done;
          if (changed) break;
        }
        k = ku;
        dctr = du;
        if (!ok) goto fail;
      } else {
        const uint32_t cnt = lim - k < (uint32_t)KVR_WAVE ? lim - k : (uint32_t)KVR_WAVE;
        if (dctr + cnt > have && have < iq.rn) {
          const uint32_t need = (uint32_t)dctr + cnt < iq.rn ? (uint32_t)dctr + cnt : iq.rn;
          have = await_words(iq, need);
          if (have == 0u) iq.rn = 0;
        }
        uint32_t done = 0;
        if (!evict_block(P, s, iq, dctr, cnt, done)) goto fail;
        dctr += done;
        k += done;
      }
    }
    // no fence: the insertion's last fence orders these stores before any
    // later read
    if (staged) stage_out(P, s, ustage, false);
    clock_mark<PT>(clk, ph_evict);
    if (reset_at >= 0 && !applied) {
      s.phase += 1;
      s.U_valid = 0;
      applied = true;
    }
    if (applied) {
      const int32_t lo = reset_at - h;
      s.cnt = (uint32_t)(L - reset_at);
      if (lo == 0) {
        if (lane_id() == 0) {
          P.nodes[l].mphase = s.phase;
          P.nodes[l].ma = nload;
        }
      } else {
        s.rnode = l;
        s.rlo = lo;
        s.rhi = nload;
        s.rphase = s.phase;
      }
    } else {
      s.cnt = c0 + (uint32_t)nload;
      if (lane_id() == 0) {
        P.nodes[l].mphase = s.phase;
        P.nodes[l].ma = nload;
      }
    }
    s.size = s.size + (uint32_t)nload - nev;
    hdr_count(&P.hdr->loads, (uint64_t)nload);
    hdr_count(&P.hdr->evictions, nev);
  }
  store_st(P.hdr, s);
  wave_mem_sync();
  clock_mark<PT>(clk, ph_finish);
  return 0;
fail:
  store_st(P.hdr, s);
  if (dbg) {
    dbg[0] = s.dbg_check;
    dbg[1] = s.dbg_val[0];
    dbg[2] = s.dbg_val[1];
    dbg[3] = s.dbg_val[2];
  }
  return s.err ? s.err : (uint32_t)KVR_DEV_INTERNAL;
}

// RLT insertion of q[0, L) into the worker's cache on one wave: the front
// half, then the back half.  On return pr holds the path of q in the
// updated cache.  Returns the KVR_DEV_* error bits (0 on success).
template <bool PT = false>
__device__ __forceinline__ uint32_t rlt_insert(const Ptrs& P, const InsertArgs& ia, const int32_t* qs, int32_t L,
                                               int32_t h, const UStage& ustage, const PathRef& pr, int64_t* dbg,
                                               PhaseClock* clk = nullptr) {
  EvictJob job;
  uint32_t err = rlt_insert_front<PT>(P, ia, qs, L, h, pr, dbg, job, clk);
  if (err) return err;
  err = rlt_insert_back<PT>(P, job, ustage, dbg, clk);
  if (err && lane_id() == 0) *pr.cnt = kPathMax + 1;
  return err;
}

// ---------------------------------------------------------------- continuous batching

// Lower the in-progress count of every node from x up to the root (the
// nodes of a path leaving the running batch).  A leaf released that way
// whose leaf token is unmarked is a candidate again: U is rebuilt from its
// definition at the next draw.
__device__ __forceinline__ bool unpin_chain(const Ptrs& P, St& s, int32_t x) {
  for (uint32_t guard = 0; x > 0; ++guard) {
    if (guard > P.NC || (uint32_t)x >= s.hwm) {
      KVR_FAIL_CHECK(s, 21, x, guard, 0);
      return false;
    }
    const NodeRec nx = P.nodes[x];
    const int32_t c = P.pin[x] - 1;
    if (c < 0) {
      KVR_FAIL_CHECK(s, 22, x, c, 0);
      return false;
    }
    if (lane_id() == 0) P.pin[x] = c;
    if (c == 0 && nx.nchild == 0 && !is_marked(s, nx, x, nx.len - 1)) s.U_valid = 0;
    x = nx.parent;
  }
  return true;
}

// Continuous batching (Sec. 3.2, Theorem 2): the path q[0, L) just inserted
// joins the worker's running batch, and once beta - 1 paths run, the oldest
// one leaves it.  A running path ends at a node boundary, so a node is
// either wholly on it or not: a path ending inside an edge splits the edge
// there (splits are not semantic).  The in-progress count of every node of
// the path is raised (one lane per node of the recorded path, else up the
// parent chain), and the leaving path's counts are lowered.  pr holds the
// inserted path and is updated for the split.  Returns KVR_DEV_* bits.
__device__ __forceinline__ uint32_t batch_admit(const Ptrs& P, const PathRef& pr, const int32_t* qs, int32_t L,
                                                int64_t* dbg) {
  St s = load_st(P.hdr);
  const uint32_t ring = P.beta - 1u;
  int32_t e = -1, st = 0;
  int32_t pc = *pr.cnt;
  const bool have_path = pc >= 1 && pc <= kPathMax && pr.start[pc - 1] < L && pr.end[pc - 1] >= L;
  if (have_path) {
    e = pr.node[pc - 1];
    st = pr.start[pc - 1];
  } else {
    // walk down the cached path by first tokens
    const int32_t* ar = arena_of(P, s.arena_sel);
    int32_t x = 0, d = 0;
    while (d < L) {
      const int32_t c = child_find(ar, P.nodes[x], qs[d]);
      if (c <= 0 || (uint32_t)c >= s.hwm) {
        KVR_FAIL_CHECK(s, 20, x, d, L);
        goto fail;
      }
      const int32_t len = P.nodes[c].len;
      if (len <= 0) {
        KVR_FAIL_CHECK(s, 20, c, d, len);
        goto fail;
      }
      if (d + len >= L) {
        e = c;
        st = d;
        break;
      }
      d += len;
      x = c;
    }
  }
  if (e <= 0) {
    KVR_FAIL_CHECK(s, 20, e, L, 0);
    goto fail;
  }
  {
    const int32_t elen = P.nodes[e].len;
    if (st + elen > L) {  // the path ends inside the edge of e: split it there
      const int32_t hd = split_node(P, s, e, L - st);
      if (hd < 0) goto fail;
      wave_mem_sync();
      if (have_path && lane_id() == 0) {
        pr.node[pc - 1] = hd;
        pr.end[pc - 1] = L;
      }
      e = hd;
    }
  }
  // raise the counts of the new running path
  if (have_path && (KVR_WAVE >= kPathMax || pc <= KVR_WAVE)) {
    for (int32_t k = lane_id(); k < pc; k += KVR_WAVE) {
      const int32_t x = (k == pc - 1) ? e : pr.node[k];
      P.pin[x] = P.pin[x] + 1;
    }
  } else {
    int32_t x = e;
    for (uint32_t guard = 0; x > 0; ++guard) {
      if (guard > P.NC || (uint32_t)x >= s.hwm) {
        KVR_FAIL_CHECK(s, 21, x, guard, 1);
        goto fail;
      }
      const int32_t par = P.nodes[x].parent;
      if (lane_id() == 0) P.pin[x] = P.pin[x] + 1;
      x = par;
    }
  }
  wave_mem_sync();
  // the ring of end nodes: push e, release the oldest once beta - 1 run
  {
    WorkerHdr* w = P.hdr;
    const uint32_t head = w->run_head, cnt = w->run_count;
    if (cnt < ring) {
      uint32_t slot = head + cnt;
      if (slot >= ring) slot -= ring;
      if (lane_id() == 0) {
        P.run[slot] = e;
        w->run_count = cnt + 1;
      }
    } else {
      const int32_t old = P.run[head];
      if (lane_id() == 0) {
        P.run[head] = e;
        w->run_head = head + 1 == ring ? 0u : head + 1;
      }
      if (!unpin_chain(P, s, old)) goto fail;
    }
  }
  store_st(P.hdr, s);
  wave_mem_sync();
  return 0;
fail:
  if (lane_id() == 0) *pr.cnt = kPathMax + 1;
  store_st(P.hdr, s);
  if (dbg) {
    dbg[0] = s.dbg_check;
    dbg[1] = s.dbg_val[0];
    dbg[2] = s.dbg_val[1];
    dbg[3] = s.dbg_val[2];
  }
  return s.err ? s.err : (uint32_t)KVR_DEV_INTERNAL;
}

// The rank in the leaf list of the leaf the insertion of q (h cached tokens,
// h < L) creates in the routed worker's cache, for the insertion wave, on
// the tree before the insertion: from the recorded match path of q, when
// that match ends at a node boundary (an edge split would change what this
// reads).  Publishes *rank and sets *ready to 1, or to 2 without a rank.
__device__ __forceinline__ void rank_for_insertion(const Ptrs& P, const PathRef& pr, const int32_t* qs, int32_t h,
                                                   int32_t* rank, uint32_t* ready) {
  int32_t pos = -1;
  const int32_t pc = *pr.cnt;
  if (pc <= kPathMax) {
    int32_t last = 0, cov = 0, len = 0;
    bool ok = true;
    if (h > 0) {
      int32_t e = pc - 1;
      while (e > 0 && pr.start[e] >= h) --e;
      ok = pc > 0 && pr.start[e] < h && pr.end[e] >= h;
      if (ok) {
        last = pr.node[e];
        cov = h - pr.start[e];
        len = pr.end[e] - pr.start[e];
      }
    }
    if (ok && cov == len) {
      const St s = load_st(P.hdr);
      pos = new_leaf_rank(P, s, arena_of(P, s.arena_sel), last, cov, len, qs[h]);
    }
  }
  if (lane_id() == 0) {
    *rank = pos;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __hip_atomic_store(ready, pos >= 0 ? 1u : 2u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
}

// ---------------------------------------------------------------- matching

// ---------------------------------------------------------------- L-LRU

// L-LRU (Sec. 3.2): every access stamps the tokens of its path with the
// global query index; a miss in a full cache evicts the leaf token accessed
// least recently.  One query's path holds at most one leaf token, so no two
// leaf tokens share a stamp and the stamp alone orders them.  Along an edge
// the stamps never increase with depth (an access covers a prefix), so once
// a leaf's tail token is the least recent, the tokens above it with the same
// stamp follow it in the eviction order: they go as one segment.

// Index in the leaf list of the leaf whose last token has the oldest stamp,
// skipping node `excl` and the running batch's nodes; -1 if there is none.
__device__ __forceinline__ int32_t lru_pick(const Ptrs& P, const St& s, const int32_t* st, int32_t excl) {
  constexpr int kUnroll = 4;
  uint64_t best = ~0ull;  // (stamp << 32) | list index
  for (uint32_t b = 0; b < s.nleaves; b += kUnroll * KVR_WAVE) {
    int32_t id[kUnroll];
#pragma unroll
    for (int v = 0; v < kUnroll; ++v) {
      const uint32_t k = b + (uint32_t)(v * KVR_WAVE) + (uint32_t)lane_id();
      id[v] = k < s.nleaves ? P.leaf[k] : -1;
      if (id[v] == excl || (uint32_t)id[v] >= s.hwm) id[v] = -1;
    }
    NodeRec nd[kUnroll];
#pragma unroll
    for (int v = 0; v < kUnroll; ++v)
      if (id[v] > 0) {
        nd[v] = P.nodes[id[v]];
        if (pinned(P, id[v])) id[v] = -1;  // on a running path
      }
#pragma unroll
    for (int v = 0; v < kUnroll; ++v) {
      const uint32_t k = b + (uint32_t)(v * KVR_WAVE) + (uint32_t)lane_id();
      if (id[v] > 0 && nd[v].len > 0) {
        const uint64_t key = ((uint64_t)(uint32_t)st[nd[v].off + (uint32_t)(nd[v].len - 1)] << 32) | k;
        best = key < best ? key : best;
      }
    }
  }
  best = wave_min_u64(best);
  return best == ~0ull ? -1 : (int32_t)(uint32_t)best;
}

// Number of tokens at the end of the edge [off, off+len) stamped j, at most cap.
__device__ __forceinline__ int32_t lru_segment(const int32_t* st, uint32_t off, int32_t len, uint32_t j, int32_t cap) {
  int32_t c = 0;
  while (c < len && c < cap) {
    const int32_t k = len - 1 - c - lane_id();
    const uint64_t m = __ballot(k < 0 || (uint32_t)st[off + (uint32_t)(k < 0 ? 0 : k)] != j);
    if (m) {
      c += first_lane(m);
      break;
    }
    c += KVR_WAVE;
  }
  c = c < len ? c : len;
  return c < cap ? c : cap;
}

// Stamp positions [0, n) of the edge at arena offset off with j.
__device__ __forceinline__ void lru_stamp(int32_t* st, uint32_t off, int32_t n, uint32_t j) {
  for (int32_t k = lane_id(); k < n; k += KVR_WAVE) st[off + (uint32_t)k] = (int32_t)j;
}

// L-LRU insertion of q[0, L) into the worker's cache (the oracle's insertion
// loop with the evictions taken before the loads: loaded tokens and the
// insertion point carry the current stamp, the newest, so they are never the
// least recent leaf and the evicted tokens are the same).  h and pr as for
// rlt_insert.  Returns the KVR_DEV_* error bits.
__device__ __forceinline__ uint32_t lru_insert(const Ptrs& P, const InsertArgs& ia, const int32_t* qs, int32_t L,
                                               int32_t h, const PathRef& pr, int64_t* dbg) {
  St s = load_st(P.hdr);
  const uint32_t B = ia.B;
  const uint32_t jq = (uint32_t)ia.jg;
  int32_t* ar = arena_of(P, s.arena_sel);
  int32_t* st = P.stamp0 + (size_t)s.arena_sel * P.A;
  const int32_t pc = *pr.cnt;
  const bool have_path = pc <= kPathMax;
  bool split = false;
  int32_t a = 0, l = 0, laststart = 0, pe = 0;
  int32_t x = 0, d = 0, last = 0, lastcov = 0;

  // ---- walk the cached part of the path, stamping it
  while (d < h) {
    int32_t c;
    if (have_path) {
      if (pe >= pc || pr.start[pe] != d) {
        KVR_FAIL_CHECK(s, 21, pe, d, h);
        goto fail;
      }
      c = pr.node[pe++];
    } else {
      NodeRec nx = P.nodes[x];
      c = child_find(ar, nx, qs[d]);
    }
    if (c <= 0 || (uint32_t)c >= s.hwm) {
      KVR_FAIL_CHECK(s, 21, c, d, h);
      goto fail;
    }
    const NodeRec nc = P.nodes[c];
    const int32_t cov = nc.len < h - d ? nc.len : h - d;
    if (cov <= 0) {
      KVR_FAIL_CHECK(s, 22, c, nc.len, d);
      goto fail;
    }
    lru_stamp(st, nc.off, cov, jq);
    laststart = d;
    d += cov;
    last = c;
    lastcov = cov;
    x = c;
  }
  wave_mem_sync();

  if (h < L) {
    const int32_t nload = L - h;
    // ---- attachment point: end of `last`, splitting it if needed
    a = last;
    if (h > 0) {
      const NodeRec nl = P.nodes[last];
      if (lastcov < nl.len) {
        a = split_node(P, s, last, lastcov);
        if (a < 0) goto fail;
        split = true;
      }
    }
    // ---- the new leaf holding q[h, L), stamped; it takes the list slot of
    // the attachment point when that was a leaf, else a new one
    int32_t pos = (int32_t)s.nleaves;
    bool replace = false;
    {
      const NodeRec na = P.nodes[a];
      if (a != 0 && na.nchild == 0) {
        pos = arr_find(P.leaf, s.nleaves, a);
        replace = true;
        if (pos < 0) {
          KVR_FAIL_CHECK(s, 23, a, s.nleaves, 0);
          goto fail;
        }
      }
    }
    uint32_t eoff;
    if (!arena_alloc(P, s, (uint32_t)nload, false, eoff)) goto fail;
    ar = arena_of(P, s.arena_sel);
    st = P.stamp0 + (size_t)s.arena_sel * P.A;
    wave_copy(ar + eoff, qs + h, nload);
    lru_stamp(st, eoff, nload, jq);
    wave_mem_sync();
    l = node_alloc(P, s);
    if (l < 0) goto fail;
    {
      NodeRec nl;
      nl.parent = a;
      nl.off = eoff;
      nl.len = nload;
      nl.nchild = 0;
      nl.coff = 0;
      nl.ccap = 0;
      nl.mphase = 0;
      nl.ma = 0;
      node_put(P, l, nl);
    }
    if (!child_add(P, s, a, qs[h], l)) goto fail;
    ar = arena_of(P, s.arena_sel);
    st = P.stamp0 + (size_t)s.arena_sel * P.A;
    if (lane_id() == 0) P.leaf[pos] = l;
    if (!replace) s.nleaves += 1;
    wave_mem_sync();

    // ---- evictions: whole stamp segments of the least recent leaf
    const uint32_t nfree = B - s.size;
    const uint32_t nev = (uint32_t)nload > nfree ? (uint32_t)nload - nfree : 0u;
    uint32_t rem = nev;
    while (rem > 0) {
      const int32_t li = lru_pick(P, s, st, l);
      if (li < 0) {
        KVR_FAIL_CHECK(s, 24, rem, s.nleaves, L);
        goto fail;
      }
      const int32_t v = P.leaf[li];
      const NodeRec nv = P.nodes[v];
      if (nv.nchild != 0 || nv.len <= 0 || nv.parent < 0) {
        KVR_FAIL_CHECK(s, 25, v, nv.nchild, nv.len);
        goto fail;
      }
      const uint32_t jv = (uint32_t)st[nv.off + (uint32_t)(nv.len - 1)];
      const int32_t t = lru_segment(st, nv.off, nv.len, jv, (int32_t)rem);
      if (t <= 0) {
        KVR_FAIL_CHECK(s, 26, v, nv.len, (int64_t)jv);
        goto fail;
      }
      rem -= (uint32_t)t;
      if (t < nv.len) {
        if (lane_id() == 0) P.nodes[v].len = nv.len - t;
      } else {
        // the node empties: drop it; its parent, if now a leaf, takes its slot
        const int32_t pv = nv.parent;
        if (!child_remove(P, s, pv, v)) {
          KVR_FAIL_CHECK(s, 27, v, pv, 0);
          goto fail;
        }
        node_free(P, s, v);
        const NodeRec np = P.nodes[pv];
        if (pv != 0 && np.nchild == 0) {
          if (lane_id() == 0) P.leaf[li] = pv;
        } else {
          const int32_t lastid = P.leaf[s.nleaves - 1];
          if (lane_id() == 0) P.leaf[li] = lastid;
          s.nleaves -= 1;
        }
      }
      wave_mem_sync();
    }
    s.size = s.size + (uint32_t)nload - nev;
    hdr_count(&P.hdr->loads, (uint64_t)nload);
    hdr_count(&P.hdr->evictions, nev);
  }
  store_st(P.hdr, s);
  wave_mem_sync();
  {
    int32_t fc = have_path ? pe : kPathMax + 1;
    if (fc <= kPathMax) {
      if (split) {
        int32_t f1 = fc - 1;
        path_add(pr, f1, a, laststart, laststart + lastcov);
      }
      if (h < L) path_add(pr, fc, l, h, L);
    }
    if (lane_id() == 0) *pr.cnt = fc;
  }
  return 0;
fail:
  if (lane_id() == 0) *pr.cnt = kPathMax + 1;
  store_st(P.hdr, s);
  if (dbg) {
    dbg[0] = s.dbg_check;
    dbg[1] = s.dbg_val[0];
    dbg[2] = s.dbg_val[1];
    dbg[3] = s.dbg_val[2];
  }
  return s.err ? s.err : (uint32_t)KVR_DEV_INTERNAL;
}

// First index k < n with e[k] != q[k] (e in global memory, q in LDS), or
// n.  The edge is read in aligned 16-byte blocks of four tokens, one block
// per lane and KVR_MATCH_UNROLL blocks per lane in flight (up to 2,048
// tokens per round trip on a 64-lane wave).  The first block may start up
// to three tokens before e and the last end up to three after e + n, always
// inside the same aligned 16 bytes; those tokens are not compared.
#ifndef KVR_MATCH_UNROLL
#define KVR_MATCH_UNROLL 8
#endif
template <int kUnroll = KVR_MATCH_UNROLL>
__device__ int32_t first_mismatch(const int32_t* e, const int32_t* q, int32_t n) {
  const uintptr_t ea = reinterpret_cast<uintptr_t>(e);
  const int32_t lead = (int32_t)((ea & 15u) >> 2);
  const int4* base = reinterpret_cast<const int4*>(ea - (uintptr_t)lead * 4u);
  const int32_t nb = (lead + n + 3) >> 2;  // blocks covering e[-lead, n)
  for (int32_t b = 0; b < nb; b += kUnroll * KVR_WAVE) {
    int4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int32_t blk = b + u * KVR_WAVE + lane_id();
      v[u].x = v[u].y = v[u].z = v[u].w = 0;
      if (blk < nb) v[u] = base[blk];
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int32_t blk = b + u * KVR_WAVE + lane_id();
      const int32_t x0 = blk * 4 - lead;  // index into e of v[u].x
      int32_t mm = n;
      if (blk < nb) {
        const int32_t t4[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
        for (int c = 3; c >= 0; --c) {
          const int32_t x = x0 + c;
          if (x >= 0 && x < n && t4[c] != q[x]) mm = x;
        }
      }
      const uint64_t m = __ballot(mm < n);
      if (m) return __builtin_amdgcn_readlane(mm, first_lane(m));
    }
  }
  return n;
}

// Continue matching q[0, L) from inside node x (x = 0: the root), `off`
// tokens into its edge, with d tokens matched so far.  Entries of the nodes
// entered are appended at pc.  Returns h.
template <int kU = KVR_MATCH_UNROLL>
__device__ __forceinline__ int32_t match_from(const Ptrs& P, uint32_t sel, const int32_t* qs, int32_t L, int32_t x, int32_t off,
                              int32_t d, const PathRef& pr, int32_t& pc) {
  const int32_t* ar = arena_of(P, sel);
  if (d >= L) return d;
  // the record of the current node is loaded once and carried down
  NodeRec nx = P.nodes[x];
  if (x != 0 && off < nx.len) {  // the rest of this edge first
    const int32_t rest = nx.len - off;
    const int32_t n = rest < L - d ? rest : L - d;
    const int32_t k = first_mismatch<kU>(ar + nx.off + off, qs + d, n);
    d += k;
    if (k < rest) return d;
  }
  while (d < L) {
    const int32_t c = child_find(ar, nx, qs[d]);
    if (c < 0) break;
    const NodeRec nc = P.nodes[c];
    if (nc.len <= 0) break;  // never true for a consistent tree
    path_add(pr, pc, c, d, d + nc.len);
    const int32_t n = nc.len < L - d ? nc.len : L - d;
    const int32_t k = 1 + first_mismatch<kU>(ar + nc.off + 1, qs + d + 1, n - 1);
    d += k;
    if (k < nc.len) break;
    nx = nc;
  }
  return d;
}

// h = length of the longest prefix of q[0, L) cached in the worker's tree,
// recording the path.
template <int kU = KVR_MATCH_UNROLL>
__device__ __forceinline__ int32_t match_lcp(const Ptrs& P, uint32_t sel, const int32_t* qs, int32_t L,
                                             const PathRef& pr) {
  int32_t pc = 0;
  const int32_t h = match_from<kU>(P, sel, qs, L, 0, 0, 0, pr, pc);
  if (lane_id() == 0) *pr.cnt = pc;
  return h;
}

// h of q_new on a worker whose tree holds the recorded match path of the
// previous query q_old, h_old = h of q_old there, ell = LCP(q_old, q_new).
// Up to depth min(h_old, ell) both walks are the same.  If the old match
// stopped first (h_old < ell) the new one stops at the same point.  Else the
// new one leaves q_old's path at depth ell: inside an edge that the old
// match followed further it stops there; otherwise it continues from that
// point.  The path record is updated to the new match.
template <int kU = KVR_MATCH_UNROLL>
__device__ __forceinline__ int32_t match_incremental(const Ptrs& P, uint32_t sel, const int32_t* qn, int32_t Ln, int32_t h_old,
                                     int32_t ell, const PathRef& pr) {
  int32_t pc = *pr.cnt;
  if (pc > kPathMax || ell == 0) return match_lcp<kU>(P, sel, qn, Ln, pr);
  if (h_old < ell) return h_old;
  // the entry holding depth ell: the last one starting above it
  int32_t e = pc - 1;
  while (e > 0 && pr.start[e] >= ell) --e;
  const int32_t x = pr.node[e], st = pr.start[e], en = pr.end[e];
  if (pc == 0 || st >= ell || en < ell) return match_lcp<kU>(P, sel, qn, Ln, pr);  // inconsistent record
  pc = e + 1;
  int32_t h;
  if (ell == Ln || (ell < en && h_old > ell)) {
    h = ell;
  } else {
    h = match_from<kU>(P, sel, qn, Ln, x, ell - st, ell, pr, pc);
  }
  if (lane_id() == 0) *pr.cnt = pc;
  return h;
}

// match_incremental that reads the worker's active semispace only when it
// walks the tree (the common outcomes need no global memory at all).
template <int kU = KVR_MATCH_UNROLL>
__device__ __forceinline__ int32_t match_incremental_lazy(const Ptrs& P, const int32_t* qn, int32_t Ln, int32_t h_old,
                                                          int32_t ell, const PathRef& pr) {
  int32_t pc = *pr.cnt;
  if (pc > kPathMax || ell == 0) return match_lcp<kU>(P, P.hdr->arena_sel, qn, Ln, pr);
  if (h_old < ell) return h_old;
  int32_t e = pc - 1;
  while (e > 0 && pr.start[e] >= ell) --e;
  const int32_t x = pr.node[e], st = pr.start[e], en = pr.end[e];
  if (pc == 0 || st >= ell || en < ell) return match_lcp<kU>(P, P.hdr->arena_sel, qn, Ln, pr);
  pc = e + 1;
  int32_t h;
  if (ell == Ln || (ell < en && h_old > ell)) {
    h = ell;
  } else {
    h = match_from<kU>(P, P.hdr->arena_sel, qn, Ln, x, ell - st, ell, pr, pc);
  }
  if (lane_id() == 0) *pr.cnt = pc;
  return h;
}

// ---------------------------------------------------------------- LBGR (one lane per worker)

__device__ void online_update(const Consts& C, WorkerHdr* w, const double phi[4], double e) {
  if (C.update == KVR_UPD_NLMS) {
    double ss = phi[0] * phi[0];
    ss = ss + phi[1] * phi[1];
    ss = ss + phi[2] * phi[2];
    ss = ss + phi[3] * phi[3];
    double g = (C.lr * e) / (C.nlms_eps + ss);
    for (int a = 0; a < 4; ++a) w->theta[a] = w->theta[a] + g * phi[a];
  } else if (C.update == KVR_UPD_RLS) {
    double pi[4];
    for (int a = 0; a < 4; ++a) {
      double acc = w->Pm[a * 4 + 0] * phi[0];
      acc = acc + w->Pm[a * 4 + 1] * phi[1];
      acc = acc + w->Pm[a * 4 + 2] * phi[2];
      acc = acc + w->Pm[a * 4 + 3] * phi[3];
      pi[a] = acc;
    }
    double den = phi[0] * pi[0];
    den = den + phi[1] * pi[1];
    den = den + phi[2] * pi[2];
    den = den + phi[3] * pi[3];
    den = C.lr + den;
    double k[4];
    for (int a = 0; a < 4; ++a) k[a] = pi[a] / den;
    for (int a = 0; a < 4; ++a) w->theta[a] = w->theta[a] + k[a] * e;
    for (int a = 0; a < 4; ++a)
      for (int b = 0; b < 4; ++b) w->Pm[a * 4 + b] = (w->Pm[a * 4 + b] - k[a] * pi[b]) / C.lr;
  }
}

// Completions with t_done <= t (FIFO), then decay to t and drain the
// observed-latency backlog.
__device__ __forceinline__ void complete_and_decay(const Consts& C, const Ptrs& P, int64_t t, int64_t tprev) {
  WorkerHdr* w = P.hdr;
  const int64_t dt = C.dt_us;
  double Pl = w->P;
  int64_t tl = w->tl;
  uint32_t head = w->pend_head, cnt = w->pend_count;
  uint64_t done = 0;
  while (cnt > 0) {
    PendRec pr = P.pend[head];
    if (pr.t_done > t) break;
    head = head + 1 == P.PC ? 0u : head + 1;
    cnt -= 1;
    Pl = Pl * pow_int(C.rho, (uint64_t)(pr.t_done / dt - tl / dt));
    tl = pr.t_done;
    double rem = pr.chat * pow_int(C.rho, (uint64_t)(pr.t_done / dt - pr.t_route / dt));
    double np = Pl - rem;
    Pl = np > 0.0 ? np : 0.0;
    double phi[4];
    phi[0] = (double)pr.h * 0.001;
    phi[1] = (double)(pr.L - pr.h) * 0.001;
    phi[2] = pr.x3;
    phi[3] = 1.0;
    double res = w->theta[0] * phi[0];
    res = res + w->theta[1] * phi[1];
    res = res + w->theta[2] * phi[2];
    res = res + w->theta[3] * phi[3];
    double ehat_now = pr.base + res;
    double e_obs = (double)(pr.t_done - pr.t_route) * 1e-6;
    online_update(C, w, phi, e_obs - ehat_now);
    done += 1;
  }
  Pl = Pl * pow_int(C.rho, (uint64_t)(t / dt - tl / dt));
  w->P = Pl;
  w->tl = t;
  w->pend_head = head;
  w->pend_count = cnt;
  w->completions += done;
  int64_t nb = w->Wb - (t - tprev);
  w->Wb = nb > 0 ? nb : 0;
}


// ---------------------------------------------------------------- routing (one thread per worker)

// Output length of query k: the given one, else 4 (the paper's default).
__device__ __forceinline__ int32_t query_out_len(const uint16_t* out_len, uint64_t k) {
  return out_len ? (int32_t)out_len[k] : 4;
}

// The fields of a worker header that scoring and the commit read, loaded
// together by the worker's lane (one round trip for all of them).
struct RouteView {
  double P, theta[4];
  int64_t Wb;
  uint32_t pend_head, pend_count, pending_max, size;
  uint64_t routed, prompt_tokens, hit_tokens, lat_sum_us, lat_max_us;
};

__device__ __forceinline__ RouteView load_view(const WorkerHdr* w) {
  RouteView v;
  v.P = w->P;
  for (int a = 0; a < 4; ++a) v.theta[a] = w->theta[a];
  v.Wb = w->Wb;
  v.pend_head = w->pend_head;
  v.pend_count = w->pend_count;
  v.pending_max = (uint32_t)w->pending_max;
  v.size = w->size;
  v.routed = w->routed;
  v.prompt_tokens = w->prompt_tokens;
  v.hit_tokens = w->hit_tokens;
  v.lat_sum_us = w->lat_sum_us;
  v.lat_max_us = w->lat_max_us;
  return v;
}

// LBGR score of one worker (Eq. LBGR-score with the features of Sec. 4.2
// and the per-1k-token scaling of App. A).  *chat = estimated service time.
__device__ double lbgr_score(const Consts& C, const RouteView& w, int32_t h, int32_t L, double* chat) {
  double x1 = (double)h * 0.001;
  double x2 = (double)(L - h) * 0.001;
  double x3 = w.P;
  double x4 = 1.0;
  double ch = C.alpha_cached * x1 + C.alpha_miss * x2;
  double res = w.theta[0] * x1;
  res = res + w.theta[1] * x2;
  res = res + w.theta[2] * x3;
  res = res + w.theta[3] * x4;
  *chat = ch;
  return (ch + w.P) + res;
}

// Commit a query on its routed worker, whose header fields v holds: add the
// estimated service time to the load estimate (Algorithm 2), advance the
// observed-latency queue and queue the completion record.  hb = the worker's
// true hit (observed latency, hit counter), hf = the hit the router scored
// with (the completion's features; the same unless the router keeps its own
// tree).  Returns KVR_DEV_* bits.
__device__ __forceinline__ uint32_t commit_route(const Consts& C, const Ptrs& P, const RouteView& v, double chat,
                                                 int32_t hb, int32_t hf, int32_t L, int64_t t, int32_t olen) {
  WorkerHdr* w = P.hdr;
  const double base = chat + v.P;
  const double x3 = v.P;
  w->P = v.P + chat;
  const int64_t cost = C.true_cached_us * hb + C.true_miss_us * (int64_t)(L - hb) + C.true_out_us * (int64_t)olen;
  const int64_t e_us = v.Wb + cost;
  w->Wb = v.Wb + cost;
  uint32_t err = 0;
  if (v.pend_count >= P.PC) {
    err |= KVR_DEV_PENDING_FULL;
  } else {
    uint32_t slot = v.pend_head + v.pend_count;
    if (slot >= P.PC) slot -= P.PC;
    PendRec pr;
    pr.t_route = t;
    pr.t_done = t + e_us;
    pr.chat = chat;
    pr.base = base;
    pr.x3 = x3;
    pr.h = hf;
    pr.L = L;
    P.pend[slot] = pr;
    const uint32_t cnt = v.pend_count + 1u;
    w->pend_count = cnt;
    if (cnt > v.pending_max) w->pending_max = cnt;
  }
  w->routed = v.routed + 1u;
  w->prompt_tokens = v.prompt_tokens + (uint64_t)L;
  w->hit_tokens = v.hit_tokens + (uint64_t)hb;
  w->lat_sum_us = v.lat_sum_us + (uint64_t)e_us;
  if ((uint64_t)e_us > v.lat_max_us) w->lat_max_us = (uint64_t)e_us;
  return err;
}

// Empty cache, phase 1, zero load and model (one thread per worker).
__device__ void init_worker(const Ptrs& P, double rls_p0) {
  WorkerHdr h;
  uint8_t* hb = reinterpret_cast<uint8_t*>(&h);
  for (size_t b = 0; b < sizeof(WorkerHdr); ++b) hb[b] = 0;
  h.phase = 1;
  h.hwm = 1;
  h.free_head = -1;
  h.rnode = -1;
  for (int k = 0; k < 16; ++k) h.Pm[k] = (k % 5 == 0) ? rls_p0 : 0.0;
  *P.hdr = h;
  NodeRec root;
  root.parent = -1;
  root.off = 0;
  root.len = 0;
  root.nchild = 0;
  root.coff = 0;
  root.ccap = 0;
  root.mphase = 0;
  root.ma = 0;
  P.nodes[0] = root;
}

// Wave sums and exclusive-or of 64-bit values (butterfly over the lanes).
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  for (int o = 1; o < KVR_WAVE; o <<= 1) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, o, KVR_WAVE);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), o, KVR_WAVE);
    v += ((uint64_t)hi << 32) | lo;
  }
  return v;
}

__device__ __forceinline__ uint64_t wave_xor_u64(uint64_t v) {
  for (int o = 1; o < KVR_WAVE; o <<= 1) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, o, KVR_WAVE);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), o, KVR_WAVE);
    v ^= ((uint64_t)hi << 32) | lo;
  }
  return v;
}

// Final state of one worker (whole wave), with the path-hash digest of the
// cached tokens H(v) = mix64(H(parent) + G*(tok+1)), H(root) = 0.  A
// token's hash needs its parent's, so the tree is walked top-down: P.scratch
// holds a FIFO of (node, hash before its edge), starting with the root.  An
// idle lane takes the next queued node, hashes its edge 16 tokens per round
// (the loads of a round in flight together) and, at the edge's end, appends
// the node's children with the edge's last hash.  Long and short edges so
// share the wave.  Returns false on an inconsistent tree (the counts are
// then partial).
__device__ bool worker_stats(const Ptrs& P, kvr_worker_stats* out, uint64_t* fifo = nullptr, uint64_t fifo_cap = 0) {
  constexpr int kTok = 16;
  const WorkerHdr* h = P.hdr;
  const St s = load_st(h);
  const int32_t* ar = arena_of(P, s.arena_sel);
  // the FIFO (entry e: q[2e] = node, q[2e + 1] = hash before its edge): the
  // worker's scratch region, or the caller's
  uint64_t* q = fifo ? fifo : P.scratch;
  const uint64_t cap = fifo ? fifo_cap : P.NC;
  uint64_t count = 0, dsum = 0, dxor = 0, mcount = 0, msum = 0;
  if (lane_id() == 0) {
    q[0] = 0;
    q[1] = 0;
  }
  wave_mem_sync();
  uint64_t head = 0, tail = 1;  // wave-uniform
  int32_t x = -1, k = 0;
  uint64_t hx = 0;
  NodeRec nd;
  nd.parent = nd.len = nd.nchild = nd.ccap = nd.ma = 0;
  nd.off = nd.coff = nd.mphase = 0;
  bool bad = false, done = false;
  const uint64_t bound = (uint64_t)s.hwm + (uint64_t)s.size + 2u;
  for (uint64_t it = 0; it < bound; ++it) {
    // idle lanes take queued nodes, in lane order
    const uint64_t idle = __ballot(x < 0);
    const uint64_t avail = tail - head;
    if (x < 0) {
      const uint64_t rank = (uint64_t)__popcll(idle & lanemask_lt());
      if (rank < avail) {
        const uint64_t e = head + rank;
        const uint64_t id = q[2 * e];
        hx = q[2 * e + 1];
        k = 0;
        if (id < (uint64_t)s.hwm && id < (uint64_t)P.NC) {
          nd = P.nodes[id];
          x = (int32_t)id;
          if (nd.parent == -2 || nd.len < 0 || (uint64_t)nd.off + (uint64_t)nd.len > P.A || nd.nchild < 0 ||
              (nd.nchild > 0 && (uint64_t)nd.coff + 2ull * (uint64_t)nd.nchild > P.A)) {
            bad = true;
            x = -1;
          }
        } else {
          bad = true;
        }
      }
    }
    const uint64_t nidle = (uint64_t)__popcll(idle);
    head += nidle < avail ? nidle : avail;
    if (__ballot(bad)) break;
    if (!__ballot(x >= 0)) {
      done = true;
      break;
    }
    if (x >= 0) {
      int32_t t[kTok];
#pragma unroll
      for (int c = 0; c < kTok; ++c) t[c] = k + c < nd.len ? ar[nd.off + (uint32_t)(k + c)] : 0;
#pragma unroll
      for (int c = 0; c < kTok; ++c) {
        if (k + c < nd.len) {
          hx = mix64(hx + 0x9E3779B97F4A7C15ull * (uint64_t)(int64_t)(t[c] + 1));
          count += 1;
          dsum += hx;
          dxor ^= hx;
          if (is_marked(s, nd, x, k + c)) {
            mcount += 1;
            msum += hx;
          }
        }
      }
      k += kTok;
    }
    // lanes at the end of their edge queue its children
    const bool fin = x >= 0 && k >= nd.len;
    const uint32_t nc = fin ? (uint32_t)nd.nchild : 0u;
    const uint32_t incl = wave_inclusive_sum(nc);
    const uint64_t total = (uint32_t)__builtin_amdgcn_readlane((int)incl, KVR_WAVE - 1);
    if (tail + total > cap) {
      bad = true;
      break;
    }
    if (fin) {
      const uint64_t e0 = tail + incl - nc;
      for (uint32_t c = 0; c < nc; ++c) {
        q[2 * (e0 + c)] = (uint64_t)(uint32_t)ar[nd.coff + 2u * c + 1u];
        q[2 * (e0 + c) + 1] = hx;
      }
      x = -1;
    }
    tail += total;
    wave_mem_sync();  // the queued entries before other lanes read them
  }
  count = wave_sum_u64(count);
  dsum = wave_sum_u64(dsum);
  dxor = wave_xor_u64(dxor);
  mcount = wave_sum_u64(mcount);
  msum = wave_sum_u64(msum);
  if (lane_id() == 0) {
    kvr_worker_stats o;
    o.routed = h->routed;
    o.prompt_tokens = h->prompt_tokens;
    o.hit_tokens = h->hit_tokens;
    o.matched_tokens = h->matched_tokens;
    o.loads = h->loads;
    o.evictions = h->evictions;
    o.phase = h->phase;
    o.cnt = h->cnt;
    o.forced_resets = h->forced_resets;
    o.resident = count;
    o.digest_sum = dsum;
    o.digest_xor = dxor;
    o.marked_count = mcount;
    o.marked_sum = msum;
    o.completions = h->completions;
    o.pending_depth = h->pend_count;
    o.pending_max = h->pending_max;
    o.latency_sum_us = h->lat_sum_us;
    o.latency_max_us = h->lat_max_us;
    o.backlog_us = h->Wb;
    o.last_decay_us = h->tl;
    o.load_est = h->P;
    for (int a = 0; a < 4; ++a) o.theta[a] = h->theta[a];
    o.nodes = h->nnodes;
    o.gc_runs = h->gc_runs;
    o.router_resident = o.router_digest_sum = o.router_digest_xor = o.router_evictions = 0;
    *out = o;
  }
  return done && !bad;
}

}  // namespace kvr

#endif  // KVR_CORE_H
