"""HIP path vs the CPU oracle, through the C ABI, on an MI355X.

Bit-exact on routes, every h_ij, hit counts, cache digests (path hashes of
every cached token), marking state and counters; the load estimate and the
residual model to 1e-9 relative.  Sizes are ones the oracle finishes in
seconds but that still cover many 64-token tiles, ragged tails, phase
resets, forced resets and collector runs.
"""
import ctypes
import math

import numpy as np
import pytest

import paper_2601_18999_amd as K
from oracle import oracle as O
from workload import PRESETS, generate, small_spec
from gpu_helpers import assert_parity, gpu_run, note
import spec_model as SM

pytestmark = pytest.mark.gpu


def test_device_present():
    import torch
    assert torch.cuda.is_available()
    note(f"device: {torch.cuda.get_device_name(0)}")
    K.load_library()


@pytest.mark.parametrize("case", range(12))
def test_small_random_parity(case):
    rng = np.random.default_rng(100 + case)
    vocab = int(rng.integers(2, 40))
    sp = small_spec(n=int(rng.integers(60, 400)), groups=int(rng.integers(1, 9)),
                    prefix_len=(1, int(rng.integers(3, 90))), suffix_len=(1, int(rng.integers(2, 70))),
                    vocab=vocab, seed=case)
    s = generate(sp)
    W = int(rng.integers(1, 7))
    B = int(max(s.max_len, rng.integers(2, 600)))
    R = 3
    upd = ["nlms", "rls", "none"][case % 3]
    note(f"case {case}: R={R} W={W} B={B} n={s.n} vocab={vocab} update={upd}")
    res, stats = gpu_run(s, R, W, B, update=upd, seed=case)
    assert_parity(s, res, stats, W, B, range(R), update=upd, seed=case)


def test_collector_under_small_arena():
    s = generate(small_spec(n=500, groups=6, prefix_len=(10, 70), suffix_len=(5, 50), vocab=30))
    W, B, R = 3, 320, 4
    note("collector stress")
    res, stats = gpu_run(s, R, W, B, arena_words=B + 2 * s.max_len + 100)
    assert sum(w["gc_runs"] for rr in stats for w in rr) > 50
    assert_parity(s, res, stats, W, B, range(R))


def test_many_waves_per_replica():
    """W = 24 workers: the 12-wave form of the pipelined kernel (ten helpers,
    several match items each per query)."""
    s = generate(small_spec(n=300, groups=12, prefix_len=(20, 120), suffix_len=(5, 40), vocab=200))
    W, B, R = 24, 500, 3
    res, stats = gpu_run(s, R, W, B)
    assert_parity(s, res, stats, W, B, range(R))


@pytest.mark.parametrize("W", [16, 17, 31])
def test_wave_form_threshold_small_vocab(W):
    """Both sides of the worker count at which the pipelined kernel takes
    its 12-wave form, on a small vocabulary (frequent splits, inexact early
    matches and evictions into shared prefixes)."""
    s = generate(small_spec(n=400, groups=8, prefix_len=(4, 60), suffix_len=(2, 40), vocab=6, seed=W))
    B, R = int(max(s.max_len, 90)), 3
    note(f"wave form threshold: W={W} B={B} n={s.n}")
    res, stats = gpu_run(s, R, W, B, seed=W)
    assert_parity(s, res, stats, W, B, range(R), seed=W)
    assert sum(w["evictions"] for rr in stats for w in rr) > 0


def test_config1_full_all_replicas_ragged_batches():
    p = PRESETS[1]
    s = generate(p["stream"])
    R = 8
    note("config 1, R=8, batches of 333")
    res, stats = gpu_run(s, R, p["W"], p["B"], batch=333)
    assert_parity(s, res, stats, p["W"], p["B"], range(R))


def test_config2_full_sampled_replicas():
    p = PRESETS[2]
    s = generate(p["stream"])
    import time
    t0 = time.time()
    res, stats = gpu_run(s, p["R"], p["W"], p["B"], batch=2500)
    t1 = time.time()
    assert_parity(s, res, stats, p["W"], p["B"], [0, 21, 42, 63])
    note(f"config 2, R=64, n={s.n}: gpu {t1 - t0:.2f}s, oracle x4 {time.time() - t1:.2f}s, "
         f"evictions {sum(w['evictions'] for rr in stats for w in rr)}")


def test_batch_split_invariance_and_determinism():
    s = generate(small_spec(n=400, groups=5, prefix_len=(5, 50), suffix_len=(3, 30), vocab=12))
    W, B, R = 3, 200, 4
    a, sa = gpu_run(s, R, W, B, batch=0)
    b, sb = gpu_run(s, R, W, B, batch=37)
    c, sc = gpu_run(s, R, W, B, batch=1)
    d, sd = gpu_run(s, R, W, B, batch=0)
    for x, sx in ((b, sb), (c, sc), (d, sd)):
        np.testing.assert_array_equal(a["route"], x["route"])
        np.testing.assert_array_equal(a["all_hits"], x["all_hits"])
        assert sa == sx


def test_replicas_differ_only_by_random_key():
    """All replicas see the same stream; with no eviction they are identical."""
    s = generate(small_spec(n=200, groups=4, prefix_len=(5, 30), suffix_len=(3, 20), vocab=9))
    W, R = 3, 5
    res, stats = gpu_run(s, R, W, 10**5)
    for r in range(1, R):
        np.testing.assert_array_equal(res["route"][0], res["route"][r])
        assert stats[0] == stats[r]
    assert sum(w["evictions"] for w in stats[0]) == 0


# ---------------------------------------------------------------- randomised semantics

EXACT_CASES = [
    (5, [(0, 1, 2), (0, 1, 3), (0, 2), (1, 2, 3), (0, 1, 2), (1, 2), (0, 1, 3), (0, 2, 1),
         (1, 2, 3), (0, 1, 2)]),
    (4, [(0, 1), (0, 2), (1, 0), (0, 1, 2), (1, 1), (0, 2), (2,), (0, 1), (1, 0, 1), (0, 2)]),
]


@pytest.mark.parametrize("case", range(len(EXACT_CASES)))
def test_mean_hits_match_exact_enumeration(case):
    B, queries = EXACT_CASES[case]
    exact = SM.expected_hits(queries, B)
    s = generate({"kind": "paths", "paths": [list(q) for q in queries],
                  "order": list(range(len(queries)))})
    R = 20000
    res, _ = gpu_run(s, R, 1, B, all_hits=False)
    assert res["status"] == K.KVR_OK, (res["status"], res["bits"])
    tot = res["hits"].sum(1).astype(float)
    sd = tot.std(ddof=1) / math.sqrt(R)
    assert abs(tot.mean() - float(sum(exact))) < 4 * sd, (tot.mean(), float(sum(exact)), sd)


def test_uniform_tail_miss_probability():
    B, L = 16, 4
    n_t = B - L + 2
    prefix = list(range(100, 100 + L - 1))
    paths = [prefix + [k] for k in range(n_t)]
    rng = np.random.default_rng(4)
    order = [int(x) for x in rng.integers(0, n_t, size=2000)]
    s = generate({"kind": "paths", "paths": paths, "order": order})
    R = 64
    res, _ = gpu_run(s, R, 1, B, all_hits=False)
    assert res["status"] == K.KVR_OK, (res["status"], res["bits"])
    h = res["hits"][:, 500:]
    assert (h >= L - 1).all()
    misses, total = int((h == L - 1).sum()), h.size
    p = 1.0 / n_t
    assert abs(misses - total * p) < 4 * math.sqrt(total * p * (1 - p))


# ---------------------------------------------------------------- error paths

def _sim_for(s, **cfg):
    return K.Simulator(2, 2, 100, max(1, s.max_len), **cfg)


def test_invalid_batches_are_rejected_before_any_state_change():
    import torch
    s = generate(small_spec(n=50, groups=3, prefix_len=(3, 10), suffix_len=(2, 8), vocab=7))
    for kind in ("empty_query", "negative_token", "decreasing_arrival"):
        sim = _sim_for(s)
        ds = sim.upload(s)
        sim.route(ds, 0, 20)
        before = sim.stats()
        bad = generate(small_spec(n=10, groups=2, prefix_len=(3, 10), suffix_len=(2, 8), vocab=7, seed=9))
        if kind == "empty_query":
            bad.offsets = bad.offsets.copy()
            bad.offsets[3] = bad.offsets[2]
        elif kind == "negative_token":
            bad.tokens = bad.tokens.copy()
            bad.tokens[5] = -3
        else:
            bad.arrival_us = np.zeros(bad.n, np.int64)
        dbad = sim.upload(bad)
        sim.route(dbad, 0, bad.n)
        st, bits = sim.check()
        assert st == K.KVR_EINVAL, (kind, st, bits)
        # a stats buffer one entry short is refused before anything is written
        short = (K.KvrWorkerStats * (sim.R * sim.W))()
        assert K.load_library().kvr_stats(ctypes.c_void_p(sim.ctx), None, 0, short,
                                          sim.R * sim.W - 1) == K.KVR_EINVAL
        assert all(short[i].routed == 0 for i in range(sim.R * sim.W))
        rshort = (K.KvrReplicaStats * sim.R)()
        assert K.load_library().kvr_stats(ctypes.c_void_p(sim.ctx), rshort, sim.R - 1, short,
                                          sim.R * sim.W) == K.KVR_EINVAL
        assert all(rshort[i].queries == 0 for i in range(sim.R))
        assert all(short[i].routed == 0 for i in range(sim.R * sim.W))
        after = sim.stats(check=False)
        assert before == after, kind
        with pytest.raises(K.KvrError) as ei:
            sim.route(ds, 20, 5)
        assert ei.value.status == K.KVR_ESTATE
        sim.close()
        torch.cuda.synchronize()


def test_capacity_errors_are_reported():
    s = generate(small_spec(n=200, groups=3, prefix_len=(3, 20), suffix_len=(2, 15), vocab=50))
    s.arrival_us = np.arange(s.n, dtype=np.int64)  # arrivals 1 us apart: completions pile up
    sim = K.Simulator(2, 1, 400, s.max_len, pending_capacity=2)
    sim.run(s)
    st, bits = sim.check()
    assert st == K.KVR_ECAPACITY and bits & 8
    sim.close()
    sim = K.Simulator(2, 2, 400, s.max_len, node_capacity=4)
    sim.run(s)
    st, bits = sim.check()
    assert st == K.KVR_ECAPACITY and bits & 16
    sim.close()


# ---------------------------------------------------------------- L-LRU

LRU = dict(evict=K.KVR_EVICT_LRU)


@pytest.mark.parametrize("case", range(6))
def test_lru_small_random_parity(case):
    rng = np.random.default_rng(700 + case)
    vocab = int(rng.integers(2, 40))
    sp = small_spec(n=int(rng.integers(60, 400)), groups=int(rng.integers(1, 9)),
                    prefix_len=(1, int(rng.integers(3, 90))), suffix_len=(1, int(rng.integers(2, 70))),
                    vocab=vocab, seed=50 + case)
    s = generate(sp)
    W = int(rng.integers(1, 7))
    B = int(max(s.max_len, rng.integers(2, 600)))
    upd = ["nlms", "rls", "none"][case % 3]
    note(f"lru case {case}: W={W} B={B} n={s.n} vocab={vocab} update={upd}")
    res, stats = gpu_run(s, 3, W, B, update=upd, seed=case, **LRU)
    assert_parity(s, res, stats, W, B, range(3), update=upd, seed=case, evict="lru")
    for r in range(1, 3):  # no randomness in L-LRU: the replicas are identical
        np.testing.assert_array_equal(res["route"][0], res["route"][r])


def test_lru_collector_under_small_arena():
    s = generate(small_spec(n=500, groups=6, prefix_len=(10, 70), suffix_len=(5, 50), vocab=30))
    W, B = 3, 320
    res, stats = gpu_run(s, 2, W, B, arena_words=B + 2 * s.max_len + 100, **LRU)
    assert sum(w["gc_runs"] for rr in stats for w in rr) > 20
    assert_parity(s, res, stats, W, B, range(2), evict="lru")


def test_lru_theorem1_worst_case():
    """Theorem 1 construction: B-L+2 paths with a shared (L-1)-token prefix
    queried cyclically; L-LRU misses the last token of every query once
    the cache is full."""
    for B, L in [(10, 4), (33, 7), (64, 2)]:
        n = B - L + 2
        prefix = list(range(1000, 1000 + L - 1))
        paths = [prefix + [k] for k in range(n)]
        s = generate({"kind": "paths", "paths": paths, "order": list(range(n)) * 6})
        res, stats = gpu_run(s, 2, 1, B, **LRU)
        assert res["status"] == K.KVR_OK
        assert (res["hits"][:, n:] == L - 1).all()
        assert stats[0][0]["evictions"] == 6 * n - n + 1


def test_lru_config2_full():
    p = PRESETS[2]
    s = generate(p["stream"])
    res, stats = gpu_run(s, 4, p["W"], p["B"], batch=2500, **LRU)
    assert_parity(s, res, stats, p["W"], p["B"], [0, 3], evict="lru")


# ---------------------------------------------------------------- baseline routers

ROUTER = {"random": K.KVR_ROUTE_RANDOM, "round_robin": K.KVR_ROUTE_ROUND_ROBIN,
          "cache_aware": K.KVR_ROUTE_CACHE_AWARE}


@pytest.mark.parametrize("router", sorted(ROUTER))
@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_baseline_router_parity(router, evict):
    rng = np.random.default_rng(31 + len(router) + 7 * (evict == "lru"))
    for case in range(3):
        sp = small_spec(n=int(rng.integers(100, 400)), groups=int(rng.integers(2, 9)),
                        prefix_len=(1, int(rng.integers(3, 90))), suffix_len=(1, int(rng.integers(2, 40))),
                        vocab=int(rng.integers(2, 40)), seed=900 + case)
        s = generate(sp)
        s.arrival_us = np.cumsum(rng.integers(1, 3000, size=s.n)).astype(np.int64)
        W = int(rng.integers(2, 7))
        B = int(max(s.max_len, rng.integers(20, 600)))
        ab = int(rng.integers(0, 8))
        note(f"{router}/{evict} case {case}: W={W} B={B} n={s.n} balance_abs={ab}")
        res, stats = gpu_run(s, 3, W, B, seed=case, router=ROUTER[router], ca_balance_abs=ab,
                             evict={"rlt": K.KVR_EVICT_RLT, "lru": K.KVR_EVICT_LRU}[evict])
        assert_parity(s, res, stats, W, B, range(3), seed=case, evict=evict, router=router, ca_balance_abs=ab)


# ---------------------------------------------------------------- cached responses

@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_cached_responses_random_parity(evict):
    """Complete paths q || a (Sec. 3.2): the prompt is matched and scored,
    the whole path inserted; small vocabularies make whole-prompt hits that
    continue into cached responses common."""
    from streams import random_response_stream
    rng = np.random.default_rng(61 + (evict == "lru"))
    ev = {"rlt": K.KVR_EVICT_RLT, "lru": K.KVR_EVICT_LRU}[evict]
    for case in range(4):
        B = int(rng.integers(20, 300))
        s = random_response_stream(rng, int(rng.integers(100, 400)), int(rng.integers(2, 6)), 40, 12, B)
        W = int(rng.integers(1, 5))
        upd = ["nlms", "rls", "none"][case % 3]
        note(f"responses/{evict} case {case}: W={W} B={B} n={s.n} update={upd}")
        res, stats = gpu_run(s, 3, W, B, update=upd, seed=case, evict=ev, cache_responses=1)
        assert_parity(s, res, stats, W, B, range(3), update=upd, seed=case, evict=evict, cache_responses=1)
        prompts = s.lengths - s.out_len.astype(np.int64)
        assert (res["hits"] <= prompts[None, :]).all()


@pytest.mark.parametrize("router", ["lbgr", "cache_aware"])
def test_cached_responses_multiturn_parity(router):
    """Multi-turn sessions whose responses are part of the next turn's
    prompt, with the whole path cached, under eviction pressure; batches of
    250 so staging crosses batch boundaries."""
    sp = {"kind": "sessions", "n_sessions": 300, "turns": (1, 8), "start_len": 64, "ext_len": (8, 96),
          "vocab": 32000, "responses": True, "out_len": 4, "turn_rate": 1.0, "seed": 3}
    s = generate(sp)
    W, B, R = 4, 3000, 4
    note(f"responses multiturn/{router}: n={s.n} max_len={s.max_len}")
    res, stats = gpu_run(s, R, W, B, batch=250, router=ROUTER.get(router, K.KVR_ROUTE_LBGR), cache_responses=1)
    assert_parity(s, res, stats, W, B, range(R), router=router, cache_responses=1)
    assert sum(w["evictions"] for w in stats[0]) > B


def test_cached_responses_invalid_path_rejected():
    """A path no longer than its response (an empty prompt) is rejected as a
    whole before any state changes."""
    s = generate(small_spec(n=50, groups=3, prefix_len=(2, 8), suffix_len=(1, 4), vocab=9))
    s.out_len = np.full(s.n, 2, dtype=np.uint16)
    s.out_len[17] = int(s.lengths[17])
    sim = K.Simulator(2, 2, 100, s.max_len, cache_responses=1)
    try:
        ds = sim.upload(s)
        sim.route(ds, 0, s.n)
        st, bits = sim.check()
        assert st == K.KVR_EINVAL and bits & 1, (st, bits)
        assert all(w["routed"] == 0 for rr in sim.stats(check=False) for w in rr)
    finally:
        sim.close()


# ---------------------------------------------------------------- continuous batching

@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_batching_random_parity(evict):
    """Continuous batching (Sec. 3.2, Theorem 2): the beta - 1 paths routed
    to a worker before the current one are never evicted."""
    rng = np.random.default_rng(71 + (evict == "lru"))
    ev = {"rlt": K.KVR_EVICT_RLT, "lru": K.KVR_EVICT_LRU}[evict]
    for case in range(5):
        beta = int(rng.integers(2, 9))
        sp = small_spec(n=int(rng.integers(100, 400)), groups=int(rng.integers(1, 9)),
                        prefix_len=(1, int(rng.integers(3, 40))), suffix_len=(1, int(rng.integers(2, 30))),
                        vocab=int(rng.integers(2, 30)), seed=40 + case)
        s = generate(sp)
        W = int(rng.integers(1, 6))
        B = int(max(beta * s.max_len, rng.integers(2, 600)))
        upd = ["nlms", "rls", "none"][case % 3]
        note(f"batching/{evict} case {case}: beta={beta} W={W} B={B} n={s.n}")
        res, stats = gpu_run(s, 3, W, B, update=upd, seed=case, evict=ev, batch_size=beta)
        assert_parity(s, res, stats, W, B, range(3), update=upd, seed=case, evict=evict, batch_size=beta)


def test_batching_multiturn_with_responses_and_collector():
    sp = {"kind": "sessions", "n_sessions": 300, "turns": (1, 8), "start_len": 32, "ext_len": (8, 48),
          "vocab": 32000, "responses": True, "out_len": 4, "turn_rate": 1.0, "seed": 4}
    s = generate(sp)
    beta = 4
    W, B, R = 4, 4 * s.max_len, 3
    note(f"batching multiturn: n={s.n} max_len={s.max_len} B={B}")
    res, stats = gpu_run(s, R, W, B, batch=200, batch_size=beta, cache_responses=1,
                         arena_words=B + 2 * s.max_len + 64)
    assert_parity(s, res, stats, W, B, range(R), batch_size=beta, cache_responses=1)
    assert sum(w["evictions"] for w in stats[0]) > B
    assert sum(w["gc_runs"] for rr in stats for w in rr) > 0


def test_batching_rejects_a_running_batch_larger_than_the_cache():
    with pytest.raises(K.KvrError):
        K.kvr_workspace_size(K.kvr_config_default(1, 2, 100, 30, batch_size=4))


# ---------------------------------------------------------------- approximate router tree

@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_router_tree_random_parity(evict):
    """The approximate router of App. E: the router's own L-LRU tree per
    worker gives the estimates it scores with; the commit, the observed
    latency and the hit counts take the cache's own match."""
    rng = np.random.default_rng(81 + (evict == "lru"))
    ev = {"rlt": K.KVR_EVICT_RLT, "lru": K.KVR_EVICT_LRU}[evict]
    for case in range(5):
        sp = small_spec(n=int(rng.integers(100, 400)), groups=int(rng.integers(1, 9)),
                        prefix_len=(1, int(rng.integers(3, 60))), suffix_len=(1, int(rng.integers(2, 40))),
                        vocab=int(rng.integers(2, 30)), seed=60 + case)
        s = generate(sp)
        W = int(rng.integers(1, 7))
        B = int(max(s.max_len, rng.integers(2, 600)))
        RB = int(max(s.max_len, rng.integers(2, 800)))
        router = ["lbgr", "cache_aware"][case % 2]
        note(f"router tree/{evict} case {case}: W={W} B={B} RB={RB} n={s.n} router={router}")
        res, stats = gpu_run(s, 3, W, B, seed=case, evict=ev, router=ROUTER.get(router, K.KVR_ROUTE_LBGR),
                             router_tree=1, router_tree_tokens=RB)
        assert_parity(s, res, stats, W, B, range(3), seed=case, evict=evict, router=router, router_tree=1,
                      router_tree_tokens=RB)


def test_router_tree_with_responses_and_batching():
    sp = {"kind": "sessions", "n_sessions": 300, "turns": (1, 8), "start_len": 32, "ext_len": (8, 48),
          "vocab": 32000, "responses": True, "out_len": 4, "turn_rate": 1.0, "seed": 6}
    s = generate(sp)
    W, R, beta = 4, 3, 3
    B = beta * s.max_len
    note(f"router tree multiturn: n={s.n} max_len={s.max_len} B={B}")
    res, stats = gpu_run(s, R, W, B, batch=300, batch_size=beta, cache_responses=1, router_tree=1,
                         router_tree_tokens=B // 2)
    assert_parity(s, res, stats, W, B, range(R), batch_size=beta, cache_responses=1, router_tree=1,
                  router_tree_tokens=B // 2)
    assert sum(w["router_evictions"] for w in stats[0]) > 0


# ---------------------------------------------------------------- the paper's GSP shape

@pytest.mark.parametrize("cfg,evict", [(7, "rlt"), (7, "lru"), (6, "rlt")])
def test_gsp_paper_shape_full_stream(cfg, evict):
    """App. A's GSP (128 groups x 32 queries, lengths 512..8192, prefix ratio
    0.5, 4 workers with 200k-token caches), in the worst-case round-robin
    order and in random order: the whole stream against the oracle."""
    p = PRESETS[cfg]
    s = generate(p["stream"])
    ev = {"rlt": K.KVR_EVICT_RLT, "lru": K.KVR_EVICT_LRU}[evict]
    note(f"{p['name']}/{evict}: n={s.n}")
    res, stats = gpu_run(s, 4, p["W"], p["B"], batch=1024, evict=ev)
    assert_parity(s, res, stats, p["W"], p["B"], [0, 3], evict=evict)
    assert sum(w["evictions"] for w in stats[0]) > 0


# ---------------------------------------------------------------- extreme shapes

def test_largest_worker_count_and_query_length():
    """W = 64 workers (the most a replica holds) and queries up to the largest
    max_query_tokens (16,384): the query buffers leave little LDS, so the
    candidate list stays in global memory and most draw words are computed
    by the inserting wave itself."""
    rng = np.random.default_rng(5)
    groups = [[int(x) for x in rng.integers(0, 1000, size=int(rng.integers(2000, 12000)))] for _ in range(6)]
    paths, order = [], []
    for j in range(40):
        g = groups[int(rng.integers(0, 6))]
        paths.append(g + [int(x) for x in rng.integers(0, 1000, size=int(rng.integers(1, 16384 - len(g) + 1)))])
        order.append(j)
    s = generate({"kind": "paths", "paths": paths, "order": order})
    assert s.max_len <= 16384
    W, B = 64, 40000
    note(f"W={W} B={B} max_len={s.max_len} n={s.n}")
    res, stats = gpu_run(s, 2, W, B, max_len=16384)
    assert_parity(s, res, stats, W, B, range(2))
    s2 = generate({"kind": "paths", "paths": paths[:20], "order": list(range(20)) * 3})
    res, stats = gpu_run(s2, 2, 3, 16384, max_len=16384)
    assert_parity(s2, res, stats, 3, 16384, range(2))
    assert sum(w["evictions"] for w in stats[0]) > 16384


def test_single_token_queries_in_a_one_token_cache():
    """B = 1: every miss evicts the only cached token (the degenerate case of
    Algorithm 1: the marking set resets at every new token)."""
    rng = np.random.default_rng(9)
    paths = [[int(rng.integers(0, 3))] for _ in range(200)]
    s = generate({"kind": "paths", "paths": paths, "order": list(range(200))})
    for evict in ("rlt", "lru"):
        res, stats = gpu_run(s, 3, 2, 1, evict={"rlt": K.KVR_EVICT_RLT, "lru": K.KVR_EVICT_LRU}[evict])
        assert_parity(s, res, stats, 2, 1, range(3), evict=evict)
        assert all(w["resident"] <= 1 for rr in stats for w in rr)


def test_one_query_repeated():
    """The same query over and over: everything after the first is a full
    hit on the worker it went to, and nothing is ever evicted."""
    q = list(range(100, 400))
    s = generate({"kind": "paths", "paths": [q], "order": [0] * 300})
    res, stats = gpu_run(s, 2, 4, 1000, batch=7)
    assert_parity(s, res, stats, 4, 1000, range(2))
    for r in range(2):
        assert (res["all_hits"][r][1:].max(axis=1) == len(q)).all()
        assert sum(w["evictions"] for w in stats[r]) == 0


def test_two_live_contexts_with_different_lds_needs():
    """Two contexts alive at once, the second created with a much shorter
    query buffer (so a smaller LDS footprint) than the first: batches of the
    two interleave, and each context still matches the oracle."""
    rng = np.random.default_rng(13)
    base = [int(x) for x in rng.integers(0, 500, size=6000)]
    long_paths = [base[:int(rng.integers(100, 6000))] + [int(x) for x in rng.integers(0, 500, size=int(
        rng.integers(1, 6000)))] for _ in range(30)]
    s1 = generate({"kind": "paths", "paths": long_paths, "order": [int(x) for x in rng.integers(0, 30, size=60)]})
    s2 = generate({"kind": "paths", "paths": [[int(x) for x in rng.integers(0, 5, size=int(rng.integers(1, 40)))]
                                              for _ in range(50)],
                   "order": [int(x) for x in rng.integers(0, 50, size=300)]})
    W1, B1, W2, B2 = 4, 20000, 3, 120
    note(f"long: max_len={s1.max_len} n={s1.n}; short: max_len={s2.max_len} n={s2.n}")
    a = K.Simulator(2, W1, B1, s1.max_len)
    b = K.Simulator(2, W2, B2, s2.max_len)
    try:
        da, db = a.upload(s1), b.upload(s2)
        outs_a, outs_b = [], []
        for k in range(6):
            outs_a.append(a.route(da, 10 * k, 10, all_hits=True))
            outs_b.append(b.route(db, 50 * k, 50, all_hits=True))
        res = {}
        for sim, outs, key in ((a, outs_a, "a"), (b, outs_b, "b")):
            sim.stream.synchronize()
            st, bits = sim.check()
            res[key] = {"route": np.concatenate([o["route"].cpu().numpy() for o in outs], 1),
                        "hits": np.concatenate([o["hits"].cpu().numpy() for o in outs], 1),
                        "all_hits": np.concatenate([o["all_hits"].cpu().numpy() for o in outs], 1),
                        "status": st, "bits": bits}
            res[key + "_stats"] = sim.stats(check=False)
    finally:
        a.close()
        b.close()
    assert_parity(s1, res["a"], res["a_stats"], W1, B1, range(2))
    assert_parity(s2, res["b"], res["b_stats"], W2, B2, range(2))
    assert sum(w["evictions"] for w in res["a_stats"][0]) > 0
    assert sum(w["evictions"] for w in res["b_stats"][0]) > 0


def test_phase_timers_change_nothing_but_the_ticks():
    """phase_timers = 1 builds the step kernel with the routing wave's
    per-part timers: the same routes, hits and state as the oracle, and
    every part of the step timed (ticks > 0 in total)."""
    s = generate(small_spec(n=300, groups=6, prefix_len=(10, 80), suffix_len=(5, 40), vocab=40, seed=5))
    R, W, B = 4, 3, 300
    sim = K.Simulator(R, W, B, s.max_len, phase_timers=1)
    try:
        res = sim.run(s, batch=97, all_hits=True)
        st, bits = sim.check()
        reps, stats = sim.replica_stats(check=False)
    finally:
        sim.close()
    res["status"], res["bits"] = st, bits
    assert_parity(s, res, stats, W, B, replicas=range(R))
    for rep in reps:
        assert rep["queries"] == s.n
        assert sum(rep["phase_ticks"]) > 0
        # the evictions: on the evicting wave (pipelined kernel) or the routing wave
        assert (rep["phase_ticks"][K.PHASE_NAMES.index("e_evict")] +
                rep["phase_ticks"][K.PHASE_NAMES.index("evict")]) > 0
