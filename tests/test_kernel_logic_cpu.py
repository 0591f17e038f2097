"""The step kernel's per-wave logic (paper_2601_18999_amd/csrc/kvr_core.h),
compiled for one lane with g++ and replayed on the CPU, against the oracle:
compressed tree, interval marks, ordered candidate list and the copying
collector must reproduce the per-token definition exactly."""
import numpy as np
import pytest

import emul_kernel as E
from oracle import oracle as O
from workload import PRESETS, generate, small_spec
from streams import random_response_stream


ROUTERS = {"lbgr": 0, "random": 1, "round_robin": 2, "cache_aware": 3}


def _compare(s, R, W, B, update="nlms", seed=0, ucap=8192, evict="rlt", router="lbgr", **cfg):
    e = E.run(s, R, W, B, update={"nlms": 0, "rls": 1, "none": 2}[update], seed=seed, ucap=ucap,
              evict={"rlt": 0, "lru": 1}[evict], router=ROUTERS[router], **cfg)
    assert e["rc"] == 0
    for r in range(R):
        o = O.run(s, W, B, replica=r, all_hits=True, update=update, seed=seed, evict=evict, router=router,
                  **{k: v for k, v in cfg.items() if k.startswith("ca_") or k in ("cache_responses", "batch_size", "router_tree", "router_tree_tokens")})
        np.testing.assert_array_equal(e["route"][r], o["route"])
        np.testing.assert_array_equal(e["all_hits"][r], o["all_hits"])
        for i in range(W):
            g, c = e["workers"][r][i], o["workers"][i]
            assert {k: g[k] for k in c} == c, (r, i)
    return e


@pytest.mark.parametrize("block", range(4))
def test_random_instances(block):
    rng = np.random.default_rng(77 + block)
    for case in range(40):
        vocab = int(rng.integers(2, 12))
        sp = small_spec(n=int(rng.integers(20, 160)), groups=int(rng.integers(1, 8)),
                        prefix_len=(1, int(rng.integers(2, 30))), suffix_len=(1, int(rng.integers(2, 20))),
                        vocab=vocab, seed=1000 * block + case)
        s = generate(sp)
        W = int(rng.integers(1, 5))
        B = int(max(s.max_len, rng.integers(2, 150)))
        _compare(s, 2, W, B, update=["nlms", "rls", "none"][case % 3], seed=case)


def test_pipelined_order_takes_both_branches_of_the_early_match():
    """The pipelined kernel matches the next query on the routed worker
    before the evictions; that match is exact when it stays on the inserted
    path, otherwise it is taken again after them.  On small vocabularies both
    happen often; the replay checks every early match that it keeps against
    the post-eviction one, and the whole run against the oracle."""
    unsafe = steps = 0
    rng = np.random.default_rng(5)
    for case in range(30):
        s = generate(small_spec(n=200, groups=int(rng.integers(2, 8)), prefix_len=(2, 30), suffix_len=(1, 20),
                                vocab=int(rng.integers(2, 8)), seed=300 + case))
        e = _compare(s, 2, int(rng.integers(1, 5)), int(max(s.max_len, rng.integers(20, 120))), seed=case)
        unsafe += e["pipe_unsafe"]
        steps += e["pipe_steps"]
    assert steps > 1000 and 0 < unsafe < steps, (unsafe, steps)


def test_collector_stress():
    s = generate(small_spec(n=400, groups=6, prefix_len=(10, 60), suffix_len=(5, 40), vocab=30))
    B = 300
    e = _compare(s, 2, 3, B, arena_words=B + 2 * s.max_len + 64)
    assert sum(w["gc_runs"] for rr in e["workers"] for w in rr) > 50


@pytest.mark.parametrize("cfg", [1, 2])
def test_presets(cfg):
    p = PRESETS[cfg]
    s = generate(p["stream"])
    if cfg == 2:
        s = s.head(4000)
    _compare(s, 2, p["W"], p["B"])


def test_tiny_caches_from_the_exact_enumeration_cases():
    """Caches of 4-6 tokens: the node table must hold the transient split
    head and new leaf of an insertion into a full cache."""
    from test_oracle_pins import EXACT_CASES
    for B, queries in EXACT_CASES:
        s = generate({"kind": "paths", "paths": [list(q) for q in queries],
                      "order": list(range(len(queries)))})
        _compare(s, 64, 1, B)


@pytest.mark.parametrize("ucap", [0, 3, 8])
def test_candidate_staging_capacity(ucap):
    """U staged in LDS, in global memory, or switching between the two as it
    grows past the staging capacity: the same run every time."""
    rng = np.random.default_rng(900 + ucap)
    for case in range(25):
        sp = small_spec(n=int(rng.integers(40, 160)), groups=int(rng.integers(2, 9)),
                        prefix_len=(1, 25), suffix_len=(1, 15), vocab=int(rng.integers(2, 9)), seed=case)
        s = generate(sp)
        W = int(rng.integers(1, 4))
        B = int(max(s.max_len, rng.integers(10, 120)))
        _compare(s, 2, W, B, ucap=ucap, seed=case)


def test_draw_index_from_high_half():
    """The eviction blocks index U with floor(r * |U| / 2^64) from the high
    32 bits of r when they decide it, and from the whole word otherwise: the
    result must equal the full product for every word, including words whose
    low half carries into the index."""
    lib = E.lib()
    rng = np.random.default_rng(77)
    M = (1 << 64) - 1
    for n in [1, 2, 3, 7, 96, 203, 4096, 8191, 262147, (1 << 31) + 11]:
        words = [int(x) for x in rng.integers(0, 2**63, size=300, dtype=np.uint64)] + [0, M, 1 << 63]
        # words whose high half puts r_hi * n just below a multiple of 2^32,
        # with the largest low half: the carry case
        for m in range(1, 40):
            r_hi = ((m << 32) - 1) // n
            for lo in (0, 1, (1 << 31), (1 << 32) - 1):
                w = ((r_hi & 0xFFFFFFFF) << 32) | lo
                words.append(w)
        decided = 0
        for w in words:
            assert lib.emul_draw_index(w, n) == (w * n) >> 64, (hex(w), n)
            decided += lib.emul_draw_index_decided(w, n)
        if n <= 8192:
            assert decided >= 300  # the random words are (almost surely) all decided


@pytest.mark.parametrize("block", range(3))
def test_lru_random_instances(block):
    """L-LRU on the compressed tree (stamp segments, unordered leaf list)
    against the oracle's per-token L-LRU."""
    rng = np.random.default_rng(500 + block)
    for case in range(40):
        vocab = int(rng.integers(2, 12))
        sp = small_spec(n=int(rng.integers(20, 160)), groups=int(rng.integers(1, 8)),
                        prefix_len=(1, int(rng.integers(2, 30))), suffix_len=(1, int(rng.integers(2, 20))),
                        vocab=vocab, seed=3000 * block + case)
        s = generate(sp)
        W = int(rng.integers(1, 5))
        B = int(max(s.max_len, rng.integers(2, 150)))
        e = _compare(s, 2, W, B, update=["nlms", "rls", "none"][case % 3], seed=case, evict="lru")
        # no randomness: every replica is the same
        np.testing.assert_array_equal(e["route"][0], e["route"][1])


def test_lru_collector_and_presets():
    s = generate(small_spec(n=400, groups=6, prefix_len=(10, 70), suffix_len=(5, 50), vocab=30))
    W, B = 3, 320
    e = _compare(s, 1, W, B, evict="lru", arena_words=B + 2 * s.max_len + 100)
    assert sum(w["gc_runs"] for w in e["workers"][0]) > 20
    p = PRESETS[2]
    _compare(generate(p["stream"]).head(3000), 1, p["W"], p["B"], evict="lru")


@pytest.mark.parametrize("router", ["random", "round_robin", "cache_aware"])
@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_baseline_routers(router, evict):
    rng = np.random.default_rng(40 + len(router) + (evict == "lru"))
    for case in range(15):
        sp = small_spec(n=int(rng.integers(40, 200)), groups=int(rng.integers(1, 8)),
                        prefix_len=(1, int(rng.integers(2, 40))), suffix_len=(1, int(rng.integers(2, 20))),
                        vocab=int(rng.integers(2, 12)), seed=7000 + case)
        s = generate(sp)
        s.arrival_us = np.cumsum(rng.integers(1, 3000, size=s.n)).astype(np.int64)  # loads build up
        W = int(rng.integers(1, 6))
        B = int(max(s.max_len, rng.integers(2, 150)))
        _compare(s, 2, W, B, seed=case, evict=evict, router=router, ca_balance_abs=int(rng.integers(0, 6)))


@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_cached_responses_random_paths(evict):
    """Complete paths q || a (Sec. 3.2): matches and scores on the prompt,
    insertion of the whole path, continued into a cached response whenever
    the whole prompt hits."""
    rng = np.random.default_rng(31 + (evict == "lru"))
    full_prompt_hits = 0
    for case in range(60):
        B = int(rng.integers(6, 60))
        s = random_response_stream(rng, int(rng.integers(10, 120)), int(rng.integers(2, 5)), 12, 4, B)
        W = int(rng.integers(1, 4))
        e = _compare(s, 2, W, B, update=["nlms", "rls", "none"][case % 3], seed=case, evict=evict,
                     cache_responses=1)
        prompts = s.lengths - s.out_len.astype(np.int64)
        full_prompt_hits += int((e["hits"][0] == prompts).sum())
    assert full_prompt_hits > 100


@pytest.mark.parametrize("router", ["lbgr", "cache_aware"])
def test_cached_responses_multiturn_sessions(router):
    """Multi-turn sessions whose responses are part of the next turn's
    prompt, under eviction pressure."""
    sp = {"kind": "sessions", "n_sessions": 60, "turns": (1, 6), "start_len": 20, "ext_len": (2, 30),
          "vocab": 50, "responses": True, "out_len": 6, "turn_rate": 2.0, "seed": 5}
    s = generate(sp)
    W, B = 3, 600
    e = _compare(s, 2, W, B, router=router, cache_responses=1)
    assert sum(w["evictions"] for w in e["workers"][0]) > 0


def test_cached_responses_collector():
    rng = np.random.default_rng(8)
    s = random_response_stream(rng, 400, 3, 40, 12, 200)
    B = 200
    e = _compare(s, 2, 2, B, cache_responses=1, arena_words=B + 2 * s.max_len + 64)
    assert sum(w["gc_runs"] for rr in e["workers"] for w in rr) > 10


@pytest.mark.parametrize("evict", ["rlt", "lru"])
@pytest.mark.parametrize("block", range(2))
def test_continuous_batching_random_instances(evict, block):
    """Continuous batching (Sec. 3.2, Theorem 2): the running batch's nodes
    are excluded from eviction, ends of running paths split their edges, and
    a released unmarked leaf makes U be rebuilt; against the oracle's
    per-token pin counts."""
    rng = np.random.default_rng(123 + block + 10 * (evict == "lru"))
    evicted = 0
    for case in range(40):
        beta = int(rng.integers(2, 7))
        sp = small_spec(n=int(rng.integers(30, 200)), groups=int(rng.integers(1, 8)),
                        prefix_len=(1, int(rng.integers(2, 20))), suffix_len=(1, int(rng.integers(2, 12))),
                        vocab=int(rng.integers(2, 10)), seed=500 * block + case)
        s = generate(sp)
        W = int(rng.integers(1, 4))
        B = int(max(beta * s.max_len, rng.integers(2, 150)))
        e = _compare(s, 2, W, B, update=["nlms", "rls", "none"][case % 3], seed=case, evict=evict,
                     batch_size=beta, ucap=[0, 8192][case % 2])
        evicted += sum(w["evictions"] for w in e["workers"][0])
    assert evicted > 1000


def test_continuous_batching_with_responses_routers_and_collector():
    rng = np.random.default_rng(99)
    gc = 0
    for case in range(20):
        beta = int(rng.integers(2, 5))
        B = int(rng.integers(40, 200))
        s = random_response_stream(rng, int(rng.integers(50, 200)), int(rng.integers(2, 5)),
                                   max(1, B // beta - 6), 6, B // beta)
        W = int(rng.integers(1, 4))
        router = ["lbgr", "random", "round_robin", "cache_aware"][case % 4]
        # small vocabularies branch at almost every token: child arrays need
        # about B more words than the edges
        e = _compare(s, 2, W, B, seed=case, batch_size=beta, cache_responses=1, router=router,
                     evict=["rlt", "lru"][case % 2], arena_words=2 * B + 2 * s.max_len + 64)
        gc += sum(w["gc_runs"] for w in e["workers"][0])
    assert gc > 20


@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_router_tree_random_instances(evict):
    """The approximate router (App. E): a second, L-LRU tree per worker holds
    the routed prompts; the router scores with its matches, the commit and
    the hit counts take the cache's own."""
    rng = np.random.default_rng(808 + (evict == "lru"))
    for case in range(40):
        sp = small_spec(n=int(rng.integers(30, 200)), groups=int(rng.integers(1, 8)),
                        prefix_len=(1, int(rng.integers(2, 25))), suffix_len=(1, int(rng.integers(2, 15))),
                        vocab=int(rng.integers(2, 10)), seed=900 + case)
        s = generate(sp)
        W = int(rng.integers(1, 5))
        B = int(max(s.max_len, rng.integers(2, 150)))
        RB = int(max(s.max_len, rng.integers(2, 200)))
        router = ["lbgr", "cache_aware"][case % 2]
        e = _compare(s, 2, W, B, update=["nlms", "rls", "none"][case % 3], seed=case, evict=evict, router=router,
                     router_tree=1, router_tree_tokens=RB, ucap=[0, 8192][case % 2])
        assert all(w["router_resident"] <= RB for w in e["workers"][0])


def test_router_tree_with_responses_batching_and_collector():
    rng = np.random.default_rng(77)
    gc = 0
    for case in range(16):
        beta = int(rng.integers(1, 4))
        B = int(rng.integers(40, 200))
        s = random_response_stream(rng, int(rng.integers(50, 200)), int(rng.integers(2, 5)),
                                   max(1, B // beta - 6), 6, B // beta)
        W = int(rng.integers(1, 4))
        RB = int(max(s.max_len, rng.integers(10, 100)))
        e = _compare(s, 2, W, B, seed=case, batch_size=beta, cache_responses=1, router_tree=1,
                     router_tree_tokens=RB, evict=["rlt", "lru"][case % 2], arena_words=2 * B + 2 * s.max_len + 64)
        gc += sum(w["gc_runs"] for w in e["workers"][0])
    assert gc > 0
