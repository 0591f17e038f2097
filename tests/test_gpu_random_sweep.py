"""Randomized sweep of the HIP path against the CPU oracle, through the C
ABI, on an MI355X: many small seeded cases that vary every shape parameter
at once (workers 1..64, cache budgets of one to four longest queries, long
queries whose maximum length leaves little LDS, so that candidates are not
staged and draw words are partly computed by the inserting wave, replica
counts, transport batches) and the modes (eviction policy, router,
continuous batching, approximate router tree).  Bit-exact as in the other
parity tests."""
import numpy as np
import pytest

import paper_2601_18999_amd as K
from gpu_helpers import assert_parity, gpu_run, note
from workload import generate, small_spec

pytestmark = pytest.mark.gpu

EVICT = {"rlt": K.KVR_EVICT_RLT, "lru": K.KVR_EVICT_LRU}
ROUTER = {"lbgr": K.KVR_ROUTE_LBGR, "random": K.KVR_ROUTE_RANDOM, "round_robin": K.KVR_ROUTE_ROUND_ROBIN,
          "cache_aware": K.KVR_ROUTE_CACHE_AWARE}


def make_case(rng, case):
    W = int(rng.choice([1, 2, 3, 7, 16, 33, 64]))
    long_q = case % 4 == 3
    n = int(rng.integers(50, 150 if long_q else 400))
    plen = int(rng.integers(2, 6000 if long_q else 300))
    sp = small_spec(n=n, groups=int(rng.integers(1, 12)), prefix_len=(1, plen),
                    suffix_len=(1, int(rng.integers(2, 1500 if long_q else 200))), vocab=int(rng.integers(2, 50)),
                    seed=int(rng.integers(1 << 30)))
    s = generate(sp)
    evict = ["rlt", "lru"][int(rng.integers(0, 2)) if case % 3 else 0]
    router = str(rng.choice(["lbgr", "lbgr", "cache_aware", "random", "round_robin"]))
    beta = int(rng.choice([1, 1, 1, 2, 4]))
    B = int(rng.integers(beta * s.max_len, 4 * beta * s.max_len + 2))
    maxL = min(16384, B // beta) if long_q else int(rng.choice([s.max_len, B // beta]))
    rt = int(rng.integers(0, 4) == 0)
    RB = int(rng.integers(maxL, 3 * maxL + 2)) if rt else 0
    R = int(rng.integers(1, 5))
    batch = int(rng.choice([0, 1, 7, 64]))
    return s, dict(W=W, B=B, maxL=maxL, evict=evict, router=router, beta=beta, rt=rt, RB=RB, R=R, batch=batch)


@pytest.mark.parametrize("seed", [101, 202, 303])
def test_random_cases_match_the_oracle(seed):
    rng = np.random.default_rng(seed)
    for case in range(100):
        s, c = make_case(rng, case)
        note(f"seed {seed} case {case}: {c} max_len={s.max_len} n={s.n}")
        extra = dict(batch_size=c["beta"]) if c["beta"] > 1 else {}
        if c["rt"]:
            extra.update(router_tree=1, router_tree_tokens=c["RB"])
        res, stats = gpu_run(s, c["R"], c["W"], c["B"], batch=c["batch"], max_len=c["maxL"],
                             evict=EVICT[c["evict"]], router=ROUTER[c["router"]], **extra)
        assert_parity(s, res, stats, c["W"], c["B"], range(c["R"]), evict=c["evict"], router=c["router"], **extra)


@pytest.mark.parametrize("seed", [4041])
def test_random_wide_cases_match_the_oracle(seed):
    """As above, with every other case given 17 to 48 workers: the pipelined
    kernel's 12-wave form under the same variety of shapes."""
    rng = np.random.default_rng(seed)
    for case in range(100):
        s, c = make_case(rng, case)
        if case % 2 == 0:
            c["W"] = int(rng.choice([17, 20, 24, 32, 40, 48]))
        note(f"wide seed {seed} case {case}: {c} max_len={s.max_len} n={s.n}")
        extra = dict(batch_size=c["beta"]) if c["beta"] > 1 else {}
        if c["rt"]:
            extra.update(router_tree=1, router_tree_tokens=c["RB"])
        res, stats = gpu_run(s, c["R"], c["W"], c["B"], batch=c["batch"], max_len=c["maxL"],
                             evict=EVICT[c["evict"]], router=ROUTER[c["router"]], **extra)
        assert_parity(s, res, stats, c["W"], c["B"], range(c["R"]), evict=c["evict"], router=c["router"], **extra)
