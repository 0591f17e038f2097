"""Pins of the CPU oracle against facts it does not compute itself.

* Philox4x64-10 against the generator's published known-answer vector and
  numpy's independent implementation.
* rho^k by square-and-multiply against the exact rational power.
* The whole step against a brute-force model (tests/spec_model.py): caches
  as sets of token tuples, U recomputed and sorted at every draw, random
  words from numpy.
* Cache matching against brute-force LCP over everything routed earlier when
  nothing is evicted.
* The lower-bound construction of Theorem 1 (L-LRU misses every query).
* The uniform-tail construction of Theorem 5 (any policy misses with
  probability exactly 1/(B-L+2) once full).
* Exact expected hits of RLT by enumerating every random choice.
* LBGR closed forms: decayed load, full release on completion, one NLMS
  step, RLS = exponentially weighted ridge least squares.
* Cached responses (complete paths q || a): the brute-force model, the
  reduction to prompt-only caching when every response is empty, and the
  match and cache contents as closed forms over the routed history.
"""
from fractions import Fraction
import math
import os

import numpy as np
import pytest

from oracle import oracle as O
from workload import generate, small_spec
from workload.gen import Stream
import spec_model as SM


def _paths_stream(paths, order, gap_us=83333, out_len=4):
    return generate({"kind": "paths", "paths": paths, "order": order, "gap_us": gap_us,
                     "out_len": out_len})


# ---------------------------------------------------------------------------
# RNG

def _kat_vectors():
    path = os.path.join(os.path.dirname(__file__), "golden", "philox4x64_10_kat.txt")
    with open(path) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                w = [int(x, 16) for x in line.split()]
                yield w[0:4], w[4:6], w[6:10]


def test_philox_known_answer_vectors():
    vecs = list(_kat_vectors())
    assert len(vecs) == 2
    for ctr, key, want in vecs:
        assert [int(x) for x in O.philox4x64_10(ctr, key)] == want
        assert SM.philox_word0(key[0], key[1], tuple(ctr)) == want[0]


def test_philox_matches_numpy():
    rng = np.random.default_rng(7)
    for _ in range(200):
        ctr = [int(x) for x in rng.integers(0, 2**63, size=4)]
        key = [int(x) for x in rng.integers(0, 2**63, size=2)]
        ours = O.philox4x64_10(ctr, key)
        assert int(ours[0]) == SM.philox_word0(key[0], key[1], tuple(ctr))


def test_pow_int_exact_within_rounding():
    rho = 31.0 / 32.0
    exact_rho = Fraction(31, 32)
    # (31/32)^k underflows below the smallest subnormal past k ~ 23600
    assert O.pow_int(rho, 10**7) == 0.0
    for k in [0, 1, 2, 3, 7, 50, 51, 1000, 4097, 20000]:
        got = Fraction(O.pow_int(rho, k))
        if k == 0:
            assert got == 1
            continue
        ex = exact_rho ** k
        # squaring doubles the relative error of the running base, so the
        # error of the product is at most about 2k roundings of 2^-53
        bound = (2 * k + 2 * k.bit_length()) * 2.0 ** -53
        assert abs(float((got - ex) / ex)) <= bound


# ---------------------------------------------------------------------------
# brute-force model equality on random tiny instances

def _random_tiny_stream(rng, n, vocab, max_len, B):
    paths = []
    for _ in range(n):
        L = int(rng.integers(1, min(max_len, B) + 1))
        paths.append([int(x) for x in rng.integers(0, vocab, size=L)])
    gaps = rng.integers(1, 400000, size=n)
    s = _paths_stream(paths, list(range(n)))
    s.arrival_us = np.cumsum(gaps).astype(np.int64)
    s.out_len = rng.integers(0, 6, size=n).astype(np.uint16)
    return s


def _path_hashes(S):
    """Path hash of every cached path (same definition as the oracle's
    statistics: H(v) = mix64(H(parent) + G*(tok+1)), H(root) = 0)."""
    M = (1 << 64) - 1

    def mix(z):
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M
        return z ^ (z >> 31)

    H = {(): 0}
    for x in sorted(S, key=len):
        H[x] = mix((H[x[:-1]] + 0x9E3779B97F4A7C15 * (x[-1] + 1)) & M)
    return H


def _digest_of_set(S, sub=None):
    H = _path_hashes(S)
    sub = S if sub is None else sub
    s = x_ = 0
    for x in sub:
        s = (s + H[x]) & ((1 << 64) - 1)
        x_ ^= H[x]
    return len(sub), s, x_


@pytest.mark.parametrize("evict", ["rlt", "lru"])
@pytest.mark.parametrize("update", ["nlms", "rls", "none"])
def test_oracle_equals_bruteforce_model(evict, update):
    rng = np.random.default_rng(1000 + 7 * len(evict) + len(update))
    for case in range(60):
        W = int(rng.integers(1, 4))
        B = int(rng.integers(2, 13))
        vocab = int(rng.integers(2, 5))
        n = int(rng.integers(5, 30))
        s = _random_tiny_stream(rng, n, vocab, 6, B)
        replica = int(rng.integers(0, 1000))
        kw = dict(evict=evict, update=update, seed=int(rng.integers(0, 2**32)))
        r = O.run(s, W, B, replica=replica, all_hits=True, check=1, **kw)
        assert r["rc"] == 0
        sim, routes, hits, allh = SM.run_spec(s, W, B, replica=replica, **kw)
        np.testing.assert_array_equal(r["route"], routes)
        np.testing.assert_array_equal(r["hits"], hits)
        np.testing.assert_array_equal(r["all_hits"], allh)
        for i in range(W):
            ws, sw = r["workers"][i], sim.w[i]
            assert ws["evictions"] == sw.evictions and ws["loads"] == sw.loads
            cnt, dsum, dxor = _digest_of_set(sw.S)
            assert (ws["resident"], ws["digest_sum"], ws["digest_xor"]) == (cnt, dsum, dxor)
            assert ws["theta"] == sw.theta
            assert ws["load_est"] == sw.P
            if evict == "rlt":
                marked = {x for x in sw.S if sw.mark.get(x, 0) == sw.phase}
                assert ws["marked_count"] == len(marked) == ws["cnt"] == sw.cnt
                assert ws["marked_sum"] == _digest_of_set(sw.S, marked)[1]
                assert ws["phase"] == sw.phase and ws["forced_resets"] == sw.forced


@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_candidate_list_equals_definition(evict):
    """The maintained ordered candidate list (RLT), or the leaf set ordered
    by stamp (L-LRU), gives the same run as recomputing U from its
    definition, or scanning every leaf, at each eviction."""
    rng = np.random.default_rng(5)
    for case in range(12):
        sp = small_spec(n=int(rng.integers(100, 250)), groups=int(rng.integers(2, 8)),
                        prefix_len=(4, 30), suffix_len=(1, 20), vocab=int(rng.integers(3, 40)),
                        seed=case)
        s = generate(sp)
        W = int(rng.integers(1, 4))
        B = int(max(s.max_len, rng.integers(40, 300)))
        a = O.run(s, W, B, replica=case, u_mode=0, all_hits=True, evict=evict)
        b = O.run(s, W, B, replica=case, u_mode=1, all_hits=True, evict=evict)
        np.testing.assert_array_equal(a["route"], b["route"])
        np.testing.assert_array_equal(a["all_hits"], b["all_hits"])
        assert a["workers"] == b["workers"]


# ---------------------------------------------------------------------------
# matching: brute-force LCP when the cache never evicts

def test_match_is_lcp_over_routed_history():
    s = generate(small_spec(n=300, groups=5, prefix_len=(5, 25), suffix_len=(1, 15), vocab=6))
    W, B = 3, 10**6
    r = O.run(s, W, B, all_hits=True)
    assert sum(w["evictions"] for w in r["workers"]) == 0
    qs = [tuple(int(x) for x in s.query(j)) for j in range(s.n)]
    for j in range(s.n):
        for i in range(W):
            best = 0
            for k in range(j):
                if r["route"][k] == i:
                    a, b = qs[j], qs[k]
                    l = 0
                    while l < min(len(a), len(b)) and a[l] == b[l]:
                        l += 1
                    best = max(best, l)
            assert r["all_hits"][j, i] == best


# ---------------------------------------------------------------------------
# constructions from the proofs

def _tail_paths(B, L, vocab_base=100):
    n = B - L + 2
    prefix = list(range(vocab_base, vocab_base + L - 1))
    return [prefix + [k] for k in range(n)], n


def test_lru_worst_case_misses_every_query():
    """Theorem 1 lower bound: B-L+2 paths share an (L-1)-token prefix and
    differ in the last token; queried cyclically, L-LRU misses the tail of
    every query once the cache is full."""
    for B, L in [(10, 4), (33, 7), (64, 2)]:
        paths, n = _tail_paths(B, L)
        order = list(range(n)) * 6
        s = _paths_stream(paths, order)
        r = O.run(s, 1, B, evict="lru", check=1)
        assert r["rc"] == 0
        assert (r["hits"][n:] == L - 1).all()
        assert r["workers"][0]["evictions"] == len(order) - n + 1


def test_uniform_tail_miss_probability():
    """Theorem 5 distribution: tails drawn uniformly from n = B-L+2 paths;
    once full, the cache holds n-1 tails whatever the policy, so each query
    misses with probability exactly 1/n."""
    B, L = 16, 4
    paths, n = _tail_paths(B, L)
    rng = np.random.default_rng(11)
    N, skip = 3000, 500
    for evict, reps in [("lru", 1), ("rlt", 40)]:
        misses = total = 0
        for rep in range(reps):
            order = [int(x) for x in rng.integers(0, n, size=N)]
            s = _paths_stream(paths, order)
            r = O.run(s, 1, B, evict=evict, replica=rep, check=1)
            h = r["hits"][skip:]
            assert (h >= L - 1).all()
            misses += int((h == L - 1).sum())
            total += h.shape[0]
        p = 1.0 / n
        sd = math.sqrt(total * p * (1 - p))
        assert abs(misses - total * p) < 4 * sd, (evict, misses, total * p, sd)


EXACT_CASES = [
    (5, [(0, 1, 2), (0, 1, 3), (0, 2), (1, 2, 3), (0, 1, 2), (1, 2), (0, 1, 3), (0, 2, 1),
         (1, 2, 3), (0, 1, 2)]),
    (4, [(0, 1), (0, 2), (1, 0), (0, 1, 2), (1, 1), (0, 2), (2,), (0, 1), (1, 0, 1), (0, 2)]),
    (6, [(3, 1, 2, 0), (3, 1, 0), (2, 2, 2), (3, 1, 2, 1), (0,), (2, 2, 1), (3, 1, 2, 0),
         (3, 0), (2, 2, 2)]),
]


@pytest.mark.parametrize("case", range(len(EXACT_CASES)))
def test_rlt_mean_hits_match_exact_enumeration(case):
    B, queries = EXACT_CASES[case]
    exact = SM.expected_hits(queries, B)
    s = _paths_stream([list(q) for q in queries], list(range(len(queries))))
    R = 20000
    tot = np.zeros(R)
    per = np.zeros((R, len(queries)))
    for rep in range(R):
        r = O.run(s, 1, B, replica=rep)
        per[rep] = r["hits"]
        tot[rep] = r["hits"].sum()
    ex_tot = float(sum(exact))
    sd = tot.std(ddof=1) / math.sqrt(R)
    assert abs(tot.mean() - ex_tot) < 4 * sd + 1e-12, (tot.mean(), ex_tot, sd)
    # every query's mean too (4.5 sigma: several comparisons)
    for j, e in enumerate(exact):
        sdj = per[:, j].std(ddof=1) / math.sqrt(R)
        assert abs(per[:, j].mean() - float(e)) < 4.5 * sdj + 1e-12


# ---------------------------------------------------------------------------
# LBGR closed forms

def test_decayed_load_and_routing_away():
    """A query routed to worker 0 at t1 leaves load C*rho^(ticks) at t2, so
    an equal query at t2 goes to the idle worker 1."""
    dt = 20000
    L1 = 800  # completes at t1 + 1000*L1 + 40000 us, after t2
    t1, t2 = 30000, 30000 + 37 * dt + 1234
    s = _paths_stream([list(range(1, L1 + 1)), [7000, 8, 9, 10, 11]], [0, 1])
    s.arrival_us = np.array([t1, t2], np.int64)
    r = O.run(s, 2, 1000, update="none")
    assert list(r["route"]) == [0, 1]
    c = L1 * 0.001
    k = t2 // dt - t1 // dt
    got = Fraction(r["workers"][0]["load_est"])
    ex = Fraction(c) * Fraction(31, 32) ** k
    assert abs(float((got - ex) / ex)) < 1e-14
    assert r["workers"][1]["load_est"] == 5 * 0.001


def test_release_returns_load_to_zero():
    """After its completion a query's remaining share is released, so a
    lone query leaves no load and the next query ties and goes to worker 0."""
    L = 20
    s = _paths_stream([list(range(L)), list(range(100, 100 + L))], [0, 1])
    done = 1000 * L + 10000 * 4
    s.arrival_us = np.array([5000, 5000 + done + 7], np.int64)
    r = O.run(s, 2, 100, update="none")
    assert list(r["route"]) == [0, 0]
    # worker 0's load is exactly the second query's estimate
    assert r["workers"][0]["load_est"] == L * 0.001
    assert r["workers"][0]["completions"] == 1


def test_nlms_single_step_closed_form():
    L, o = 37, 3
    s = _paths_stream([list(range(L)), list(range(200, 210))], [0, 1], out_len=o)
    s.arrival_us = np.array([0, 10**9], np.int64)
    r = O.run(s, 1, 1000, update="nlms")
    phi = np.array([0.0, L * 0.001, 0.0, 1.0])
    E = (1000 * L + 10000 * o) * 1e-6
    e = E - (L * 0.001 + 0.0)
    theta = 0.992 * e / (1e-9 + phi @ phi) * phi
    np.testing.assert_allclose(r["workers"][0]["theta"], theta, rtol=1e-13, atol=1e-18)


def _nlms_step(theta, phi, e, mu=0.992, eps=1e-9):
    """One normalised-LMS step, every sum left to right (Sec. 4.2 update)."""
    ss = phi[0] * phi[0]
    ss = ss + phi[1] * phi[1]
    ss = ss + phi[2] * phi[2]
    ss = ss + phi[3] * phi[3]
    g = (mu * e) / (eps + ss)
    return [theta[a] + g * phi[a] for a in range(4)]


def _dot4(theta, phi):
    acc = theta[0] * phi[0]
    acc = acc + theta[1] * phi[1]
    acc = acc + theta[2] * phi[2]
    return acc + theta[3] * phi[3]


def test_nlms_error_uses_current_model_when_completions_lag_routing():
    """Algorithm 2's update thread minimises the squared loss of Sec. 4.2 at
    the current parameters: the error fed to the update is the observed
    latency minus the current model's prediction on the features stored at
    routing.  Two queries are routed to one worker before the first
    completes, so the second update differs from one that feeds the
    prediction made at routing time (when theta was still 0): the pin tells
    the two readings apart."""
    L1, L2, shared, o = 30, 50, 10, 4
    q1 = list(range(L1))
    q2 = list(range(shared)) + list(range(500, 500 + L2 - shared))
    s = _paths_stream([q1, q2, [900]], [0, 1, 2], out_len=o)
    s.arrival_us = np.array([0, 1000, 10**9], np.int64)  # q2 routed before q1 completes
    r = O.run(s, 1, 1000, update="nlms")
    assert list(r["hits"]) == [0, shared, 0]
    # query 1 at t = 0: empty cache, zero load
    x2_1 = float(L1 - 0) * 0.001
    phi1 = [0.0, x2_1, 0.0, 1.0]
    chat1 = 0.0 * 0.0 + 1.0 * x2_1
    base1 = chat1 + 0.0
    cost1 = 1000 * L1 + 10000 * o
    E1 = cost1 * 1e-6
    # query 2 at t = 1 ms (same decay tick): load = chat1, backlog = cost1 - 1 ms
    P2 = 0.0 + chat1
    x1_2, x2_2 = float(shared) * 0.001, float(L2 - shared) * 0.001
    phi2 = [x1_2, x2_2, P2, 1.0]
    chat2 = 0.0 * x1_2 + 1.0 * x2_2
    base2 = chat2 + P2
    E2 = ((cost1 - 1000) + (1000 * (L2 - shared) + 10000 * o)) * 1e-6
    # both complete before query 3: updates in FIFO order
    theta1 = _nlms_step([0.0] * 4, phi1, E1 - (base1 + _dot4([0.0] * 4, phi1)))
    theta_now = _nlms_step(theta1, phi2, E2 - (base2 + _dot4(theta1, phi2)))
    theta_routing = _nlms_step(theta1, phi2, E2 - (base2 + _dot4([0.0] * 4, phi2)))
    got = r["workers"][0]["theta"]
    np.testing.assert_allclose(got, theta_now, rtol=1e-15, atol=0.0)
    # the readings differ by far more than rounding on this stream
    diff = np.abs(np.array(theta_now) - np.array(theta_routing))
    assert diff.max() > 1e-3 * np.abs(theta_now).max(), (theta_now, theta_routing)


def test_rls_equals_weighted_ridge_least_squares():
    """RLS with forgetting factor lam and P0 = p0*I minimises
    sum_t lam^(n-t) (y_t - theta.phi_t)^2 + lam^n |theta|^2 / p0."""
    rng = np.random.default_rng(3)
    sp = small_spec(n=120, groups=4, prefix_len=(10, 60), suffix_len=(5, 40), vocab=30)
    s = generate(sp)
    s.arrival_us = (np.arange(1, s.n + 1) * 10**8).astype(np.int64)  # every query completes first
    s.out_len = rng.integers(0, 9, size=s.n).astype(np.uint16)
    lam, p0 = 0.992, 100.0
    r = O.run(s, 1, 10**6, update="rls", lr=lam, rls_p0=p0)
    L = s.lengths
    h = r["hits"].astype(np.int64)
    n_upd = s.n - 1  # the last query has not completed
    Phi = np.stack([h * 0.001, (L - h) * 0.001, np.zeros_like(h, float), np.ones_like(h, float)], 1)[:n_upd]
    E = (1000 * (L - h) + 10000 * s.out_len.astype(np.int64)) * 1e-6
    y = (E - (L - h) * 0.001)[:n_upd]
    wts = lam ** np.arange(n_upd - 1, -1, -1, dtype=float)
    A = (Phi * wts[:, None]).T @ Phi + (lam ** n_upd / p0) * np.eye(4)
    b = (Phi * wts[:, None]).T @ y
    theta = np.linalg.solve(A, b)
    np.testing.assert_allclose(r["workers"][0]["theta"], theta, rtol=1e-7, atol=1e-9)


def test_ties_route_to_lowest_index():
    s = _paths_stream([[1, 2], [3, 4], [5, 6]], [0, 1, 2])
    s.arrival_us = np.array([10**9, 2 * 10**9, 3 * 10**9], np.int64)
    r = O.run(s, 4, 100, update="none")
    assert list(r["route"]) == [0, 0, 0]


# ---------------------------------------------------------------------------
# invariants on generated workloads

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_invariants_hold(seed):
    s = generate(small_spec(n=400, groups=7, prefix_len=(10, 60), suffix_len=(5, 40),
                            vocab=20, seed=seed))
    W, B = 3, 250
    r = O.run(s, W, B, replica=seed, check=1, all_hits=True)
    assert r["rc"] == 0
    L = s.lengths
    assert (r["all_hits"] <= L[:, None]).all() and (r["all_hits"] >= 0).all()
    assert ((r["route"] >= 0) & (r["route"] < W)).all()
    assert sum(w["routed"] for w in r["workers"]) == s.n
    for w in r["workers"]:
        assert w["resident"] <= B
        assert w["resident"] == w["loads"] - w["evictions"]
        assert w["marked_count"] == w["cnt"] <= B
        assert w["load_est"] >= 0.0


@pytest.mark.parametrize("which", [1, 2, 3])
def test_invariant_checks_catch_planted_violations(which):
    """The oracle's own checks fire on a planted violation (on the CPU):
    1 = a negative load estimate on a worker, 2 = a change to a worker the
    step did not route to (Eq. 3), 3 = a token whose parent is gone."""
    assert O.check_selftest(which)


@pytest.mark.parametrize("mode", ["rlt", "lru", "responses", "batch", "router_tree", "cache_aware"])
def test_invariants_and_eq3_hold_every_step(mode):
    """check = 1: after every step capacity, prefix closure, marks, running
    batch counts and P >= 0 hold, and only the routed worker's cache (and
    router tree) changed (Sec. 3.1, Eq. 3)."""
    s = generate(small_spec(n=300, groups=6, prefix_len=(8, 40), suffix_len=(4, 24), vocab=12, seed=7))
    kw = {"rlt": {}, "lru": {"evict": "lru"}, "responses": {"cache_responses": 1},
          "batch": {"batch_size": 3}, "router_tree": {"router_tree": 1, "router_tree_tokens": 90},
          "cache_aware": {"router": "cache_aware", "ca_balance_abs": 2}}[mode]
    if mode == "responses":
        s = generate(dict(small_spec(n=300, groups=6, prefix_len=(8, 40), suffix_len=(4, 24), vocab=12,
                                     seed=7), responses=True))
    B = 3 * s.max_len if mode == "batch" else 160  # batching assumes beta * L_max <= B
    r = O.run(s, 3, B, replica=1, check=1, **kw)
    assert r["rc"] == 0
    assert sum(w["evictions"] for w in r["workers"]) > 0
    assert len(set(r["route"].tolist())) > 1


# ---------------------------------------------------------------------------
# baseline routers (Sec. 5 "Baselines")

def test_round_robin_cycles_through_workers():
    s = generate(small_spec(n=97, groups=3, prefix_len=(3, 9), suffix_len=(1, 5), vocab=7))
    for W in (1, 3, 5):
        r = O.run(s, W, 40, router="round_robin")
        assert r["rc"] == 0
        assert list(r["route"]) == [j % W for j in range(s.n)]


def test_random_router_is_uniform_and_keyed():
    """Random routing draws word 0 of Philox4x64-10 (numpy's implementation
    here) with key (seed, replica) and counter (j, 0, 0, 1); the routes are
    uniform over the workers and differ between replicas."""
    s = generate(small_spec(n=4000, groups=4, prefix_len=(2, 6), suffix_len=(1, 4), vocab=50))
    W = 5
    r0 = O.run(s, W, 10**6, router="random", replica=0, seed=3)
    r1 = O.run(s, W, 10**6, router="random", replica=1, seed=3)
    want = [(SM.philox_word0(3, 0, (j, 0, 0, 1)) * W) >> 64 for j in range(s.n)]
    assert list(r0["route"]) == want
    assert (r0["route"] != r1["route"]).mean() > 0.7
    counts = np.bincount(r0["route"], minlength=W)
    chi2 = float(((counts - s.n / W) ** 2 / (s.n / W)).sum())
    assert chi2 < 18.5  # chi-square, 4 degrees of freedom, p = 0.001


def test_cache_aware_switches_on_load_imbalance():
    """W = 2, queries sharing one long prefix, arrivals 1 us apart (nothing
    completes): the highest hit (worker 0) takes queries until it has more
    than ca_balance_abs more in flight than worker 1; then the least loaded
    worker takes one, and the two alternate."""
    prefix = list(range(100, 150))
    paths = [prefix + [1000 + k] * 10 for k in range(40)]
    s = generate({"kind": "paths", "paths": paths, "order": list(range(40)), "gap_us": 1})
    r = O.run(s, 2, 10**5, router="cache_aware", ca_balance_abs=32)
    assert r["rc"] == 0
    route = list(r["route"])
    # query 0: no hits anywhere, equal caches -> worker 0; then worker 0 has
    # the prefix (hit share 50/60 > 0.5) until 33 queries are in flight there
    assert route[:33] == [0] * 33
    assert route[33:37] == [1, 0, 1, 0]


def test_cache_aware_low_hits_go_to_the_emptiest_cache():
    """Unrelated queries (hit share 0): each goes to the worker with the
    fewest cached tokens, the lowest index on ties."""
    paths = [[10 * k + t for t in range(5 + k)] for k in range(6)]
    s = generate({"kind": "paths", "paths": paths, "order": list(range(6)), "gap_us": 10**7})
    r = O.run(s, 3, 10**5, router="cache_aware")
    assert r["rc"] == 0
    # sizes after each query: w0 5 | w1 6 | w2 7 | w0 5+8 | w1 6+9 | w2 7+10
    assert list(r["route"]) == [0, 1, 2, 0, 1, 2]


# ---------------------------------------------------------------------------
# cached responses: a path is q_j || a_j, the last out_len[j] tokens

def _random_response_stream(rng, n, vocab, max_prompt, max_resp, B):
    paths, olen = [], []
    for _ in range(n):
        L = int(rng.integers(1, max(1, min(max_prompt, B - max_resp)) + 1))
        o = int(rng.integers(0, max_resp + 1))
        paths.append([int(x) for x in rng.integers(0, vocab, size=L + o)])
        olen.append(o)
    gaps = rng.integers(1, 400000, size=n)
    s = _paths_stream(paths, list(range(n)))
    s.arrival_us = np.cumsum(gaps).astype(np.int64)
    s.out_len = np.array(olen, dtype=np.uint16)
    return s


@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_responses_equal_bruteforce_model(evict):
    rng = np.random.default_rng(77 + len(evict))
    for case in range(60):
        W = int(rng.integers(1, 4))
        B = int(rng.integers(4, 14))
        vocab = int(rng.integers(2, 5))
        n = int(rng.integers(5, 30))
        s = _random_response_stream(rng, n, vocab, 5, 3, B)
        replica = int(rng.integers(0, 1000))
        kw = dict(evict=evict, seed=int(rng.integers(0, 2**32)), cache_responses=1)
        r = O.run(s, W, B, replica=replica, all_hits=True, check=1, **kw)
        assert r["rc"] == 0
        sim, routes, hits, allh = SM.run_spec(s, W, B, replica=replica, **kw)
        np.testing.assert_array_equal(r["route"], routes)
        np.testing.assert_array_equal(r["all_hits"], allh)
        prompts = s.lengths - s.out_len.astype(np.int64)
        assert (r["hits"] <= prompts).all()
        for i in range(W):
            ws, sw = r["workers"][i], sim.w[i]
            assert ws["evictions"] == sw.evictions and ws["loads"] == sw.loads
            assert (ws["resident"], ws["digest_sum"], ws["digest_xor"]) == _digest_of_set(sw.S)
            assert ws["load_est"] == sw.P and ws["theta"] == sw.theta


@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_empty_responses_reduce_to_prompt_caching(evict):
    s = generate(small_spec(n=250, groups=4, prefix_len=(4, 20), suffix_len=(1, 12), vocab=8))
    s.out_len = np.zeros(s.n, dtype=np.uint16)
    a = O.run(s, 3, 60, replica=3, all_hits=True, evict=evict)
    b = O.run(s, 3, 60, replica=3, all_hits=True, evict=evict, cache_responses=1)
    np.testing.assert_array_equal(a["route"], b["route"])
    np.testing.assert_array_equal(a["all_hits"], b["all_hits"])
    assert a["workers"] == b["workers"]
    assert sum(w["evictions"] for w in a["workers"]) > 0


def test_responses_match_and_contents_over_routed_history():
    """Nothing evicted: h_ij is the longest common prefix of the prompt with
    any complete path routed to worker i before, the cache of i holds exactly
    the prefixes of those paths, and only a prompt's tokens count as hits."""
    sp = {"kind": "sessions", "n_sessions": 40, "turns": (1, 5), "start_len": 6,
          "ext_len": (1, 6), "vocab": 5, "responses": True, "out_len": 3, "turn_rate": 3.0}
    s = generate(sp)
    W, B = 3, 10**6
    r = O.run(s, W, B, all_hits=True, cache_responses=1)
    assert r["rc"] == 0 and sum(w["evictions"] for w in r["workers"]) == 0
    paths = [tuple(int(x) for x in s.query(j)) for j in range(s.n)]
    prompts = [p[: len(p) - int(s.out_len[j])] for j, p in enumerate(paths)]
    seen = [set() for _ in range(W)]
    seen_prompts = [set() for _ in range(W)]

    def lcp_max(xs, q):
        best = 0
        for x in xs:
            l = 0
            while l < min(len(x), len(q)) and x[l] == q[l]:
                l += 1
            best = max(best, l)
        return best

    carried = 0
    for j in range(s.n):
        for i in range(W):
            assert r["all_hits"][j, i] == lcp_max(seen[i], prompts[j])
        i = int(r["route"][j])
        # the hit reaches into a cached response: more than any prompt gives
        carried += int(r["hits"][j] > lcp_max(seen_prompts[i], prompts[j]))
        seen[i].add(paths[j])
        seen_prompts[i].add(prompts[j])
    for i in range(W):
        prefixes = {x[:k] for x in seen[i] for k in range(1, len(x) + 1)}
        assert r["workers"][i]["resident"] == len(prefixes) == r["workers"][i]["loads"]
    # a later turn's prompt contains the previous turn's response, and hits reach into it
    assert carried > 0


# ---------------------------------------------------------------------------
# continuous batching: the paths of a worker's running batch (the beta - 1
# queries routed there before the current one) are never evicted
# (Sec. 3.2, Theorem 2 and its assumption beta * L_max <= B)

@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_batching_equals_bruteforce_model(evict):
    rng = np.random.default_rng(300 + len(evict))
    for case in range(80):
        W = int(rng.integers(1, 4))
        beta = int(rng.integers(2, 5))
        B = int(rng.integers(2 * beta, 16))
        vocab = int(rng.integers(2, 5))
        n = int(rng.integers(5, 35))
        s = _random_tiny_stream(rng, n, vocab, B // beta, B)
        replica = int(rng.integers(0, 1000))
        kw = dict(evict=evict, seed=int(rng.integers(0, 2**32)), batch_size=beta)
        r = O.run(s, W, B, replica=replica, all_hits=True, check=1, **kw)
        assert r["rc"] == 0
        sim, routes, hits, allh = SM.run_spec(s, W, B, replica=replica, **kw)
        np.testing.assert_array_equal(r["route"], routes)
        np.testing.assert_array_equal(r["all_hits"], allh)
        for i in range(W):
            ws, sw = r["workers"][i], sim.w[i]
            assert ws["evictions"] == sw.evictions and ws["loads"] == sw.loads
            assert (ws["resident"], ws["digest_sum"], ws["digest_xor"]) == _digest_of_set(sw.S)
            assert ws["load_est"] == sw.P and ws["theta"] == sw.theta
            # the running batch is cached whole
            for p in sw.running:
                assert all(p[:k] in sw.S for k in range(1, len(p) + 1))


@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_batching_candidate_list_equals_definition(evict):
    """The maintained candidate list, rebuilt when a released path leaves an
    unmarked leaf, gives the same run as U recomputed at every draw."""
    rng = np.random.default_rng(17)
    for case in range(12):
        beta = int(rng.integers(2, 9))
        sp = small_spec(n=int(rng.integers(100, 250)), groups=int(rng.integers(2, 8)),
                        prefix_len=(4, 20), suffix_len=(1, 12), vocab=int(rng.integers(3, 40)), seed=case)
        s = generate(sp)
        W = int(rng.integers(1, 4))
        B = int(max(beta * s.max_len, rng.integers(40, 300)))
        a = O.run(s, W, B, replica=case, u_mode=0, all_hits=True, evict=evict, batch_size=beta, check=1)
        b = O.run(s, W, B, replica=case, u_mode=1, all_hits=True, evict=evict, batch_size=beta)
        assert a["rc"] == 0 and b["rc"] == 0
        np.testing.assert_array_equal(a["route"], b["route"])
        np.testing.assert_array_equal(a["all_hits"], b["all_hits"])
        assert a["workers"] == b["workers"]
        assert sum(w["evictions"] for w in a["workers"]) > 0


def test_batching_without_eviction_changes_nothing():
    s = generate(small_spec(n=200, groups=5, prefix_len=(5, 25), suffix_len=(1, 15), vocab=6))
    a = O.run(s, 3, 10**6, all_hits=True)
    b = O.run(s, 3, 10**6, all_hits=True, batch_size=7, check=1)
    np.testing.assert_array_equal(a["all_hits"], b["all_hits"])
    assert a["workers"] == b["workers"]


@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_batching_protects_the_running_batch(evict):
    """B = 4, beta = 2: (1,2) then (3,4) fill the cache; (5) starts a new
    phase and needs one eviction.  The leaves are (1,2) and (3,4), but (3,4)
    is in the running batch, so (1,2) goes for every random key (single-query
    processing takes either with probability 1/2 under RLT)."""
    s = _paths_stream([[1, 2], [3, 4], [5], [1, 2]], [0, 1, 2, 3])
    for rep in range(40):
        r = O.run(s, 1, 4, replica=rep, evict=evict, batch_size=2, check=1)
        assert r["rc"] == 0
        assert list(r["hits"]) == [0, 0, 0, 1]
    one = [O.run(s, 1, 4, replica=rep, evict="rlt")["hits"][3] for rep in range(200)]
    assert 0 < one.count(2) < 200 and one.count(1) + one.count(2) == 200


BATCH_EXACT_CASES = [
    (6, 2, [(0, 1, 2), (0, 1, 3), (0, 2, 0), (1, 2, 3), (0, 1, 2), (1, 2), (0, 1, 3), (0, 2, 1),
            (1, 2, 3), (0, 1, 2), (2, 0, 1), (0, 1, 3)]),
    (6, 3, [(0, 1), (0, 2), (1, 0), (0, 1), (1, 1), (0, 2), (2, 2), (0, 1), (1, 0), (0, 2), (2, 1)]),
]


@pytest.mark.parametrize("case", range(len(BATCH_EXACT_CASES)))
def test_batching_mean_hits_match_exact_enumeration(case):
    """Mean hits over many random keys = the exact expectation, enumerated
    over every draw with the running batch excluded from U; the expectation
    differs from single-query processing, so the pins have an effect."""
    B, beta, queries = BATCH_EXACT_CASES[case]
    exact = SM.expected_hits(queries, B, batch_size=beta)
    assert exact != SM.expected_hits(queries, B)
    s = _paths_stream([list(q) for q in queries], list(range(len(queries))))
    R = 20000
    per = np.zeros((R, len(queries)))
    for rep in range(R):
        per[rep] = O.run(s, 1, B, replica=rep, batch_size=beta)["hits"]
    tot = per.sum(axis=1)
    sd = tot.std(ddof=1) / math.sqrt(R)
    assert abs(tot.mean() - float(sum(exact))) < 4 * sd + 1e-12
    for j, e in enumerate(exact):
        sdj = per[:, j].std(ddof=1) / math.sqrt(R)
        assert abs(per[:, j].mean() - float(e)) < 4.5 * sdj + 1e-12


def test_lru_batch_lower_bound_construction():
    """Theorem 2 lower bound: B-L+2 paths share an (L-1)-token prefix; batch
    u is {G_1, ..., G_(beta-1), G_(u+beta-1)} for u = 1..B-L-beta+3, queried
    in a loop.  L-LRU misses the tail of every rotating query once the
    cache is full, while the first beta-1 paths always hit."""
    for B, L, beta in [(12, 3, 3), (20, 4, 4), (30, 2, 2)]:
        paths, n = _tail_paths(B, L)
        m = B - L - beta + 3
        order = []
        for _ in range(5):
            for u in range(m):
                order += list(range(beta - 1)) + [u + beta - 1]
        s = _paths_stream(paths, order)
        r = O.run(s, 1, B, evict="lru", batch_size=beta, check=1)
        assert r["rc"] == 0
        h = r["hits"].reshape(5, m, beta)
        assert (h[1:, :, : beta - 1] == L).all()
        assert (h[1:, :, beta - 1] == L - 1).all()


# ---------------------------------------------------------------------------
# approximate router tree (App. E): the router matches against a tree of its
# own per worker (routed prompts, L-LRU under its own budget); the observed
# latency and the hit counts take the worker's true match

@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_router_tree_equals_bruteforce_model(evict):
    rng = np.random.default_rng(600 + len(evict))
    for case in range(80):
        W = int(rng.integers(1, 4))
        B = int(rng.integers(5, 14))
        vocab = int(rng.integers(2, 5))
        n = int(rng.integers(5, 35))
        resp = case % 2
        if resp:
            s = _random_response_stream(rng, n, vocab, 5, 3, B)
        else:
            s = _random_tiny_stream(rng, n, vocab, 6, B)
        RB = int(rng.integers(int(s.lengths.max()), 16))
        replica = int(rng.integers(0, 1000))
        kw = dict(evict=evict, seed=int(rng.integers(0, 2**32)), router_tree=1, router_tree_tokens=RB,
                  cache_responses=resp)
        r = O.run(s, W, B, replica=replica, all_hits=True, check=1, **kw)
        assert r["rc"] == 0
        sim, routes, hits, allh = SM.run_spec(s, W, B, replica=replica, **kw)
        np.testing.assert_array_equal(r["route"], routes)
        np.testing.assert_array_equal(r["hits"], hits)
        np.testing.assert_array_equal(r["all_hits"], allh)
        for i in range(W):
            ws, sw = r["workers"][i], sim.w[i]
            assert ws["evictions"] == sw.evictions and ws["loads"] == sw.loads
            assert (ws["resident"], ws["digest_sum"], ws["digest_xor"]) == _digest_of_set(sw.S)
            assert (ws["router_resident"], ws["router_digest_sum"], ws["router_digest_xor"]) == \
                _digest_of_set(sim.rt[i])
            assert ws["router_evictions"] == sim.rt_evictions[i]
            assert ws["load_est"] == sw.P and ws["theta"] == sw.theta


def test_router_tree_without_eviction_is_exact():
    """Neither the caches nor the router's trees evict: the router's trees
    hold exactly the routed prompts, as the caches do, so the estimate is
    the true match and the run is that of the exact router."""
    s = generate(small_spec(n=250, groups=5, prefix_len=(5, 25), suffix_len=(1, 15), vocab=6))
    a = O.run(s, 3, 10**6, all_hits=True)
    b = O.run(s, 3, 10**6, all_hits=True, router_tree=1, check=1)
    np.testing.assert_array_equal(a["route"], b["route"])
    np.testing.assert_array_equal(a["all_hits"], b["all_hits"])
    for x, y in zip(a["workers"], b["workers"]):
        assert {k: x[k] for k in x if not k.startswith("router_")} == {k: y[k] for k in y if not k.startswith("router_")}
        assert y["router_resident"] == y["resident"] and y["router_digest_sum"] == y["digest_sum"]


def _lcp_max(xs, q):
    best = 0
    for x in xs:
        l = 0
        while l < min(len(x), len(q)) and x[l] == q[l]:
            l += 1
        best = max(best, l)
    return best


@pytest.mark.parametrize("evict", ["rlt", "lru"])
def test_router_tree_overestimates_an_evicting_cache(evict):
    """A router tree that never evicts: its estimate is the longest common
    prefix with any prompt routed to the worker before (a closed form over
    the routed history); the worker's cache evicts, so its true match, which
    the hit counts report, is at most that."""
    s = generate(small_spec(n=300, groups=6, prefix_len=(5, 30), suffix_len=(2, 15), vocab=7))
    W, B = 3, 60
    r = O.run(s, W, B, all_hits=True, evict=evict, router_tree=1, router_tree_tokens=10**6, check=1)
    assert r["rc"] == 0 and sum(w["evictions"] for w in r["workers"]) > 0
    assert sum(w["router_evictions"] for w in r["workers"]) == 0
    qs = [tuple(int(x) for x in s.query(j)) for j in range(s.n)]
    seen = [[] for _ in range(W)]
    under = 0
    for j in range(s.n):
        for i in range(W):
            assert r["all_hits"][j, i] == _lcp_max(seen[i], qs[j])
        i = int(r["route"][j])
        assert r["hits"][j] <= r["all_hits"][j, i]
        under += int(r["hits"][j] < r["all_hits"][j, i])
        seen[i].append(qs[j])
    assert under > 0  # the estimate is off where the cache evicted


def test_router_tree_underestimates_with_a_small_budget():
    """A router tree with a small budget and caches that never evict: the
    true match is the closed form over the routed history and the router's
    estimate is at most that."""
    s = generate(small_spec(n=300, groups=6, prefix_len=(5, 30), suffix_len=(2, 15), vocab=7))
    W = 3
    r = O.run(s, W, 10**6, all_hits=True, router_tree=1, router_tree_tokens=int(s.lengths.max()) + 5, check=1)
    assert r["rc"] == 0 and sum(w["router_evictions"] for w in r["workers"]) > 0
    qs = [tuple(int(x) for x in s.query(j)) for j in range(s.n)]
    seen = [[] for _ in range(W)]
    over = 0
    for j in range(s.n):
        i = int(r["route"][j])
        assert r["hits"][j] == _lcp_max(seen[i], qs[j])
        assert r["all_hits"][j, i] <= r["hits"][j]
        over += int(r["all_hits"][j, i] < r["hits"][j])
        seen[i].append(qs[j])
    assert over > 0


# ---------------------------------------------------------------------------
# Theorem 3's phase bound: in a phase with c clean tokens RLT misses at most
# c + c(H_n - H_c) tokens in expectation, n = min(B - L + c, B)

def _harmonic(k):
    return sum(Fraction(1, i) for i in range(1, k + 1))


@pytest.mark.parametrize("c", [1, 4, 8])
def test_rlt_phase_miss_bound_on_the_proofs_adversary(c):
    """Paths share an (L-1)-token prefix and differ in the last token, so a
    phase of the marking algorithm covers B-L+1 distinct tails.  Every phase
    first asks for c tails never seen (clean), then for B-L+1-c tails of the
    previous phase (stale): the order the proof calls the worst.  The mean
    misses per phase over many random keys stay within the bound, and at
    least the c clean misses happen."""
    B, L = 20, 4
    k = B - L + 1  # tails per phase
    prefix = [500, 501, 502]
    nxt = 0
    phases = [list(range(k))]
    nxt = k
    for p in range(12):
        clean = list(range(nxt, nxt + c))
        nxt += c
        phases.append(clean + phases[-1][: k - c])
    tails = [t for ph in phases for t in ph]
    paths = {t: prefix + [10000 + t] for t in set(tails)}
    ids = sorted(paths)
    s = _paths_stream([paths[t] for t in ids], [ids.index(t) for t in tails])
    reps = 600
    per_phase = np.zeros((reps, len(phases) - 1))
    for rep in range(reps):
        r = O.run(s, 1, B, replica=rep, check=1)
        assert r["rc"] == 0
        miss = L - r["hits"]
        for p in range(1, len(phases)):
            per_phase[rep, p - 1] = miss[p * k:(p + 1) * k].sum()
    n = min(B - L + c, B)
    bound = float(c + c * (_harmonic(n) - _harmonic(c)))
    m = per_phase[:, 1:].mean()  # phase 1 follows the fill, start from the next
    sd = per_phase[:, 1:].mean(axis=1).std(ddof=1) / math.sqrt(reps)
    assert per_phase.min() >= c
    assert m <= bound + 4 * sd, (m, bound)
    # the stale requests do miss sometimes: the bound is not vacuous here
    assert m > c
