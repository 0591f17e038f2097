"""Brute-force model of the simulation for tiny inputs (test pins only).

The cache of a worker is a Python ``set`` of token tuples (every cached root
path); nothing is compressed, nothing is maintained incrementally:

* the hit count is the largest l with ``tuple(q[:l]) in S`` (Sec. 3.2,
  "Cache Matching");
* U is recomputed at every draw by filtering S for leaves (paths with no
  cached one-token extension) that are not in the marking set, are not the
  insertion point and are not a prefix of a path in the worker's running
  batch (continuous batching: the last beta - 1 paths routed there), sorted
  with Python's tuple order, which is lexicographic order of root paths
  (Algorithm 1);
* random words come from numpy's Philox bit generator (a library
  implementation of Philox4x64-10), not from the oracle's own code.

The LBGR arithmetic (Algorithm 2, Sec. 4.2, App. A constants) is evaluated
in Python floats, which are IEEE doubles without fused multiply-add, in the
same order the oracle documents.

``expected_hits`` enumerates every random choice of RLT with its exact
probability (``fractions.Fraction``) for one worker, giving the exact
expectation the randomized algorithm must reach.
"""
from __future__ import annotations

from fractions import Fraction
from typing import Dict, List, Tuple

import numpy as np

MASK64 = (1 << 64) - 1


def philox_word0(seed: int, replica: int, ctr: Tuple[int, int, int, int]) -> int:
    """Word 0 of Philox4x64-10(counter=ctr, key=(seed, replica)) via numpy.

    numpy's generator increments its 256-bit counter before producing a
    block, so it is started one below the wanted counter."""
    c = ctr[0] | (ctr[1] << 64) | (ctr[2] << 128) | (ctr[3] << 192)
    c = (c - 1) % (1 << 256)
    words = np.array([(c >> (64 * k)) & MASK64 for k in range(4)], dtype=np.uint64)
    bg = np.random.Philox(counter=words, key=np.array([seed, replica], dtype=np.uint64))
    return int(bg.random_raw(1)[0])


def _leaves(S) -> List[tuple]:
    parents = {x[:-1] for x in S}
    return [x for x in S if x not in parents]


def lcp(S, q) -> int:
    h = 0
    while h < len(q) and tuple(q[: h + 1]) in S:
        h += 1
    return h


class SpecWorker:
    def __init__(self, rls_p0: float):
        self.S = set()
        self.mark: Dict[tuple, int] = {}
        self.phase = 1
        self.cnt = 0
        self.P = 0.0
        self.theta = [0.0, 0.0, 0.0, 0.0]
        self.Pm = [[rls_p0 if a == b else 0.0 for b in range(4)] for a in range(4)]
        self.tl = 0
        self.Wb = 0
        self.pend: List[dict] = []
        self.running: List[tuple] = []  # paths of the running batch
        self.evictions = 0
        self.loads = 0
        self.forced = 0


def pow_int(rho: float, k: int) -> float:
    res, b = 1.0, rho
    while k:
        if k & 1:
            res = res * b
        b = b * b
        k >>= 1
    return res


class SpecSim:
    def __init__(self, W: int, B: int, replica: int = 0, seed: int = 0, evict: str = "rlt",
                 update: str = "nlms", alpha_cached=0.0, alpha_miss=1.0, rho=31 / 32,
                 decay_interval_us=20000, lr=0.992, nlms_eps=1e-9, rls_p0=100.0,
                 true_cached_us=0, true_miss_us=1000, true_out_us=10000, cache_responses=0, batch_size=1,
                 router_tree=0, router_tree_tokens=0):
        self.W, self.B, self.r, self.seed = W, B, replica, seed
        self.beta = int(batch_size)
        # the router's own tree per worker (App. E): routed prompts, L-LRU
        self.approx = bool(router_tree)
        self.RB = int(router_tree_tokens) or B
        self.rt = [set() for _ in range(W)]
        self.rstamp: List[Dict[tuple, int]] = [dict() for _ in range(W)]
        self.rt_evictions = [0] * W
        self.responses = bool(cache_responses)
        self.evict, self.update = evict, update
        self.ac, self.am, self.rho, self.dt = alpha_cached, alpha_miss, rho, decay_interval_us
        self.lr, self.eps = lr, nlms_eps
        self.tc, self.tm, self.to = true_cached_us, true_miss_us, true_out_us
        self.w = [SpecWorker(rls_p0) for _ in range(W)]
        self.tprev = 0
        self.stamp: List[Dict[tuple, int]] = [dict() for _ in range(W)]

    # -- residual model
    def _update(self, w: SpecWorker, phi, e):
        if self.update == "nlms":
            ss = phi[0] * phi[0]
            ss = ss + phi[1] * phi[1]
            ss = ss + phi[2] * phi[2]
            ss = ss + phi[3] * phi[3]
            g = (self.lr * e) / (self.eps + ss)
            w.theta = [w.theta[a] + g * phi[a] for a in range(4)]
        elif self.update == "rls":
            pi = []
            for a in range(4):
                acc = w.Pm[a][0] * phi[0]
                for b in range(1, 4):
                    acc = acc + w.Pm[a][b] * phi[b]
                pi.append(acc)
            den = phi[0] * pi[0]
            for b in range(1, 4):
                den = den + phi[b] * pi[b]
            den = self.lr + den
            k = [pi[a] / den for a in range(4)]
            w.theta = [w.theta[a] + k[a] * e for a in range(4)]
            w.Pm = [[(w.Pm[a][b] - k[a] * pi[b]) / self.lr for b in range(4)] for a in range(4)]

    def step(self, jg: int, q, t: int, o: int):
        path = tuple(int(x) for x in q)
        # with cached responses the path is prompt || response and only the
        # prompt is known when routing
        q = path[: len(path) - o] if self.responses else path
        L = len(q)
        for w in self.w:
            while w.pend and w.pend[0]["t_done"] <= t:
                c = w.pend.pop(0)
                w.P = w.P * pow_int(self.rho, c["t_done"] // self.dt - w.tl // self.dt)
                w.tl = c["t_done"]
                rem = c["chat"] * pow_int(self.rho, c["t_done"] // self.dt - c["t_route"] // self.dt)
                w.P = max(0.0, w.P - rem)
                res = w.theta[0] * c["phi"][0]
                for a in range(1, 4):
                    res = res + w.theta[a] * c["phi"][a]
                self._update(w, c["phi"], c["e_obs"] - (c["base"] + res))
            w.P = w.P * pow_int(self.rho, t // self.dt - w.tl // self.dt)
            w.tl = t
            w.Wb = max(0, w.Wb - (t - self.tprev))
        self.tprev = t
        h = [lcp(self.rt[i], q) if self.approx else lcp(w.S, q) for i, w in enumerate(self.w)]
        best, ehats, chats, phis = 0, [], [], []
        for i, w in enumerate(self.w):
            x = [h[i] * 0.001, (L - h[i]) * 0.001, w.P, 1.0]
            ch = self.ac * x[0] + self.am * x[1]
            res = w.theta[0] * x[0]
            for a in range(1, 4):
                res = res + w.theta[a] * x[a]
            eh = (ch + w.P) + res
            ehats.append(eh)
            chats.append(ch)
            phis.append(x)
            if i == 0 or eh < ehats[best]:
                best = i
        w = self.w[best]
        base = chats[best] + w.P
        w.P = w.P + chats[best]
        hb = lcp(w.S, q)  # the worker's true match
        cost = self.tc * hb + self.tm * (L - hb) + self.to * o
        e_us = w.Wb + cost
        w.Wb = w.Wb + cost
        w.pend.append({"t_route": t, "t_done": t + e_us, "chat": chats[best], "base": base,
                       "e_obs": e_us * 1e-6, "phi": phis[best]})
        if self.evict == "rlt":
            self._insert_rlt(best, path, jg)
        else:
            w.loads += sum(1 for p in range(len(path)) if path[: p + 1] not in w.S)
            w.evictions += self._lru(w.S, self.stamp[best], B=self.B, q=path, jg=jg, pinned=self._pinned(w))
        if self.beta > 1:
            w.running = (w.running + [path])[-(self.beta - 1):]
        if self.approx:
            self.rt_evictions[best] += self._lru(self.rt[best], self.rstamp[best], B=self.RB, q=q, jg=jg,
                                                 pinned=set())
        return best, hb, h

    @staticmethod
    def _pinned(w: SpecWorker) -> set:
        return {p[:k] for p in w.running for k in range(1, len(p) + 1)}

    def _insert_rlt(self, i: int, q, jg: int):
        w, B = self.w[i], self.B
        pinned = self._pinned(w)
        d = 0
        for p in range(len(q)):
            v, u0 = q[: p + 1], q[:p]
            if v not in w.S or w.mark.get(v, 0) != w.phase:
                w.cnt += 1
                if w.cnt == B + 1:
                    w.phase += 1
                    w.cnt = 1
                w.mark[v] = w.phase
            if v in w.S:
                continue
            if len(w.S) == B:
                U = sorted(x for x in _leaves(w.S) if w.mark.get(x, 0) != w.phase and x != u0 and x not in pinned)
                if not U:
                    w.phase += 1
                    w.cnt = 1
                    w.mark[v] = w.phase
                    w.forced += 1
                    U = sorted(x for x in _leaves(w.S)
                               if w.mark.get(x, 0) != w.phase and x != u0 and x not in pinned)
                    if not U:
                        raise RuntimeError("path longer than the cache")
                r64 = philox_word0(self.seed, self.r, (jg, i, d, 0))
                d += 1
                victim = U[(r64 * len(U)) >> 64]
                w.S.remove(victim)
                w.mark.pop(victim, None)
                w.evictions += 1
            w.S.add(v)
            w.loads += 1

    @staticmethod
    def _lru(S: set, st: Dict[tuple, int], B: int, q, jg: int, pinned: set) -> int:
        """L-LRU insertion of q into the token set S with access stamps st;
        returns the number of evictions.  (Counting loads is left to the
        caller: it is the number of tokens of q not in S beforehand.)"""
        ev = 0
        for p in range(len(q)):
            v, u0 = q[: p + 1], q[:p]
            if v in S:
                st[v] = (jg << 32) | p
                continue
            if len(S) == B:
                cands = [x for x in _leaves(S) if x != u0 and x not in pinned]
                victim = min(cands, key=lambda x: st[x])
                S.remove(victim)
                del st[victim]
                ev += 1
            S.add(v)
            st[v] = (jg << 32) | p
        return ev


def run_spec(stream, W: int, B: int, replica: int = 0, **kw):
    sim = SpecSim(W, B, replica=replica, **kw)
    routes, hits, allh = [], [], []
    for j in range(stream.n):
        r, hb, h = sim.step(j, stream.query(j), int(stream.arrival_us[j]), int(stream.out_len[j]))
        routes.append(r)
        hits.append(hb)
        allh.append(h)
    return sim, np.array(routes, np.int32), np.array(hits, np.int32), np.array(allh, np.int32)


# ---------------------------------------------------------------------------
# exact expectation of RLT on one worker by enumeration of every draw

def _rlt_branches(S: frozenset, T: frozenset, q, B: int, pinned=frozenset()):
    """All outcomes of inserting q with probabilities: {(S', T'): Fraction}.
    ``pinned``: tokens of in-progress paths, never evicted."""
    out: Dict[Tuple[frozenset, frozenset], Fraction] = {}

    def rec(S, T, p, prob):
        if p == len(q):
            key = (S, T)
            out[key] = out.get(key, Fraction(0)) + prob
            return
        v, u0 = tuple(q[: p + 1]), tuple(q[:p])
        if v not in T:
            T = T | {v}
            if len(T) == B + 1:
                T = frozenset({v})
        if v in S:
            rec(S, T, p + 1, prob)
            return
        if len(S) < B:
            rec(S | {v}, T, p + 1, prob)
            return
        U = sorted(x for x in _leaves(S) if x not in T and x != u0 and x not in pinned)
        if not U:
            T = frozenset({v})
            U = sorted(x for x in _leaves(S) if x not in T and x != u0 and x not in pinned)
        for x in U:
            rec((S - {x}) | {v}, T, p + 1, prob / len(U))

    rec(S, T, 0, Fraction(1))
    return out


def expected_hits(queries, B: int, batch_size: int = 1) -> List[Fraction]:
    """E[h_j] for every query of a one-worker RLT run, exactly; with
    continuous batching the last batch_size - 1 paths are never evicted."""
    dist = {(frozenset(), frozenset()): Fraction(1)}
    res = []
    running: List[tuple] = []
    for q in queries:
        q = tuple(int(x) for x in q)
        res.append(sum(p * lcp(S, q) for (S, T), p in dist.items()))
        pinned = frozenset(p[:k] for p in running for k in range(1, len(p) + 1))
        nd: Dict[Tuple[frozenset, frozenset], Fraction] = {}
        for (S, T), p in dist.items():
            for key, pp in _rlt_branches(S, T, q, B, pinned).items():
                nd[key] = nd.get(key, Fraction(0)) + p * pp
        dist = nd
        if batch_size > 1:
            running = (running + [q])[-(batch_size - 1):]
    return res
