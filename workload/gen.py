"""Seeded synthetic stream generators (numpy only).

Every preset follows a stream recipe whose shape matches one of the paper's
workload families (Sec. 5 "Workloads"; App. A):

* ``groups``    - GSP-like shared-prefix groups: a query is a group prefix
  followed by a fresh random suffix; the group is drawn from a Zipf law,
  optionally re-permuted every ``permute_every`` queries, optionally in
  bursts (two-state on/off chain).
* ``two_level`` - a system prompt followed by a task template and a fresh
  suffix (two-level prefix tree).
* ``sessions``  - multi-turn conversations (ShareGPT/UltraChat-like): turn k
  of a session is the session start followed by the first k extensions.
* ``paths``     - an explicit list of token paths queried in a given order
  (used for the constructions in the paper's proofs).
* ``gsp``       - the paper's own GSP shape (App. A): G groups of Q queries
  each; a group's prompt length cycles over a list of lengths across groups,
  a fixed share of it (the prefix ratio) is the group's shared prefix and
  the rest a fresh suffix; queries come in a random order or in the
  worst-case round-robin order (one query per group per turn, the groups in
  a fixed cycle).

Arrivals are a Poisson process (exponential gaps) unless a recipe says
otherwise; times are integer microseconds.  Output length is 4 tokens
(the paper's default) unless set.

With ``responses: True`` every path is a complete token path q_j || a_j
(Sec. 3.2 "Cache Matching and Arrival Model"): the last ``out_len[j]``
tokens are a synthetic response.  In ``sessions`` the response of a turn is
part of the next turn's prompt (a conversation carries its answers); in the
other recipes it is fresh random tokens that never recur.
"""
from __future__ import annotations

import dataclasses
from typing import Any, Dict, List, Optional, Sequence

import numpy as np


@dataclasses.dataclass
class Stream:
    tokens: np.ndarray      # int32 [T]
    offsets: np.ndarray     # uint64 [n+1]
    arrival_us: np.ndarray  # int64 [n]
    out_len: np.ndarray     # uint16 [n]
    spec: Dict[str, Any]

    @property
    def n(self) -> int:
        return int(self.arrival_us.shape[0])

    @property
    def lengths(self) -> np.ndarray:
        return np.diff(self.offsets.astype(np.int64))

    @property
    def max_len(self) -> int:
        return int(self.lengths.max()) if self.n else 0

    def query(self, j: int) -> np.ndarray:
        return self.tokens[int(self.offsets[j]):int(self.offsets[j + 1])]

    def head(self, n: int) -> "Stream":
        """The first ``n`` queries of this stream (same arrays, truncated)."""
        n = min(n, self.n)
        end = int(self.offsets[n])
        return Stream(self.tokens[:end], self.offsets[: n + 1], self.arrival_us[:n],
                      self.out_len[:n], dict(self.spec, n=n))


# ---------------------------------------------------------------------------
# helpers (sampling only)

def _zipf_cdf(g: int, s: float) -> np.ndarray:
    w = np.arange(1, g + 1, dtype=np.float64) ** (-float(s))
    c = np.cumsum(w)
    return c / c[-1]


def _zipf_draw(rng: np.random.Generator, cdf: np.ndarray, size: int) -> np.ndarray:
    u = rng.random(size)
    idx = np.searchsorted(cdf, u, side="right")
    return np.minimum(idx, cdf.shape[0] - 1).astype(np.int64)


def _poisson_times_us(rng: np.random.Generator, n: int, rate: float) -> np.ndarray:
    gaps = rng.exponential(1.0 / rate, size=n)
    return np.floor(np.cumsum(gaps) * 1e6).astype(np.int64)


def _assemble(pieces_len: np.ndarray, fill) -> (np.ndarray, np.ndarray):
    offsets = np.zeros(pieces_len.shape[0] + 1, dtype=np.uint64)
    offsets[1:] = np.cumsum(pieces_len, dtype=np.uint64)
    tokens = np.empty(int(offsets[-1]), dtype=np.int32)
    fill(tokens, offsets)
    return tokens, offsets


# ---------------------------------------------------------------------------
# recipes

def _gen_groups(sp: Dict[str, Any], rng: np.random.Generator) -> Stream:
    n, g, vocab = int(sp["n"]), int(sp["groups"]), int(sp["vocab"])
    plo, phi = sp["prefix_len"]
    slo, shi = sp["suffix_len"]
    plen = rng.integers(plo, phi + 1, size=g)
    prefixes = [rng.integers(0, vocab, size=int(l), dtype=np.int32) for l in plen]
    cdf = _zipf_cdf(g, sp["zipf_s"])
    rank = _zipf_draw(rng, cdf, n)
    perm_every = int(sp.get("permute_every", 0))
    if perm_every > 0:
        n_epochs = (n + perm_every - 1) // perm_every
        perms = [rng.permutation(g) for _ in range(n_epochs)]
        group = np.array([perms[j // perm_every][rank[j]] for j in range(n)], dtype=np.int64)
    else:
        group = rank.copy()
    rate = float(sp.get("rate", 12.0))
    burst = sp.get("burst")
    if burst:
        # two-state on/off chain: an OFF query starts a burst with probability
        # p_on; a burst is `length` consecutive queries of one Zipf group at
        # `rate` arrivals/s, then the chain returns to OFF.
        u_on = rng.random(n)
        burst_group = _zipf_draw(rng, cdf, n)
        std_gaps = rng.exponential(1.0, size=n)
        gaps = np.empty(n, dtype=np.float64)
        remaining, bg, bi = 0, 0, 0
        for j in range(n):
            if remaining == 0 and u_on[j] < burst["p_on"]:
                remaining = int(burst["length"])
                bg = burst_group[bi]
                bi += 1
            if remaining > 0:
                group[j] = bg
                gaps[j] = std_gaps[j] / burst["rate"]
                remaining -= 1
            else:
                gaps[j] = std_gaps[j] / rate
        arrival = np.floor(np.cumsum(gaps) * 1e6).astype(np.int64)
    else:
        arrival = _poisson_times_us(rng, n, rate)
    slen = rng.integers(slo, shi + 1, size=n)
    suffix_tokens = rng.integers(0, vocab, size=int(slen.sum()), dtype=np.int32)
    qlen = plen[group] + slen

    def fill(tok, off):
        so = 0
        for j in range(n):
            o = int(off[j])
            p = prefixes[group[j]]
            tok[o:o + p.shape[0]] = p
            s = int(slen[j])
            tok[o + p.shape[0]:o + p.shape[0] + s] = suffix_tokens[so:so + s]
            so += s

    tokens, offsets = _assemble(qlen, fill)
    out_len = np.full(n, int(sp.get("out_len", 4)), dtype=np.uint16)
    return Stream(tokens, offsets, arrival, out_len, sp)


def _gen_two_level(sp: Dict[str, Any], rng: np.random.Generator) -> Stream:
    n, vocab = int(sp["n"]), int(sp["vocab"])
    sysp = rng.integers(0, vocab, size=(sp["n_sys"], sp["sys_len"]), dtype=np.int32)
    task = rng.integers(0, vocab, size=(sp["n_task"], sp["task_len"]), dtype=np.int32)
    s_idx = rng.integers(0, sp["n_sys"], size=n)
    t_idx = rng.integers(0, sp["n_task"], size=n)
    slo, shi = sp["suffix_len"]
    slen = rng.integers(slo, shi + 1, size=n)
    suffix_tokens = rng.integers(0, vocab, size=int(slen.sum()), dtype=np.int32)
    arrival = _poisson_times_us(rng, n, float(sp.get("rate", 12.0)))
    a, b = int(sp["sys_len"]), int(sp["task_len"])
    qlen = a + b + slen

    def fill(tok, off):
        so = 0
        for j in range(n):
            o = int(off[j])
            tok[o:o + a] = sysp[s_idx[j]]
            tok[o + a:o + a + b] = task[t_idx[j]]
            s = int(slen[j])
            tok[o + a + b:o + a + b + s] = suffix_tokens[so:so + s]
            so += s

    tokens, offsets = _assemble(qlen, fill)
    out_len = np.full(n, int(sp.get("out_len", 4)), dtype=np.uint16)
    return Stream(tokens, offsets, arrival, out_len, sp)


def _gen_sessions(sp: Dict[str, Any], rng: np.random.Generator) -> Stream:
    ns, vocab = int(sp["n_sessions"]), int(sp["vocab"])
    tlo, thi = sp["turns"]
    elo, ehi = sp["ext_len"]
    start_len = int(sp["start_len"])
    turns = rng.integers(tlo, thi + 1, size=ns)
    ext = rng.integers(elo, ehi + 1, size=int(turns.sum()))
    if sp.get("responses"):
        # a turn's extension is followed by its response, which the next
        # turn's prompt then contains
        ext = ext + int(sp.get("out_len", 4))
    ext_off = np.zeros(ns + 1, dtype=np.int64)
    ext_off[1:] = np.cumsum(turns)
    shared_start = bool(sp.get("shared_start", False))
    # full token sequence per session: start block then every extension
    seq_len = start_len + np.add.reduceat(ext, ext_off[:-1]) if ns else np.zeros(0, np.int64)
    seq_off = np.zeros(ns + 1, dtype=np.int64)
    seq_off[1:] = np.cumsum(seq_len)
    seq = rng.integers(0, vocab, size=int(seq_off[-1]), dtype=np.int32)
    if shared_start:
        common = rng.integers(0, vocab, size=start_len, dtype=np.int32)
        for s in range(ns):
            seq[seq_off[s]:seq_off[s] + start_len] = common
    start_t = np.cumsum(rng.exponential(1.0 / sp.get("session_rate", 1.0), size=ns))
    gap = rng.exponential(1.0 / sp.get("turn_rate", 1.0), size=int(turns.sum()))
    # turn k of session s arrives at start_s + sum of the gaps before it
    t_turn = np.empty(int(turns.sum()), dtype=np.float64)
    for s in range(ns):
        a, b = ext_off[s], ext_off[s + 1]
        g = gap[a:b].copy()
        g[0] = 0.0
        t_turn[a:b] = start_t[s] + np.cumsum(g)
    t_us = np.floor(t_turn * 1e6).astype(np.int64)
    sess = np.repeat(np.arange(ns), turns)
    turn_idx = np.arange(int(turns.sum())) - ext_off[sess]
    order = np.lexsort((turn_idx, sess, t_us))
    cum = np.cumsum(ext)
    base = np.zeros(ns, dtype=np.int64)
    if ns > 1:
        base[1:] = cum[ext_off[1:-1] - 1]
    qlen_all = start_len + cum - base[sess]
    limit = sp.get("n")
    if limit is not None:
        order = order[: int(limit)]
    n = order.shape[0]
    qlen = qlen_all[order]

    def fill(tok, off):
        for q in range(n):
            k = order[q]
            s = sess[k]
            o = int(off[q])
            l = int(qlen[q])
            tok[o:o + l] = seq[seq_off[s]:seq_off[s] + l]

    tokens, offsets = _assemble(qlen, fill)
    arrival = t_us[order]
    out_len = np.full(n, int(sp.get("out_len", 4)), dtype=np.uint16)
    return Stream(tokens, offsets, arrival, out_len, dict(sp, n=n))


def _gen_gsp(sp: Dict[str, Any], rng: np.random.Generator) -> Stream:
    g, per, vocab = int(sp["groups"]), int(sp["per_group"]), int(sp["vocab"])
    lengths = [int(x) for x in sp["lengths"]]
    glen = np.array([lengths[k % len(lengths)] for k in range(g)], dtype=np.int64)
    plen = np.floor(glen * float(sp["prefix_ratio"])).astype(np.int64)
    prefixes = [rng.integers(0, vocab, size=int(l), dtype=np.int32) for l in plen]
    n = g * per
    if sp.get("order", "random") == "round_robin":
        group = np.tile(np.arange(g), per)  # turn t: groups 0..G-1
    else:
        group = rng.permutation(np.repeat(np.arange(g), per))
    limit = sp.get("n")
    if limit is not None:
        group = group[: int(limit)]
        n = group.shape[0]
    slen = glen[group] - plen[group]
    suffix_tokens = rng.integers(0, vocab, size=int(slen.sum()), dtype=np.int32)
    arrival = _poisson_times_us(rng, n, float(sp.get("rate", 12.0)))

    def fill(tok, off):
        so = 0
        for j in range(n):
            o = int(off[j])
            p = prefixes[group[j]]
            tok[o:o + p.shape[0]] = p
            s = int(slen[j])
            tok[o + p.shape[0]:o + p.shape[0] + s] = suffix_tokens[so:so + s]
            so += s

    tokens, offsets = _assemble(glen[group], fill)
    out_len = np.full(n, int(sp.get("out_len", 4)), dtype=np.uint16)
    return Stream(tokens, offsets, arrival, out_len, dict(sp, n=n))


def _gen_paths(sp: Dict[str, Any], rng: np.random.Generator) -> Stream:
    paths: List[Sequence[int]] = sp["paths"]
    order = sp.get("order")
    if order is None:
        order = list(range(len(paths)))
    if sp.get("random_order"):
        order = list(rng.integers(0, len(paths), size=int(sp["n"])))
    qs = [np.asarray(paths[k], dtype=np.int32) for k in order]
    qlen = np.array([q.shape[0] for q in qs], dtype=np.int64)

    def fill(tok, off):
        for j, q in enumerate(qs):
            tok[int(off[j]):int(off[j]) + q.shape[0]] = q

    tokens, offsets = _assemble(qlen, fill)
    n = len(qs)
    gap_us = int(sp.get("gap_us", 83333))
    arrival = np.arange(1, n + 1, dtype=np.int64) * gap_us
    out_len = np.full(n, int(sp.get("out_len", 4)), dtype=np.uint16)
    return Stream(tokens, offsets, arrival, out_len, sp)


_KINDS = {"groups": _gen_groups, "two_level": _gen_two_level,
          "sessions": _gen_sessions, "paths": _gen_paths, "gsp": _gen_gsp}


def _append_responses(st: Stream, vocab: int, rng: np.random.Generator) -> Stream:
    """Append out_len[j] fresh random response tokens to every query."""
    o = st.out_len.astype(np.int64)
    qlen = st.lengths + o
    resp = rng.integers(0, vocab, size=int(o.sum()), dtype=np.int32)

    def fill(tok, off):
        ro = 0
        for j in range(st.n):
            a, L = int(off[j]), int(st.lengths[j])
            tok[a:a + L] = st.query(j)
            tok[a + L:a + L + int(o[j])] = resp[ro:ro + int(o[j])]
            ro += int(o[j])

    tokens, offsets = _assemble(qlen, fill)
    return Stream(tokens, offsets, st.arrival_us, st.out_len, st.spec)


def generate(spec: Dict[str, Any], seed: Optional[int] = None) -> Stream:
    """Draw the stream described by ``spec`` (deterministic in ``seed``)."""
    seed = int(spec.get("seed", 0) if seed is None else seed)
    rng = np.random.default_rng(seed)
    st = _KINDS[spec["kind"]](dict(spec), rng)
    if spec.get("responses") and spec["kind"] != "sessions":
        # drawn after the prompts from a generator of their own, so the
        # prompts are those of the same spec without responses
        st = _append_responses(st, int(spec.get("vocab", 32000)), np.random.default_rng([seed, 1]))
    return st


# ---------------------------------------------------------------------------
# presets: the five benchmark configurations (simulator sizes + stream recipe)

PRESETS: Dict[int, Dict[str, Any]] = {
    1: {"name": "c1_gsp_small", "R": 1, "W": 2, "B": 2048,
        "stream": {"kind": "groups", "n": 1000, "groups": 8, "prefix_len": (64, 64),
                   "suffix_len": (32, 32), "zipf_s": 1.0, "vocab": 32000, "rate": 12.0}},
    2: {"name": "c2_gsp_drift", "R": 64, "W": 4, "B": 16384,
        "stream": {"kind": "groups", "n": 10000, "groups": 64, "prefix_len": (128, 512),
                   "suffix_len": (32, 128), "zipf_s": 1.1, "permute_every": 2000,
                   "vocab": 32000, "rate": 12.0}},
    3: {"name": "c3_two_level", "R": 256, "W": 8, "B": 65536,
        "stream": {"kind": "two_level", "n": 100000, "n_sys": 16, "sys_len": 1024,
                   "n_task": 32, "task_len": 256, "suffix_len": (64, 256),
                   "vocab": 128000, "rate": 12.0}},
    4: {"name": "c4_multiturn", "R": 128, "W": 16, "B": 131072,
        "stream": {"kind": "sessions", "n_sessions": 50000, "turns": (1, 8), "start_len": 512,
                   "ext_len": (64, 512), "session_rate": 1.0, "turn_rate": 1.0,
                   "vocab": 32000}},
    5: {"name": "c5_long_bursty", "R": 32, "W": 32, "B": 262144,
        "stream": {"kind": "groups", "n": 200000, "groups": 256, "prefix_len": (2048, 8192),
                   "suffix_len": (128, 1024), "zipf_s": 0.8, "vocab": 128000, "rate": 12.0,
                   "burst": {"p_on": 1.0 / 500.0, "length": 500, "rate": 120.0}}},
    # the paper's GSP setting (App. A): 128 groups x 32 queries, prompt
    # lengths cycling over 512..8192 across groups, prefix ratio 0.5, 4
    # workers with about 200k cached tokens each, 12 req/s; random order and
    # the worst-case round-robin order (context runs, not benchmark lines)
    6: {"name": "gsp_paper_random", "R": 64, "W": 4, "B": 200000,
        "stream": {"kind": "gsp", "groups": 128, "per_group": 32, "lengths": (512, 1024, 2048, 4096, 8192),
                   "prefix_ratio": 0.5, "order": "random", "vocab": 32000, "rate": 12.0}},
    7: {"name": "gsp_paper_round_robin", "R": 64, "W": 4, "B": 200000,
        "stream": {"kind": "gsp", "groups": 128, "per_group": 32, "lengths": (512, 1024, 2048, 4096, 8192),
                   "prefix_ratio": 0.5, "order": "round_robin", "vocab": 32000, "rate": 12.0}},
}


def preset_spec(cfg: int, **stream_overrides) -> Dict[str, Any]:
    p = PRESETS[cfg]
    out = dict(p)
    out["stream"] = dict(p["stream"], **stream_overrides)
    return out


def small_spec(n: int = 200, groups: int = 6, prefix_len=(8, 40), suffix_len=(4, 24),
               zipf_s: float = 1.0, vocab: int = 50, rate: float = 12.0, **kw) -> Dict[str, Any]:
    """A small GSP-like stream for parity tests (short paths, small vocab so
    that suffixes also collide and the trie branches at many depths)."""
    sp = {"kind": "groups", "n": n, "groups": groups, "prefix_len": tuple(prefix_len),
          "suffix_len": tuple(suffix_len), "zipf_s": zipf_s, "vocab": vocab, "rate": rate}
    sp.update(kw)
    return sp
