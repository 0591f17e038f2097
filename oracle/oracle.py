"""ctypes front end of the CPU oracle (test infrastructure only).

Only ``tests/``, the smoke entry point and the benchmark's CPU-baseline leg
may use this module.  It never touches the HIP library and the HIP library
never touches it: the two share only the seeded streams from ``workload``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Any, Dict, Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "kvr_oracle.cpp")
LIB = os.path.join(HERE, "liboracle.so")

EVICT = {"rlt": 0, "lru": 1}
UPDATE = {"nlms": 0, "rls": 1, "none": 2}


class OrcConfig(ctypes.Structure):
    _fields_ = [
        ("num_workers", ctypes.c_uint32),
        ("cache_tokens", ctypes.c_uint32),
        ("seed", ctypes.c_uint64),
        ("evict", ctypes.c_int32),
        ("update", ctypes.c_int32),
        ("u_mode", ctypes.c_int32),
        ("check", ctypes.c_int32),
        ("alpha_cached", ctypes.c_double),
        ("alpha_miss", ctypes.c_double),
        ("rho", ctypes.c_double),
        ("decay_interval_us", ctypes.c_int64),
        ("lr", ctypes.c_double),
        ("nlms_eps", ctypes.c_double),
        ("rls_p0", ctypes.c_double),
        ("true_cached_us", ctypes.c_int64),
        ("true_miss_us", ctypes.c_int64),
        ("true_out_us", ctypes.c_int64),
        ("router", ctypes.c_int32),
        ("ca_balance_abs", ctypes.c_int32),
        ("ca_balance_rel", ctypes.c_double),
        ("ca_cache_threshold", ctypes.c_double),
        ("cache_responses", ctypes.c_int32),
        ("batch_size", ctypes.c_int32),
        ("router_tree", ctypes.c_int32),
        ("router_tree_tokens", ctypes.c_uint32),
    ]


_U64 = ["routed", "prompt_tokens", "hit_tokens", "matched_tokens", "loads", "evictions",
        "phase", "cnt", "forced_resets", "resident", "digest_sum", "digest_xor",
        "marked_count", "marked_sum", "completions", "pending_depth", "pending_max",
        "latency_sum_us", "latency_max_us"]


_ROUTER_U64 = ["router_resident", "router_digest_sum", "router_digest_xor", "router_evictions"]


class OrcWorkerStats(ctypes.Structure):
    _fields_ = ([(n, ctypes.c_uint64) for n in _U64]
                + [("backlog_us", ctypes.c_int64), ("last_decay_us", ctypes.c_int64),
                   ("load_est", ctypes.c_double), ("theta", ctypes.c_double * 4)]
                + [(n, ctypes.c_uint64) for n in _ROUTER_U64])


class OrcRunOpts(ctypes.Structure):
    _fields_ = [
        ("snap_every", ctypes.c_uint64),
        ("snaps", ctypes.c_void_p),
        ("time_from", ctypes.c_uint64),
        ("time_budget_s", ctypes.c_double),
        ("window_cpu_s", ctypes.c_double),
        ("window_wall_s", ctypes.c_double),
        ("done", ctypes.c_uint64),
    ]


def build(force: bool = False, sanitize: bool = False) -> str:
    """Compile the oracle with g++ (plain C++17, no FMA contraction); with
    sanitize, an AddressSanitizer + UndefinedBehaviorSanitizer build (load it
    in a process that preloads the ASan runtime)."""
    out = LIB if not sanitize else LIB.replace(".so", "_asan.so")
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(SRC):
        tmp = f"{out}.{os.getpid()}.tmp"
        flags = ["-std=c++17", "-O2", "-ffp-contract=off", "-fPIC", "-shared"]
        if sanitize:
            flags += ["-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
        subprocess.check_call(["g++", *flags, "-o", tmp, SRC])
        os.replace(tmp, out)
    return out


_lib: Optional[ctypes.CDLL] = None


def _bind(l: ctypes.CDLL) -> ctypes.CDLL:
    l.orc_run.restype = ctypes.c_int
    l.orc_run.argtypes = [ctypes.POINTER(OrcConfig), ctypes.c_uint32, ctypes.c_uint64,
                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                          ctypes.POINTER(OrcWorkerStats)]
    l.orc_run_ex.restype = ctypes.c_int
    l.orc_run_ex.argtypes = list(l.orc_run.argtypes) + [ctypes.POINTER(OrcRunOpts)]
    l.orc_check_selftest.restype = ctypes.c_int
    l.orc_check_selftest.argtypes = [ctypes.c_int]
    l.orc_philox4x64_10.restype = None
    l.orc_philox4x64_10.argtypes = [ctypes.c_void_p] * 3
    l.orc_pow_int.restype = ctypes.c_double
    l.orc_pow_int.argtypes = [ctypes.c_double, ctypes.c_uint64]
    return l


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        _lib = _bind(ctypes.CDLL(build()))
    return _lib


def use_library(path: str) -> None:
    """Route every call of this module to another build of the oracle (the
    sanitized one)."""
    global _lib
    _lib = _bind(ctypes.CDLL(path))


DEFAULTS: Dict[str, Any] = dict(
    seed=0, evict="rlt", update="nlms", u_mode=0, check=0,
    alpha_cached=0.0, alpha_miss=1.0, rho=31.0 / 32.0, decay_interval_us=20000,
    lr=0.992, nlms_eps=1e-9, rls_p0=100.0,
    true_cached_us=0, true_miss_us=1000, true_out_us=10000,
    router="lbgr", ca_balance_abs=32, ca_balance_rel=1.0001, ca_cache_threshold=0.5,
    cache_responses=0, batch_size=1, router_tree=0, router_tree_tokens=0)

ROUTER = {"lbgr": 0, "random": 1, "round_robin": 2, "cache_aware": 3}


def make_config(W: int, B: int, **kw) -> OrcConfig:
    p = dict(DEFAULTS)
    p.update(kw)
    c = OrcConfig()
    c.num_workers = W
    c.cache_tokens = B
    c.seed = int(p["seed"])
    c.evict = EVICT[p["evict"]] if isinstance(p["evict"], str) else int(p["evict"])
    c.update = UPDATE[p["update"]] if isinstance(p["update"], str) else int(p["update"])
    c.u_mode = int(p["u_mode"])
    c.check = int(p["check"])
    for f in ("alpha_cached", "alpha_miss", "rho", "lr", "nlms_eps", "rls_p0"):
        setattr(c, f, float(p[f]))
    for f in ("decay_interval_us", "true_cached_us", "true_miss_us", "true_out_us"):
        setattr(c, f, int(p[f]))
    c.router = ROUTER[p["router"]] if isinstance(p["router"], str) else int(p["router"])
    c.ca_balance_abs = int(p["ca_balance_abs"])
    c.ca_balance_rel = float(p["ca_balance_rel"])
    c.ca_cache_threshold = float(p["ca_cache_threshold"])
    c.cache_responses = int(p["cache_responses"])
    c.batch_size = int(p["batch_size"])
    c.router_tree = int(p["router_tree"])
    c.router_tree_tokens = int(p["router_tree_tokens"])
    return c


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _worker_dict(s) -> Dict[str, Any]:
    d = {name: int(getattr(s, name)) for name in _U64}
    d["backlog_us"] = int(s.backlog_us)
    d["last_decay_us"] = int(s.last_decay_us)
    d["load_est"] = float(s.load_est)
    d["theta"] = [float(x) for x in s.theta]
    for name in _ROUTER_U64:
        d[name] = int(getattr(s, name))
    return d


def run(stream, W: int, B: int, replica: int = 0, n: Optional[int] = None,
        all_hits: bool = False, snap_every: int = 0, time_from: Optional[int] = None,
        time_budget_s: float = 0.0, **kw) -> Dict[str, Any]:
    """Run one replica of the simulation over the first ``n`` queries.

    ``snap_every`` > 0 adds ``snaps``: the per-worker state after every
    ``snap_every`` queries (and after the last).  ``time_from`` times the
    queries from that index on (``window_cpu_s``, ``window_wall_s``; with
    ``time_budget_s`` > 0 the run stops once they took that much CPU time,
    and ``done`` says how many queries ran)."""
    cfg = make_config(W, B, **kw)
    n = stream.n if n is None else min(int(n), stream.n)
    tokens = np.ascontiguousarray(stream.tokens, dtype=np.int32)
    offsets = np.ascontiguousarray(stream.offsets, dtype=np.uint64)
    arrival = np.ascontiguousarray(stream.arrival_us, dtype=np.int64)
    out_len = np.ascontiguousarray(stream.out_len, dtype=np.uint16)
    route = np.zeros(n, dtype=np.int32)
    hits = np.zeros(n, dtype=np.int32)
    ah = np.zeros((n, W), dtype=np.int32) if all_hits else None
    ws = (OrcWorkerStats * W)()
    opts = OrcRunOpts()
    nsnap = (n + snap_every - 1) // snap_every if snap_every > 0 else 0
    snaps = (OrcWorkerStats * max(1, nsnap * W))()
    opts.snap_every = int(snap_every)
    opts.snaps = ctypes.cast(snaps, ctypes.c_void_p) if nsnap else None
    opts.time_from = n if time_from is None else int(time_from)
    opts.time_budget_s = float(time_budget_s)
    rc = lib().orc_run_ex(ctypes.byref(cfg), replica, n, _ptr(tokens), _ptr(offsets), _ptr(arrival),
                          _ptr(out_len), _ptr(route), _ptr(hits), _ptr(ah), ws, ctypes.byref(opts))
    done = int(opts.done)
    out = {"rc": rc, "route": route[:done], "hits": hits[:done],
           "all_hits": None if ah is None else ah[:done],
           "workers": [_worker_dict(ws[i]) for i in range(W)], "done": done,
           "window_cpu_s": float(opts.window_cpu_s), "window_wall_s": float(opts.window_wall_s)}
    if nsnap:
        out["snaps"] = [[_worker_dict(snaps[k * W + i]) for i in range(W)]
                        for k in range((done + snap_every - 1) // snap_every)]
    return out


def check_selftest(which: int) -> bool:
    """True when the oracle's invariant checks catch planted violation
    ``which`` (1: negative load estimate, 2: a non-routed cache changed,
    3: a token whose parent is gone)."""
    return bool(lib().orc_check_selftest(int(which)))


def philox4x64_10(counter, key) -> np.ndarray:
    c = np.asarray(counter, dtype=np.uint64)
    k = np.asarray(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    lib().orc_philox4x64_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def pow_int(rho: float, k: int) -> float:
    return float(lib().orc_pow_int(rho, k))
