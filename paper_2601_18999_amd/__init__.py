"""Python binding of libkvr (include/kvr.h): batched KV-cache routing and
eviction on MI355X.

The functions below carry the C ABI's names and only marshal arguments;
every step of the simulation runs in the HIP kernels of libkvr.so.  torch is
used for device memory and streams only.  The library must be built
(``python -m paper_2601_18999_amd.build``); nothing falls back to the CPU.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkvr.so")

KVR_OK, KVR_EINVAL, KVR_ENOMEM, KVR_EDEVICE, KVR_ECAPACITY, KVR_ESTATE = 0, -1, -2, -3, -4, -5
STATUS_NAMES = {0: "KVR_OK", -1: "KVR_EINVAL", -2: "KVR_ENOMEM", -3: "KVR_EDEVICE",
                -4: "KVR_ECAPACITY", -5: "KVR_ESTATE"}
KVR_EVICT_RLT, KVR_EVICT_LRU = 0, 1
KVR_ROUTE_LBGR, KVR_ROUTE_RANDOM, KVR_ROUTE_ROUND_ROBIN, KVR_ROUTE_CACHE_AWARE = 0, 1, 2, 3
KVR_UPD_NLMS, KVR_UPD_RLS, KVR_UPD_NONE = 0, 1, 2
KVR_ABI_VERSION = 8
KVR_PHASES = 18
PHASE_NAMES = ["route", "stage_wait", "mark", "load", "evict", "finish", "match", "join", "evictor_wait",
               "e_evict", "e_finish", "e_idle", "h_stage", "h_wait", "h_draw", "h_other", "h_match",
               "e_match"]

EXPORTED = ["kvr_config_default", "kvr_workspace_size", "kvr_init_replicas", "kvr_route_batch",
            "kvr_stats", "kvr_stats_noalloc", "kvr_check", "kvr_queries_done", "kvr_destroy", "kvr_last_error"]


class KvrConfig(ctypes.Structure):
    _fields_ = [
        ("abi_version", ctypes.c_uint32),
        ("struct_size", ctypes.c_uint32),
        ("num_replicas", ctypes.c_uint32),
        ("num_workers", ctypes.c_uint32),
        ("cache_tokens", ctypes.c_uint32),
        ("max_query_tokens", ctypes.c_uint32),
        ("seed", ctypes.c_uint64),
        ("evict", ctypes.c_int32),
        ("router", ctypes.c_int32),
        ("update", ctypes.c_int32),
        ("pending_capacity", ctypes.c_uint32),
        ("node_capacity", ctypes.c_uint32),
        ("arena_words", ctypes.c_uint32),
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
        ("ca_balance_abs", ctypes.c_int32),
        ("pad0", ctypes.c_int32),
        ("ca_balance_rel", ctypes.c_double),
        ("ca_cache_threshold", ctypes.c_double),
        ("cache_responses", ctypes.c_int32),
        ("batch_size", ctypes.c_int32),
        ("router_tree", ctypes.c_int32),
        ("router_tree_tokens", ctypes.c_uint32),
        ("phase_timers", ctypes.c_int32),
        ("pad1", ctypes.c_uint32),
    ]


STAT_U64 = ["routed", "prompt_tokens", "hit_tokens", "matched_tokens", "loads", "evictions",
            "phase", "cnt", "forced_resets", "resident", "digest_sum", "digest_xor",
            "marked_count", "marked_sum", "completions", "pending_depth", "pending_max",
            "latency_sum_us", "latency_max_us"]


ROUTER_U64 = ["router_resident", "router_digest_sum", "router_digest_xor", "router_evictions"]


class KvrWorkerStats(ctypes.Structure):
    _fields_ = ([(n, ctypes.c_uint64) for n in STAT_U64]
                + [("backlog_us", ctypes.c_int64), ("last_decay_us", ctypes.c_int64),
                   ("load_est", ctypes.c_double), ("theta", ctypes.c_double * 4),
                   ("nodes", ctypes.c_uint64), ("gc_runs", ctypes.c_uint64)]
                + [(n, ctypes.c_uint64) for n in ROUTER_U64])


REPLICA_U64 = ["queries", "route_digest", "prompt_tokens", "hit_tokens", "matched_tokens", "loads",
               "evictions", "completions", "latency_sum_us", "latency_max_us"]


class KvrReplicaStats(ctypes.Structure):
    _fields_ = ([(n, ctypes.c_uint64) for n in REPLICA_U64]
                + [("last_arrival_us", ctypes.c_int64), ("phase_ticks", ctypes.c_uint64 * KVR_PHASES)])


class KvrError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib: Optional[ctypes.CDLL] = None


def load_library() -> ctypes.CDLL:
    """Load libkvr.so (after torch, so both share one HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_2601_18999_amd.build`")
    try:
        import torch  # noqa: F401  (loads the HIP runtime this library binds to)
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    vp, u32, u64 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64
    lib.kvr_config_default.restype = None
    lib.kvr_config_default.argtypes = [ctypes.POINTER(KvrConfig), u32, u32, u32, u32]
    lib.kvr_workspace_size.restype = ctypes.c_int
    lib.kvr_workspace_size.argtypes = [ctypes.POINTER(KvrConfig), ctypes.POINTER(ctypes.c_size_t)]
    lib.kvr_init_replicas.restype = ctypes.c_int
    lib.kvr_init_replicas.argtypes = [ctypes.POINTER(KvrConfig), vp, ctypes.c_size_t, vp,
                                      ctypes.POINTER(vp)]
    lib.kvr_route_batch.restype = ctypes.c_int
    lib.kvr_route_batch.argtypes = [vp, u32, vp, vp, vp, vp, vp, vp, vp]
    lib.kvr_stats.restype = ctypes.c_int
    lib.kvr_stats.argtypes = [vp, ctypes.POINTER(KvrReplicaStats), ctypes.c_size_t,
                              ctypes.POINTER(KvrWorkerStats), ctypes.c_size_t]
    lib.kvr_stats_noalloc.restype = ctypes.c_int
    lib.kvr_stats_noalloc.argtypes = [vp, ctypes.POINTER(KvrReplicaStats), ctypes.c_size_t,
                                      ctypes.POINTER(KvrWorkerStats), ctypes.c_size_t]
    lib.kvr_check.restype = ctypes.c_int
    lib.kvr_check.argtypes = [vp, ctypes.POINTER(u32)]
    lib.kvr_queries_done.restype = u64
    lib.kvr_queries_done.argtypes = [vp]
    lib.kvr_destroy.restype = None
    lib.kvr_destroy.argtypes = [vp]
    lib.kvr_last_error.restype = ctypes.c_char_p
    lib.kvr_last_error.argtypes = []
    _lib = lib
    return lib


def kvr_last_error() -> str:
    return load_library().kvr_last_error().decode()


def _check(st: int, where: str) -> None:
    if st != KVR_OK:
        raise KvrError(st, where, kvr_last_error())


def kvr_config_default(R: int, W: int, B: int, max_query_tokens: int, **overrides) -> KvrConfig:
    cfg = KvrConfig()
    load_library().kvr_config_default(ctypes.byref(cfg), R, W, B, max_query_tokens)
    for k, v in overrides.items():
        if not hasattr(cfg, k):
            raise AttributeError(k)
        setattr(cfg, k, v)
    return cfg


def kvr_workspace_size(cfg: KvrConfig) -> int:
    n = ctypes.c_size_t(0)
    _check(load_library().kvr_workspace_size(ctypes.byref(cfg), ctypes.byref(n)), "kvr_workspace_size")
    return int(n.value)


def kvr_init_replicas(cfg: KvrConfig, d_workspace: int, nbytes: int, stream: int = 0) -> int:
    ctx = ctypes.c_void_p(None)
    _check(load_library().kvr_init_replicas(ctypes.byref(cfg), ctypes.c_void_p(d_workspace), nbytes,
                                            ctypes.c_void_p(stream or None), ctypes.byref(ctx)),
           "kvr_init_replicas")
    return int(ctx.value)


def kvr_route_batch(ctx: int, n: int, d_tokens: int, d_offsets: int, d_arrival_us: int,
                    d_out_len: int = 0, d_route: int = 0, d_hits: int = 0, d_all_hits: int = 0) -> None:
    vp = ctypes.c_void_p
    _check(load_library().kvr_route_batch(vp(ctx), n, vp(d_tokens), vp(d_offsets), vp(d_arrival_us),
                                          vp(d_out_len or None), vp(d_route or None),
                                          vp(d_hits or None), vp(d_all_hits or None)),
           "kvr_route_batch")


def _stats_dicts(arr, n: int) -> List[Dict]:
    out = []
    for k in range(n):
        s = arr[k]
        d = {name: int(getattr(s, name)) for name in STAT_U64}
        d["backlog_us"] = int(s.backlog_us)
        d["last_decay_us"] = int(s.last_decay_us)
        d["load_est"] = float(s.load_est)
        d["theta"] = [float(x) for x in s.theta]
        d["nodes"] = int(s.nodes)
        d["gc_runs"] = int(s.gc_runs)
        for name in ROUTER_U64:
            d[name] = int(getattr(s, name))
        out.append(d)
    return out


def _replica_dicts(arr, n: int) -> List[Dict]:
    out = []
    for k in range(n):
        s = arr[k]
        d = {name: int(getattr(s, name)) for name in REPLICA_U64}
        d["last_arrival_us"] = int(s.last_arrival_us)
        d["phase_ticks"] = [int(x) for x in s.phase_ticks]
        out.append(d)
    return out


def kvr_stats(ctx: int, R: int, W: int, check: bool = True, with_replicas: bool = False):
    """Per-worker records as [R][W] dicts; with ``with_replicas`` also the
    per-replica records: (replicas [R], workers [R][W])."""
    arr = (KvrWorkerStats * (R * W))()
    rep = (KvrReplicaStats * R)() if with_replicas else None
    st = load_library().kvr_stats(ctypes.c_void_p(ctx), rep, R if with_replicas else 0, arr, R * W)
    if check:
        _check(st, "kvr_stats")
    flat = _stats_dicts(arr, R * W)
    workers = [flat[r * W:(r + 1) * W] for r in range(R)]
    if with_replicas:
        return _replica_dicts(rep, R), workers
    return workers


def kvr_stats_noalloc(ctx: int, R: int, W: int, check: bool = True):
    """kvr_stats without any allocation by the library: (replicas [R],
    workers [R][W])."""
    arr = (KvrWorkerStats * (R * W))()
    rep = (KvrReplicaStats * R)()
    st = load_library().kvr_stats_noalloc(ctypes.c_void_p(ctx), rep, R, arr, R * W)
    if check:
        _check(st, "kvr_stats_noalloc")
    flat = _stats_dicts(arr, R * W)
    return _replica_dicts(rep, R), [flat[r * W:(r + 1) * W] for r in range(R)]


def kvr_check(ctx: int) -> (int, int):
    bits = ctypes.c_uint32(0)
    st = load_library().kvr_check(ctypes.c_void_p(ctx), ctypes.byref(bits))
    return int(st), int(bits.value)


def kvr_queries_done(ctx: int) -> int:
    return int(load_library().kvr_queries_done(ctypes.c_void_p(ctx)))


def kvr_destroy(ctx: int) -> None:
    if ctx:
        load_library().kvr_destroy(ctypes.c_void_p(ctx))


from .sim import Simulator  # noqa: E402,F401
