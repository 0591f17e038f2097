#!/usr/bin/env python3
"""Benchmark: batched KV-cache routing (LBGR) + RLT eviction on one MI355X.

A step is one kvr_route_batch call: one batch of `--batch` queries of the
synthetic stream, routed for every replica (completions and decay, the match
on every worker, LBGR score/argmin/commit, RLT insertion).  The first
`--warmup` batches fill the caches; the next `--steps` batches are the timed
window (events on the library's stream, with the stream and workspace
already resident in HBM).  The rest of the stream is then routed too, so the
line also reports the whole stream's rate.  The CPU oracle is timed on the
same window of the same stream (run untimed up to its first query).  Prints
one JSON line.

Default workload: the largest configuration (32 replicas x 32 workers,
262,144-token caches, prompts of 2,176-9,216 tokens from 256 Zipf groups in
on/off bursts).  Other configurations: --config 1..5.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E


def _code_only(text: str) -> str:
    """C/C++ source without comments and with whitespace collapsed, so that a
    comment edit does not count as a kernel change."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in sorted(os.listdir(os.path.join(ROOT, "paper_2601_18999_amd", "csrc"))):
        with open(os.path.join(ROOT, "paper_2601_18999_amd", "csrc", f), encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def load_traffic(workload: str, batch: int, warmup: int, steps: int):
    """HBM bytes per step-kernel launch measured by rocprofv3 counters, if
    they were taken on the current kernel sources over the same window
    (batch size, warm-up and timed batches)."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source_hash") != kernel_source_hash():
        return None
    if (t.get("batch"), t.get("warmup"), t.get("steps")) != (batch, warmup, steps):
        return None
    return t


def totals(stats):
    keys = ("matched_tokens", "prompt_tokens", "hit_tokens", "loads", "evictions", "routed")
    return {k: sum(w[k] for rr in stats for w in rr) for k in keys}


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def host_cores() -> int:
    """Cores for the CPU leg: this process's CPU affinity, at most 16 (one
    GPU's share of its host)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(stream, W, B, q0: int, q1: int, budget_s: float, replicas: int, evict: str = "rlt",
                 router: str = "lbgr", responses: int = 0, beta: int = 1, router_tree: int = 0,
                 router_tree_tokens: int = 0):
    """The CPU oracle on the host's cores, on the GPU's timed window: one
    single-threaded oracle run per replica, as many replicas at once as there
    are cores (its C entry point releases the GIL).  Each run goes untimed
    through queries [0, q0), then times queries q0, q0+1, ... (thread CPU
    time and wall time) until the window [q0, q1) ends or the timed part has
    taken budget_s of CPU time.  1-core rate = timed queries / timed CPU
    seconds, summed over the threads; all-core rate = the sum of the
    threads' timed queries / wall seconds (they run concurrently)."""
    from concurrent.futures import ThreadPoolExecutor
    from oracle import oracle as O
    O.lib()  # built and loaded once, before the threads
    threads = max(1, min(replicas, host_cores()))

    def one(r: int):
        o = O.run(stream, W, B, replica=r, n=q1, time_from=q0, time_budget_s=budget_s, evict=evict,
                  router=router, cache_responses=responses, batch_size=beta, router_tree=router_tree,
                  router_tree_tokens=router_tree_tokens)
        assert o["rc"] == 0, (r, o["rc"])
        return o["done"] - q0, o["window_cpu_s"], o["window_wall_s"]

    t0 = time.perf_counter()
    with ThreadPoolExecutor(max_workers=threads) as ex:
        res = list(ex.map(one, range(threads)))
    dt = time.perf_counter() - t0
    nq = sum(r[0] for r in res)
    cpu = sum(r[1] for r in res)
    agg = sum(r[0] / r[2] for r in res if r[2] > 0)
    qmin, qmax = min(r[0] for r in res), max(r[0] for r in res)
    log(f"cpu oracle: {threads} replicas, queries {q0}..{q0 + qmin}-{q0 + qmax} timed "
        f"({cpu:.1f} CPU s), {dt:.1f} s in all")
    return {"value": agg, "unit": "queries/s", "cores": threads, "kind": "oracle",
            "per_core": nq / cpu if cpu > 0 else None, "cpu_model": cpu_model(),
            "sample": f"replicas 0..{threads - 1}, one thread each; queries [0, {q0}) untimed, then "
                      f"{qmin}..{qmax} queries of the GPU's timed window from query {q0} on, "
                      f"{cpu:.1f} CPU s timed in all"}


def _pmc_rows(path: str, counter: str):
    """(dispatch id, kernel name, value) of one counter from a rocprofv3 CSV."""
    import csv
    rows = []
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            if r.get("Counter_Name") == counter:
                rows.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
    rows.sort()
    return rows


def traffic_from(args) -> int:
    """HBM bytes per timed step-kernel launch: the counters (KiB per
    dispatch) of the timed launches, each scaled by what the same counter
    reads for the plain copy of --copy-probe-mib MiB."""
    from workload import PRESETS
    workload = PRESETS[args.config]["name"]
    probe = args.copy_probe_mib << 20
    if probe <= 0:
        print("--traffic-from needs the --copy-probe-mib of the profiled runs", file=sys.stderr)
        return 2
    out = {"kernel_source_hash": kernel_source_hash(), "workload": workload, "batch": args.batch,
           "steps": args.steps, "warmup": args.warmup, "copy_probe_bytes": probe}
    per = {}
    for path, counter in zip(args.traffic_from, ("FETCH_SIZE", "WRITE_SIZE")):
        rows = _pmc_rows(path, counter)
        step = [v for _, name, v in rows if "step_kernel" in name]
        if len(step) < args.warmup + args.steps:
            print(f"{path}: {len(step)} step-kernel dispatches, expected at least {args.warmup + args.steps}",
                  file=sys.stderr)
            return 1
        timed = step[args.warmup:args.warmup + args.steps]
        # the probe: the last other dispatch whose count is near the probe size
        cand = [v for _, name, v in rows if "kvr::" not in name and 0.5 * probe <= v * 1024 <= 2 * probe]
        if not cand:
            print(f"{path}: no copy-probe dispatch found", file=sys.stderr)
            return 1
        factor = cand[-1] * 1024 / probe
        per[counter] = {"kib_per_launch": sum(timed) / len(timed), "probe_kib": cand[-1], "factor": factor,
                        "bytes_per_launch": sum(timed) / len(timed) * 1024 / factor}
    out["counters"] = per
    out["bytes_per_launch"] = per["FETCH_SIZE"]["bytes_per_launch"] + per["WRITE_SIZE"]["bytes_per_launch"]
    dst = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    with open(dst, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--batch", type=int, default=2000)
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--evict", choices=["rlt", "lru"], default="rlt",
                    help="eviction policy: RLT (the method) or L-LRU (its baseline)")
    ap.add_argument("--router", choices=["lbgr", "random", "round_robin", "cache_aware"], default="lbgr",
                    help="router: LBGR (the method) or one of its baselines")
    ap.add_argument("--responses", action="store_true",
                    help="cache complete token paths q||a (each query followed by its response; in the "
                         "multi-turn workload a turn's response is part of the next prompt)")
    ap.add_argument("--beta", type=int, default=1,
                    help="continuous batching: the batch size beta (the last beta-1 paths routed to a "
                         "worker are never evicted); 1 = single-query processing")
    ap.add_argument("--router-tree", action="store_true",
                    help="approximate router: the router scores with matches on L-LRU trees of its own "
                         "(one per worker, the routed prompts) instead of the workers' caches")
    ap.add_argument("--router-tree-tokens", type=int, default=0, help="budget of each router tree (0 = B)")
    ap.add_argument("--replicas", type=int, default=0,
                    help="replicas of the workload's shape on the GPU (0 = the configuration's R); a "
                         "scaling measurement, not a configuration's line")
    ap.add_argument("--arena-words", type=int, default=0,
                    help="arena words per semispace per (replica, worker) (0 = the library's default)")
    ap.add_argument("--pending-capacity", type=int, default=0,
                    help="completion records per (replica, worker) (0 = the library's default)")
    ap.add_argument("--cpu-budget", type=float, default=10.0,
                    help="CPU seconds per oracle thread on the timed window")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--phase-timers", action="store_true",
                    help="build the step kernel with per-part timers of the routing wave and report the "
                         "microseconds per query and replica of each part over the timed window")
    ap.add_argument("--no-whole", action="store_true",
                    help="stop after the timed window instead of routing the rest of the stream")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after the timed region, copy this many MiB device to device with a plain "
                         "copy kernel (the calibration run for rocprofv3 byte counters)")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="compute HBM bytes per step-kernel launch from two rocprofv3 --pmc runs "
                         "(FETCH_SIZE, WRITE_SIZE) of this benchmark with --copy-probe-mib, and "
                         "write profiles/traffic_<workload>.json")
    args = ap.parse_args()
    if args.traffic_from:
        return traffic_from(args)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus > 1 or world > 1:
        print("bench.py runs on one GPU only: replicas are independent, and this build measures "
              "one GPU's share; multi-GPU sharding over replicas is not built. Use --gpus 1.",
              file=sys.stderr)
        return 2

    import torch
    import paper_2601_18999_amd as K
    from workload import PRESETS, generate

    p = PRESETS[args.config]
    R, W, B = p["R"], p["W"], p["B"]
    if args.replicas:
        R = args.replicas
    t0 = time.perf_counter()
    stream = generate(dict(p["stream"], responses=True) if args.responses else p["stream"])
    log(f"{p['name']}: {stream.n} queries, {stream.tokens.size} tokens ({time.perf_counter() - t0:.1f} s)")
    need = (args.warmup + args.steps) * args.batch
    if need > stream.n:
        print(f"warmup+steps need {need} queries, the stream has {stream.n}", file=sys.stderr)
        return 2
    dev = torch.device("cuda:0")
    evict = {"rlt": K.KVR_EVICT_RLT, "lru": K.KVR_EVICT_LRU}[args.evict]
    router = {"lbgr": K.KVR_ROUTE_LBGR, "random": K.KVR_ROUTE_RANDOM, "round_robin": K.KVR_ROUTE_ROUND_ROBIN,
              "cache_aware": K.KVR_ROUTE_CACHE_AWARE}[args.router]
    sim = K.Simulator(R, W, B, stream.max_len, device="cuda:0", evict=evict, router=router,
                      cache_responses=int(args.responses), batch_size=args.beta,
                      router_tree=int(args.router_tree), router_tree_tokens=args.router_tree_tokens,
                      phase_timers=int(args.phase_timers), arena_words=args.arena_words,
                      **({"pending_capacity": args.pending_capacity} if args.pending_capacity else {}))
    ds = sim.upload(stream)
    out = sim.alloc_outputs(args.batch)
    torch.cuda.synchronize()

    log(f"workspace {sim.nbytes / 1e9:.1f} GB, stream resident")
    nb = (stream.n + args.batch - 1) // args.batch  # batches in the whole stream
    # every batch is timed with events on the library's stream; the metric
    # is the window [warmup, warmup + steps), the rest of the stream follows
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(nb)]

    def run_batch(k: int) -> None:
        b0 = k * args.batch
        m = min(args.batch, stream.n - b0)
        ev[k][0].record(sim.stream)
        sim.route(ds, b0, m, out=out if m == args.batch else None)
        ev[k][1].record(sim.stream)

    for k in range(args.warmup):
        run_batch(k)
        torch.cuda.synchronize()
        log(f"warmup batch {k + 1}/{args.warmup} done")
    reps0, ws0 = sim.replica_stats()
    before = totals(ws0)
    q0 = args.warmup * args.batch
    q = q0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.warmup, args.warmup + args.steps):
        run_batch(k)
        q += args.batch
        ev[k][1].synchronize()
        log(f"timed batch {k + 1 - args.warmup}/{args.steps}: {ev[k][0].elapsed_time(ev[k][1]):.1f} ms")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    st, bits = sim.check()
    if st != K.KVR_OK:
        print(f"device status {st} bits {bits}: {K.kvr_last_error()}", file=sys.stderr)
        return 1
    reps1, ws1 = sim.replica_stats()
    after = totals(ws1)
    d = {k: after[k] - before[k] for k in after}
    kernel_ms = sum(ev[k][0].elapsed_time(ev[k][1]) for k in range(args.warmup, args.warmup + args.steps))
    nq = R * (q - q0)
    paths = stream.lengths[q0:q].astype("int64")
    path_tokens = int(paths.sum()) * R
    prompt = path_tokens - (int(stream.out_len[q0:q].astype("int64").sum()) * R if args.responses else 0)
    assert prompt == d["prompt_tokens"]
    # algorithmic bytes of the timed launches: query (path) staging, edge
    # tokens compared on every worker (every h_ij, as a full walk reads
    # them), edge tokens written for loaded tokens, one candidate/node
    # read-modify-write per eviction, LBGR + completion record
    alg_bytes = (4 * path_tokens + 4 * d["matched_tokens"] + 4 * d["loads"] + 32 * d["evictions"]
                 + 96 * nq)
    achieved = alg_bytes / (kernel_ms * 1e-3) / 1e9
    workload = p["name"]
    default_run = (args.evict, args.router, args.responses, args.beta, args.router_tree, args.replicas,
                   args.arena_words, args.pending_capacity) == ("rlt", "lbgr", False, 1, False, 0, 0, 0)
    traffic = load_traffic(workload, args.batch, args.warmup, args.steps) if default_run else None
    launch_s = kernel_ms * 1e-3 / args.steps
    line = {
        "metric": "routed queries/sec",
        "value": nq / (kernel_ms * 1e-3),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": kernel_ms / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i32+f64",
        "data": "synthetic",
        "config": {"workload": workload + ("_responses" if args.responses else ""), "eviction": args.evict,
                   "router": args.router, "cached_responses": bool(args.responses), "batch_size": args.beta,
                   "router_tree": bool(args.router_tree), "router_tree_tokens": args.router_tree_tokens or None,
                   "replicas": R, "arena_words": args.arena_words or None,
                   "workers": W, "cache_tokens": B,
                   "batch_queries": args.batch, "timed_queries": q - q0,
                   "first_timed_query": q0, "stream_queries": stream.n},
        "prefix_matched_tokens_per_s": d["matched_tokens"] / (kernel_ms * 1e-3),
        "routed_hit_tokens_per_s": d["hit_tokens"] / (kernel_ms * 1e-3),
        "evictions_per_s": d["evictions"] / (kernel_ms * 1e-3),
        "hit_rate": d["hit_tokens"] / d["prompt_tokens"],
        "wall_s": wall,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic["bytes_per_launch"] if traffic else None,
                     "alg_bytes_per_launch": alg_bytes / args.steps,
                     # the counted HBM bytes of the same launches over their duration
                     "measured_gbs": traffic["bytes_per_launch"] / launch_s / 1e9 if traffic else None,
                     "measured_frac": traffic["bytes_per_launch"] / launch_s / 1e9 / HBM_PEAK_GBS
                     if traffic else None},
    }
    if args.phase_timers:
        # 100 MHz ticks summed over the replicas' routing waves
        ticks = [sum(b["phase_ticks"][p] - a["phase_ticks"][p] for a, b in zip(reps0, reps1))
                 for p in range(K.KVR_PHASES)]
        line["phase_us_per_query"] = {name: t * 0.01 / nq for name, t in zip(K.PHASE_NAMES, ticks)}
        line["phase_us_per_query"]["total"] = sum(ticks) * 0.01 / nq
    if not args.no_whole:
        for k in range(args.warmup + args.steps, nb):
            run_batch(k)
            if (k + 1) % 10 == 0 or k + 1 == nb:
                ev[k][1].synchronize()
                log(f"rest of the stream: batch {k + 1}/{nb}")
        torch.cuda.synchronize()
        st, bits = sim.check()
        if st != K.KVR_OK:
            print(f"device status {st} bits {bits}: {K.kvr_last_error()}", file=sys.stderr)
            return 1
        whole_ms = sum(a.elapsed_time(b) for a, b in ev)
        line["whole_stream"] = {"value": R * stream.n / (whole_ms * 1e-3), "unit": "queries/s",
                                "ms": whole_ms, "batches": nb, "queries": stream.n}
    sim.close()
    del ds, out
    torch.cuda.empty_cache()
    if args.copy_probe_mib:
        src = torch.ones(args.copy_probe_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        line["copy_probe_bytes"] = src.numel()
        del src, dst
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(stream, W, B, q0, q, args.cpu_budget, R, args.evict, args.router,
                                            int(args.responses), args.beta, int(args.router_tree),
                                            args.router_tree_tokens)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
