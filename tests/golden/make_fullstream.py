#!/usr/bin/env python3
"""Write the whole-stream oracle digests of the full-size workloads.

For each workload (two-level prompts, multi-turn sessions, long prompts: the
three largest presets, default settings: RLT eviction, LBGR routing, NLMS
update) and each sampled replica (the first and the last), run the CPU
oracle over the WHOLE stream and store, per block of 2,000 queries, the
digests of ``tests/fullstream_digests.py`` (routes and hits, every h_ij, the
integer state of every worker after the block), plus the final state of
every worker in full and a hash of the generated stream.

Calls only ``oracle/`` (and ``workload/`` for the inputs).  Slow: the
long-prompt workload takes over an hour per replica on one core, so the
replicas and workloads run on parallel threads (the oracle releases the GIL).

    python tests/golden/make_fullstream.py            # workloads 3 4 5
    python tests/golden/make_fullstream.py --config 3
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
TESTS = os.path.dirname(HERE)
ROOT = os.path.dirname(TESTS)
for p in (ROOT, TESTS):
    if p not in sys.path:
        sys.path.insert(0, p)

from oracle import oracle as O  # noqa: E402
from workload import PRESETS, generate  # noqa: E402
import fullstream_digests as D  # noqa: E402


def golden_path(cfg: int) -> str:
    return os.path.join(HERE, f"fullstream_{PRESETS[cfg]['name']}.json")


def one(cfg: int, stream, replica: int, t0: float):
    p = PRESETS[cfg]
    W, B = p["W"], p["B"]
    print(f"[golden] {p['name']} replica {replica}: start", flush=True)
    o = O.run(stream, W, B, replica=replica, all_hits=True, snap_every=D.BLOCK)
    assert o["rc"] == 0, o["rc"]
    assert o["done"] == stream.n
    d = D.block_digests(o["route"], o["hits"], o["all_hits"])
    d["state"] = [D.state_digest(ws) for ws in o["snaps"]]
    d["final_workers"] = o["workers"]
    d["evictions"] = int(sum(w["evictions"] for w in o["workers"]))
    d["hit_tokens"] = int(sum(w["hit_tokens"] for w in o["workers"]))
    print(f"[golden] {p['name']} replica {replica}: done at {time.time() - t0:.0f} s "
          f"({d['evictions']} evictions)", flush=True)
    return d


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", type=int, nargs="+", default=[3, 4, 5])
    args = ap.parse_args()
    O.lib()
    t0 = time.time()
    streams, futs = {}, {}
    with cf.ThreadPoolExecutor(max_workers=2 * len(args.config)) as ex:
        for cfg in args.config:
            p = PRESETS[cfg]
            s = generate(p["stream"])
            streams[cfg] = s
            print(f"[golden] {p['name']}: {s.n} queries, {s.tokens.size} tokens", flush=True)
            for r in sorted({0, p["R"] - 1}):
                futs[(cfg, r)] = ex.submit(one, cfg, s, r, t0)
        for cfg in args.config:
            p = PRESETS[cfg]
            s = streams[cfg]
            rep = {str(r): futs[(cfg, r)].result() for r in sorted({0, p["R"] - 1})}
            out = {"workload": p["name"], "R": p["R"], "W": p["W"], "B": p["B"], "n": s.n,
                   "block": D.BLOCK, "stream_xxh3": D.stream_hash(s),
                   "oracle": "RLT eviction, LBGR routing, NLMS update, seed 0", "replicas": rep}
            with open(golden_path(cfg), "w") as f:
                json.dump(out, f, separators=(",", ":"))
                f.write("\n")
            print(f"[golden] wrote {golden_path(cfg)}", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
