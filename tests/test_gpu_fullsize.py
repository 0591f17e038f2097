"""Full-size workloads (configs 3, 4 and 5: every replica, worker count and
cache budget at its real size) in the launch configuration the benchmark
times (batches of 2,000 queries, all replicas in one launch).

* Parity: sampled replicas are compared element by element with the CPU
  oracle over a prefix of the stream long enough to fill every cache and run
  many eviction phases (routes, every h_ij, hits, counters, digests and marks
  bit-exact; load estimate and residual model to 1e-9 relative).
* Whole stream: the remaining queries run on the GPU and are checked with
  properties that hold at any size: the device's own consistency checks,
  routes in range, h <= |q|, per-worker |S| <= B and |S| = loads - evictions,
  and the counters agreeing with the returned routes and hits.
"""
import concurrent.futures as cf
import time

import numpy as np
import pytest

import paper_2601_18999_amd as K
from oracle import oracle as O
from workload import PRESETS, generate
from gpu_helpers import compare_worker, note

pytestmark = pytest.mark.gpu

BATCH = 2000
# (config, sampled replicas, prefix compared with the oracle, eviction,
# cached responses: every turn's 4-token response is cached with its prompt
# and is part of the next turn's prompt, batch size of continuous batching,
# approximate router tree with the cache's budget)
CASES = [
    (3, [0, 85, 170, 255], 24000, "rlt", 0, 1, 0),
    (4, [0, 42, 127], 24000, "rlt", 0, 1, 0),
    (5, [0, 31], 8000, "rlt", 0, 1, 0),
    (3, [0, 255], 24000, "lru", 0, 1, 0),
    (5, [0, 31], 8000, "lru", 0, 1, 0),
    (4, [0, 127], 24000, "rlt", 1, 1, 0),
    (5, [0, 31], 8000, "rlt", 0, 16, 0),
    (4, [0, 127], 24000, "lru", 1, 16, 0),
    (5, [0, 31], 8000, "rlt", 0, 1, 1),
    (4, [0, 127], 24000, "rlt", 1, 1, 1),
]


def _oracle_many(stream, W, B, replicas, n, evict, resp, beta, rt):
    with cf.ThreadPoolExecutor(max_workers=len(replicas)) as ex:
        futs = {r: ex.submit(O.run, stream, W, B, replica=r, n=n, all_hits=True, evict=evict,
                             cache_responses=resp, batch_size=beta, router_tree=rt) for r in replicas}
        return {r: f.result() for r, f in futs.items()}


@pytest.mark.parametrize("cfg,replicas,nprefix,evict,resp,beta,rt", CASES,
                         ids=[f"config{c[0]}-{c[3]}" + ("-responses" if c[4] else "") +
                              (f"-batch{c[5]}" if c[5] > 1 else "") + ("-routertree" if c[6] else "")
                              for c in CASES])
def test_full_size(cfg, replicas, nprefix, evict, resp, beta, rt):
    p = PRESETS[cfg]
    R, W, B = p["R"], p["W"], p["B"]
    t0 = time.time()
    s = generate(dict(p["stream"], responses=True) if resp else p["stream"])
    note(f"config {cfg}: R={R} W={W} B={B} n={s.n} tokens={s.tokens.size} responses={resp} batch={beta} "
         f"router_tree={rt} ({time.time() - t0:.1f} s)")
    assert nprefix % BATCH == 0 and nprefix < s.n

    # the oracle runs on host threads while the GPU works
    pool = cf.ThreadPoolExecutor(max_workers=1)
    ofut = pool.submit(_oracle_many, s, W, B, replicas, nprefix, evict, resp, beta, rt)

    sim = K.Simulator(R, W, B, s.max_len, evict={"rlt": K.KVR_EVICT_RLT, "lru": K.KVR_EVICT_LRU}[evict],
                      cache_responses=resp, batch_size=beta, router_tree=rt)
    try:
        ds = sim.upload(s)
        route = np.empty((R, s.n), np.int32)
        hits = np.empty((R, s.n), np.int32)
        allh = np.empty((R, nprefix, W), np.int32)
        t1 = time.time()
        for start in range(0, s.n, BATCH):
            m = min(BATCH, s.n - start)
            ah = start < nprefix
            out = sim.route(ds, start, m, all_hits=ah)
            sim.stream.synchronize()
            route[:, start:start + m] = out["route"].cpu().numpy()
            hits[:, start:start + m] = out["hits"].cpu().numpy()
            if ah:
                allh[:, start:start + m] = out["all_hits"].cpu().numpy()
            if start + m == nprefix:
                st, bits = sim.check()
                assert st == K.KVR_OK, (st, bits, K.kvr_last_error())
                prefix_stats = sim.stats(check=False)
                note(f"  prefix of {nprefix} routed ({time.time() - t1:.1f} s)")
        st, bits = sim.check()
        assert st == K.KVR_OK, (st, bits, K.kvr_last_error())
        stats = sim.stats(check=False)
        note(f"  whole stream routed ({time.time() - t1:.1f} s)")
    finally:
        sim.close()

    # ---- sampled parity on the prefix
    orc = ofut.result()
    pool.shutdown()
    note(f"  oracle on replicas {replicas} done ({time.time() - t0:.1f} s since start)")
    for r in replicas:
        o = orc[r]
        assert o["rc"] == 0
        bad = np.nonzero(route[r, :nprefix] != o["route"])[0]
        assert bad.size == 0, f"replica {r}: first route mismatch at query {bad[:5]}"
        np.testing.assert_array_equal(hits[r, :nprefix], o["hits"], err_msg=f"hits r={r}")
        np.testing.assert_array_equal(allh[r], o["all_hits"], err_msg=f"all_hits r={r}")
        for i in range(W):
            compare_worker(prefix_stats[r][i], o["workers"][i], where=f"r={r} i={i}")
    ev = sum(w["evictions"] for w in orc[replicas[0]]["workers"])
    ph = sum(w["phase"] - 1 for w in orc[replicas[0]]["workers"])
    note(f"  oracle replica {replicas[0]}: {ev} evictions, {ph} phase resets in the prefix")
    assert ev > 10 * B and (ph > 0 or evict == "lru"), (ev, ph)  # the prefix runs deep into eviction
    if evict == "lru":  # no randomness: every replica is the same over the whole stream
        assert (route == route[0:1]).all() and (hits == hits[0:1]).all()

    # ---- whole stream: properties
    paths = s.lengths.astype(np.int64)
    lens = paths - s.out_len.astype(np.int64) if resp else paths  # the prompts
    assert ((route >= 0) & (route < W)).all()
    assert ((hits >= 0) & (hits <= lens[None, :])).all()
    for r in range(R):
        ws = stats[r]
        for i, w in enumerate(ws):
            assert w["resident"] <= B, (r, i, w["resident"])
            assert w["resident"] == w["loads"] - w["evictions"], (r, i)
            assert w["cnt"] <= B
            assert w["marked_count"] <= w["resident"]
        routed = np.bincount(route[r], minlength=W)
        assert [w["routed"] for w in ws] == routed.tolist(), r
        assert sum(w["hit_tokens"] for w in ws) == int(hits[r].astype(np.int64).sum()), r
        assert sum(w["prompt_tokens"] for w in ws) == int(lens.sum()), r
        per_w_prompt = np.bincount(route[r], weights=lens, minlength=W)
        assert [w["prompt_tokens"] for w in ws] == per_w_prompt.astype(np.int64).tolist(), r
        # every routed query's missed tokens are loaded (with responses, the
        # part of the path after a wholly cached prompt may be cached too)
        miss = np.bincount(route[r], weights=paths - hits[r], minlength=W).astype(np.int64)
        if resp:
            assert all(w["loads"] <= m for w, m in zip(ws, miss.tolist())), r
        else:
            assert [w["loads"] for w in ws] == miss.tolist(), r
    note(f"  evictions on the GPU: {sum(w['evictions'] for rr in stats for w in rr)}")
