"""Shared helpers for the GPU tests: run the HIP path through the C ABI and
compare with the CPU oracle element by element."""
from __future__ import annotations

import sys

import numpy as np

import paper_2601_18999_amd as K
from oracle import oracle as O

# float state (load estimate, residual model) must agree to this relative
# tolerance; everything else is compared exactly
FLOAT_RTOL = 1e-9

_UPD = {"nlms": K.KVR_UPD_NLMS, "rls": K.KVR_UPD_RLS, "none": K.KVR_UPD_NONE}


def note(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_run(stream, R, W, B, batch=0, all_hits=True, max_len=None, update="nlms", **cfg):
    sim = K.Simulator(R, W, B, max_len or max(1, stream.max_len), update=_UPD[update], **cfg)
    try:
        res = sim.run(stream, batch=batch, all_hits=all_hits)
        st, bits = sim.check()
        stats = sim.stats(check=False)
    finally:
        sim.close()
    res["status"], res["bits"] = st, bits
    return res, stats


def compare_worker(g, c, where=""):
    for k, v in c.items():
        if k in ("load_est",):
            assert np.isclose(g[k], v, rtol=FLOAT_RTOL, atol=0.0), (where, k, g[k], v)
        elif k == "theta":
            np.testing.assert_allclose(g[k], v, rtol=FLOAT_RTOL, atol=1e-300, err_msg=f"{where} theta")
        else:
            assert g[k] == v, (where, k, g[k], v)


def assert_parity(stream, res, stats, W, B, replicas, n=None, update="nlms", seed=0, check_stats=True,
                  evict="rlt", **okw):
    """okw: further oracle settings (router, cache-aware thresholds)."""
    n = stream.n if n is None else n
    assert res["status"] == K.KVR_OK, (res["status"], res["bits"])
    for r in replicas:
        o = O.run(stream, W, B, replica=int(r), n=n, all_hits=True, update=update, seed=seed, evict=evict, **okw)
        assert o["rc"] == 0
        rt = res["route"][r][:n]
        bad = np.nonzero(rt != o["route"])[0]
        assert bad.size == 0, f"replica {r}: first route mismatch at query {bad[:5]}"
        np.testing.assert_array_equal(res["hits"][r][:n], o["hits"], err_msg=f"hits r={r}")
        if res.get("all_hits") is not None:
            np.testing.assert_array_equal(res["all_hits"][r][:n], o["all_hits"], err_msg=f"all_hits r={r}")
        if check_stats:
            for i in range(W):
                compare_worker(stats[r][i], o["workers"][i], where=f"r={r} i={i}")
