"""Run in a process that preloads the AddressSanitizer runtime (see
test_sanitizers_cpu.py): the single-lane replay of the kernel's per-wave
logic and the CPU oracle, both built with AddressSanitizer and
UndefinedBehaviorSanitizer (every error aborts), on cases that reach every
path: random streams under RLT and L-LRU with continuous batching, the
approximate router tree, cached responses, collector pressure, the staged and
unstaged candidate list, the pipelined order; the oracle's brute-force and
invariant pins.  Exits non-zero on the first mismatch."""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)
sys.path.insert(0, os.path.dirname(HERE))

import ctypes  # noqa: E402

import numpy as np  # noqa: E402

import emul_kernel as E  # noqa: E402
import paper_2601_18999_amd as K  # noqa: E402
from oracle import oracle as O  # noqa: E402
from workload import generate, small_spec  # noqa: E402
import spec_model as SM  # noqa: E402
from streams import random_response_stream  # noqa: E402


def main() -> int:
    O.use_library(O.build(sanitize=True))
    lib = ctypes.CDLL(E.build(sanitize=True))
    lib.emul_run.restype = ctypes.c_int
    lib.emul_run.argtypes = [ctypes.POINTER(K.KvrConfig), ctypes.c_uint64] + [ctypes.c_void_p] * 9 + [ctypes.c_uint32]
    lib.emul_pipe_unsafe.restype = ctypes.c_uint64
    lib.emul_pipe_steps.restype = ctypes.c_uint64
    E._lib = lib
    rng = np.random.default_rng(2024)
    cases = 0
    for case in range(48):
        beta = int(rng.integers(1, 4))
        s = generate(small_spec(n=int(rng.integers(30, 160)), groups=int(rng.integers(1, 8)), prefix_len=(1, 30),
                                suffix_len=(1, 25), vocab=int(rng.integers(2, 10)), seed=500 + case))
        resp = case % 4 == 3
        if resp:
            s = random_response_stream(rng, int(rng.integers(30, 120)), int(rng.integers(2, 8)), 20, 6,
                                       int(max(60, 3 * 26)))
        W = int(rng.integers(1, 4))
        B = int(max(beta * s.max_len, rng.integers(2, 200)))
        evict = ["rlt", "lru"][case % 2]
        rt = case % 3 == 1
        arena = 2 * B + 2 * s.max_len + 64 if case % 5 == 0 else 0
        cfg = dict(batch_size=beta, evict={"rlt": 0, "lru": 1}[evict], router_tree=int(rt),
                   router_tree_tokens=int(max(s.max_len, 40)) if rt else 0, cache_responses=int(resp),
                   arena_words=arena)
        e = E.run(s, 2, W, B, ucap=[0, 8192][case % 2], **cfg)
        assert e["rc"] == 0, (case, e["rc"])
        for r in range(2):
            o = O.run(s, W, B, replica=r, all_hits=True, evict=evict, batch_size=beta, router_tree=int(rt),
                      router_tree_tokens=int(max(s.max_len, 40)) if rt else 0, cache_responses=int(resp), check=1)
            assert o["rc"] == 0, (case, r, o["rc"])
            assert (e["route"][r] == o["route"]).all(), (case, r)
            assert (e["all_hits"][r] == o["all_hits"]).all(), (case, r)
        cases += 1
    # the oracle against the brute-force model of tests/spec_model.py
    for seed in range(12):
        s = generate(small_spec(n=60, groups=4, prefix_len=(1, 8), suffix_len=(1, 5), vocab=4, seed=seed))
        B = max(12, s.max_len)
        for evict in ("rlt", "lru"):
            o = O.run(s, 2, B, replica=seed, all_hits=True, evict=evict, check=1, u_mode=seed % 2)
            _, routes, _, allh = SM.run_spec(s, 2, B, replica=seed, evict=evict)
            assert o["rc"] == 0 and (o["route"] == routes).all(), (seed, evict)
            assert (o["all_hits"] == allh).all(), (seed, evict)
    for which in (1, 2, 3):
        assert O.check_selftest(which)
    print(f"sanitized replay ok: {cases} kernel-logic cases, oracle pins", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
