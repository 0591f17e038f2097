"""kvr_stats_noalloc (the entry point for callers that cannot allocate
device memory) against kvr_stats, through the C ABI: identical records on
two calls in a row, the first on a context whose digest walks take several
groups of the static scratch, the second on a smaller one (the scratch keeps
the first call's contents); a tree too large for the scratch is refused."""
import numpy as np
import pytest

import paper_2601_18999_amd as K
from workload import generate, small_spec
from gpu_helpers import note

pytestmark = pytest.mark.gpu


def _both(sim):
    reps, ws = K.kvr_stats(sim.ctx, sim.R, sim.W, with_replicas=True)
    reps2, ws2 = K.kvr_stats_noalloc(sim.ctx, sim.R, sim.W)
    return (reps, ws), (reps2, ws2)


def _same(a, b):
    (ra, wa), (rb, wb) = a, b
    assert ra == rb
    assert wa == wb


def test_noalloc_stats_equal_kvr_stats_on_two_calls():
    # first call: 4 x 8 workers whose 200,003-node trees need 3.2 MB of FIFO
    # each, so the 32 MiB scratch takes them ten at a time
    s = generate(small_spec(n=300, groups=6, prefix_len=(10, 80), suffix_len=(5, 40), vocab=40, seed=9))
    sim = K.Simulator(4, 8, 200000, s.max_len)
    try:
        sim.run(s, batch=128, all_hits=False)
        a, b = _both(sim)
        note(f"first call: {sum(w['resident'] for rr in a[1] for w in rr)} tokens cached")
        _same(a, b)
        assert all(r["queries"] == s.n for r in b[0])
    finally:
        sim.close()
    # second call, smaller: 2 x 3 workers with 300-token caches (evicting)
    s2 = generate(small_spec(n=200, groups=5, prefix_len=(5, 40), suffix_len=(3, 25), vocab=11, seed=4))
    sim = K.Simulator(2, 3, 300, s2.max_len)
    try:
        sim.run(s2, batch=64, all_hits=False)
        a, b = _both(sim)
        assert sum(w["evictions"] for rr in b[1] for w in rr) > 0
        _same(a, b)
    finally:
        sim.close()


def test_noalloc_stats_refuse_a_tree_larger_than_the_scratch():
    # 2,097,152-token cache: its digest walk needs 32 MiB + of FIFO alone
    sim = K.Simulator(1, 1, 1 << 21, 64)
    try:
        with pytest.raises(K.KvrError) as ei:
            K.kvr_stats_noalloc(sim.ctx, 1, 1)
        assert ei.value.status == K.KVR_EINVAL
        assert "scratch" in str(ei.value)
    finally:
        sim.close()
