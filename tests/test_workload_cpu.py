"""The synthetic stream recipes keep the shapes they promise (input plumbing;
no method arithmetic here)."""
import numpy as np

from workload import PRESETS, generate


def test_gsp_paper_shape_and_orders():
    """App. A's GSP: 128 groups x 32 queries, prompt lengths cycling over
    512..8192 across groups, prefix ratio 0.5; the round-robin order issues
    one query per group per turn, the groups in a fixed cycle."""
    for cfg, order in ((6, "random"), (7, "round_robin")):
        sp = PRESETS[cfg]["stream"]
        s = generate(sp)
        assert s.n == 128 * 32 and sp["order"] == order
        lens = s.lengths
        assert sorted(set(lens.tolist())) == [512, 1024, 2048, 4096, 8192]
        # group of each query: by its prefix
        prefix_of = {}
        groups = []
        for j in range(s.n):
            q = s.query(j)
            key = (len(q), bytes(q[: len(q) // 2].tobytes()))
            groups.append(prefix_of.setdefault(key, len(prefix_of)))
        groups = np.array(groups)
        assert len(prefix_of) == 128
        assert (np.bincount(groups) == 32).all()
        if order == "round_robin":
            # every turn visits all groups in the same cycle
            cyc = groups[:128]
            assert len(set(cyc.tolist())) == 128
            assert (groups.reshape(32, 128) == cyc[None, :]).all()
        else:
            assert not (groups[:128] == groups[128:256]).all()
    # suffixes are fresh: two queries of a group share exactly the prefix
    s = generate(PRESETS[7]["stream"])
    a, b = s.query(0), s.query(128)
    half = len(a) // 2
    assert len(a) == len(b) and (a[:half] == b[:half]).all() and (a[half:] != b[half:]).any()
