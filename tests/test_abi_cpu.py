"""The C ABI on the CPU: the library loads, exports every function that
include/kvr.h declares, and rejects invalid configurations and arguments
before any device call."""
import math
import os
import re

import pytest

import paper_2601_18999_amd as K

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    txt = open(os.path.join(ROOT, "include", "kvr.h")).read()
    return sorted(set(re.findall(r"\b(kvr_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_function():
    lib = K.load_library()
    names = _declared()
    assert set(names) == set(K.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def test_config_default_holds_paper_constants():
    c = K.kvr_config_default(3, 4, 1000, 100)
    assert (c.num_replicas, c.num_workers, c.cache_tokens, c.max_query_tokens) == (3, 4, 1000, 100)
    assert c.abi_version == K.KVR_ABI_VERSION
    assert c.alpha_cached == 0.0 and c.alpha_miss == 1.0
    assert c.rho == 31.0 / 32.0 and c.decay_interval_us == 20000 and c.lr == 0.992
    assert c.cache_responses == 0 and c.batch_size == 1 and c.router_tree == 0


def test_continuous_batching_regions_only_when_used():
    base = K.kvr_workspace_size(K.kvr_config_default(2, 4, 1000, 100))
    b10 = K.kvr_workspace_size(K.kvr_config_default(2, 4, 1000, 100, batch_size=10))
    assert b10 > base
    assert K.kvr_workspace_size(K.kvr_config_default(2, 4, 1000, 100, batch_size=1)) == base


BAD = [
    dict(num_workers=0), dict(num_workers=65), dict(cache_tokens=0), dict(max_query_tokens=0),
    dict(max_query_tokens=1001), dict(evict=7), dict(router=4), dict(router=-1), dict(router=3, ca_balance_abs=-1),
    dict(update=9), dict(pending_capacity=0), dict(node_capacity=1), dict(arena_words=10),
    dict(rho=0.0), dict(rho=1.5), dict(rho=math.nan), dict(decay_interval_us=0), dict(lr=-1.0),
    dict(lr=math.inf), dict(nlms_eps=-1.0), dict(rls_p0=0.0), dict(alpha_miss=math.nan),
    dict(true_miss_us=-1), dict(num_replicas=0), dict(abi_version=1), dict(struct_size=8),
    dict(cache_responses=2), dict(batch_size=0), dict(batch_size=257), dict(batch_size=11),
    dict(router_tree=2), dict(router_tree=1, router_tree_tokens=50),
]


@pytest.mark.parametrize("bad", BAD, ids=[next(iter(b)) + "=" + str(list(b.values())[0]) for b in BAD])
def test_invalid_config_rejected_without_device(bad):
    c = K.kvr_config_default(2, 4, 1000, 100)
    for k, v in bad.items():
        setattr(c, k, v)
    with pytest.raises(K.KvrError) as ei:
        K.kvr_workspace_size(c)
    assert ei.value.status == K.KVR_EINVAL
    assert K.kvr_last_error()


def test_workspace_size_grows_with_every_dimension():
    base = K.kvr_workspace_size(K.kvr_config_default(2, 4, 1000, 100))
    for kw in (dict(R=3), dict(W=5), dict(B=2000)):
        a = dict(R=2, W=4, B=1000)
        a.update(kw)
        assert K.kvr_workspace_size(K.kvr_config_default(a["R"], a["W"], a["B"], 100)) > base


def test_null_context_and_arguments():
    lib = K.load_library()
    assert lib.kvr_route_batch(None, 1, None, None, None, None, None, None, None) == K.KVR_EINVAL
    assert lib.kvr_stats(None, None, 0, None, 0) == K.KVR_EINVAL
    assert lib.kvr_check(None, None) == K.KVR_EINVAL
    assert lib.kvr_queries_done(None) == 0
    lib.kvr_destroy(None)


def test_init_without_device_or_workspace():
    c = K.kvr_config_default(1, 2, 100, 10)
    with pytest.raises(K.KvrError) as ei:
        K.kvr_init_replicas(c, 0, 1 << 20)
    assert ei.value.status == K.KVR_EINVAL
    with pytest.raises(K.KvrError) as ei:
        K.kvr_init_replicas(c, 256, 16)  # too small
    assert ei.value.status == K.KVR_ENOMEM


def test_binding_structs_match_the_header(tmp_path):
    """Every field of kvr_config and kvr_worker_stats sits at the same offset
    in the ctypes binding as in the C header (compiled here with gcc)."""
    import ctypes
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "kvr.h"', "int main(void) {"]
    for cname, cls in (("kvr_config", K.KvrConfig), ("kvr_worker_stats", K.KvrWorkerStats),
                       ("kvr_replica_stats", K.KvrReplicaStats)):
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in cls._fields_:
            lines.append(f'  printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l}
    for cname, cls in (("kvr_config", K.KvrConfig), ("kvr_worker_stats", K.KvrWorkerStats),
                       ("kvr_replica_stats", K.KvrReplicaStats)):
        assert got[(cname, "size")] == ctypes.sizeof(cls), cname
        for f, _ in cls._fields_:
            assert got[(cname, f)] == getattr(cls, f).offset, (cname, f)
