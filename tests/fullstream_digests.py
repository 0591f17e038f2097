"""Compact digests of a whole-stream run, for bit-exact comparison of the HIP
path with the oracle over streams too long to keep every output.

Test infrastructure: hashes outputs of either side with one recipe; it holds
none of the method's arithmetic.

Per block of ``BLOCK`` queries (the benchmark's batch) and per replica:

* ``routes``  - xxh3-64 of the block's routed worker ids (int32) followed by
  the routed hits (int32);
* ``all_hits`` - xxh3-64 of the block's h_ij rows (int32, W per query);
* ``state``   - xxh3-64 of every worker's integer state after the block
  (the fields of ``INT_FIELDS``, as uint64, worker-major).

The float state (load estimate, residual model) is kept in full for the
final state only and compared to a relative tolerance.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np
import xxhash

BLOCK = 2000

INT_FIELDS = ["routed", "prompt_tokens", "hit_tokens", "matched_tokens", "loads", "evictions",
              "phase", "cnt", "forced_resets", "resident", "digest_sum", "digest_xor",
              "marked_count", "marked_sum", "completions", "pending_depth", "pending_max",
              "latency_sum_us", "latency_max_us", "backlog_us", "last_decay_us",
              "router_resident", "router_digest_sum", "router_digest_xor", "router_evictions"]

_MASK = (1 << 64) - 1


def h64(*arrays: np.ndarray) -> str:
    x = xxhash.xxh3_64()
    for a in arrays:
        x.update(np.ascontiguousarray(a).tobytes())
    return x.hexdigest()


def stream_hash(stream) -> str:
    """xxh3-64 of the four stream arrays (tokens, offsets, arrivals, output
    lengths), so a change of the generator is told apart from a change of
    either implementation."""
    return h64(stream.tokens.astype(np.int32, copy=False), stream.offsets.astype(np.uint64, copy=False),
               stream.arrival_us.astype(np.int64, copy=False), stream.out_len.astype(np.uint16, copy=False))


def route_digest(route: np.ndarray, hits: np.ndarray) -> str:
    return h64(route.astype(np.int32, copy=False), hits.astype(np.int32, copy=False))


def all_hits_digest(all_hits: np.ndarray) -> str:
    return h64(all_hits.astype(np.int32, copy=False))


def state_digest(workers: Sequence[Dict]) -> str:
    a = np.array([[int(w[f]) & _MASK for f in INT_FIELDS] for w in workers], dtype=np.uint64)
    return h64(a)


def block_digests(route: np.ndarray, hits: np.ndarray, all_hits=None, block: int = BLOCK) -> Dict[str, List[str]]:
    n = route.shape[0]
    out = {"routes": [route_digest(route[b:b + block], hits[b:b + block]) for b in range(0, n, block)]}
    if all_hits is not None:
        out["all_hits"] = [all_hits_digest(all_hits[b:b + block]) for b in range(0, n, block)]
    return out
