"""Seeded synthetic query streams for the routing/eviction simulator.

This package is input plumbing only: it draws token ids, prefix-group
structure and arrival times, and holds none of the method's arithmetic
(no matching, scoring or eviction).  Both the CPU oracle (through the tests)
and the HIP library (through the tests and the benchmark) consume the arrays
it returns; neither side imports the other.

A stream is four arrays, the same for every replica:

* ``tokens``     int32  concatenated query token ids
* ``offsets``    uint64 ``n+1`` prefix offsets into ``tokens``
* ``arrival_us`` int64  non-decreasing arrival times (microseconds)
* ``out_len``    uint16 output length per query

The paper's workloads (Sec. 5 "Workloads", App. A) are GSP shared-prefix
groups, multi-turn conversations and long-document QA under Poisson arrivals
at 12 req/s with 4 output tokens.  Its datasets are not available here, so the
presets in :mod:`workload.gen` are synthetic stand-ins with the same shapes.
"""
from .gen import Stream, PRESETS, generate, preset_spec, small_spec  # noqa: F401
