"""Small hand-built query streams shared by the CPU and GPU tests (input
plumbing only: no matching, scoring or eviction here)."""
from __future__ import annotations

import numpy as np

from workload.gen import Stream


def random_response_stream(rng: np.random.Generator, n: int, vocab: int, max_prompt: int, max_resp: int,
                           B: int) -> Stream:
    """Random complete paths q || a (prompt 1..max_prompt tokens, response
    0..max_resp tokens, |q| + |a| <= B) over a small vocabulary, so prompts
    are often cached whole and the responses after them partly cached too;
    Poisson-like arrivals up to 0.4 s apart."""
    lens, olen, toks = [], [], []
    for _ in range(n):
        L = int(rng.integers(1, max(1, min(max_prompt, B - max_resp)) + 1))
        o = int(rng.integers(0, max_resp + 1))
        toks.append(rng.integers(0, vocab, size=L + o).astype(np.int32))
        lens.append(L + o)
        olen.append(o)
    off = np.zeros(n + 1, dtype=np.uint64)
    off[1:] = np.cumsum(lens)
    return Stream(tokens=np.concatenate(toks), offsets=off,
                  arrival_us=np.cumsum(rng.integers(1, 400000, size=n)).astype(np.int64),
                  out_len=np.array(olen, dtype=np.uint16), spec={"kind": "random_responses", "n": n})
